/*
 * nuna.h -- C ABI of libnuna: single-GPU collective copy/reduce kernels for
 * MI355X (gfx950) with NUNA-aware (XCD) or locality-unaware (linear)
 * placement of workgroups and the data chunks they touch.
 *
 * What is computed.  The collectives are the ones the paper names as the
 * common AI patterns (Sec. 2.1 "Collective Communications": all-reduce for
 * gradients and partial activations, all-gather for split weights,
 * all-to-all for MoE token routing; reduce-scatter with all-gather in the
 * tensor-parallel traces of the same section).  P "ranks" are P buffers in
 * this GPU's own HBM: one call runs the copy/reduce work of all P ranks of a
 * direct (all-pairs) collective (Sec. 5.1 evaluates that algorithm).
 *
 * Numerics.  Reductions are sums.  Each output element is
 *     acc = in[0][i]; acc = acc + in[1][i]; ... ; acc = acc + in[P-1][i]
 * in fp32 (bf16 inputs are widened exactly), then rounded once to the buffer
 * dtype with round-to-nearest-even.  The order is fixed (ascending rank), so
 * results are bitwise reproducible and independent of placement mode,
 * algorithm and launch shape.  Copies (all-gather, all-to-all) move bytes.
 *
 * Placement (Sec. 4.2, Algorithm 1; configurations UA and NAP* of Sec. 5.3).
 * Workgroup b of a launch runs on XCD (b mod 8) on MI355X.
 *   NUNA_PLACE_LINEAR  work item w runs on workgroup w (grid-stride): the
 *                      round-robin, locality-unaware baseline (UA).
 *   NUNA_PLACE_XCD     work items that touch the same data form one logical
 *                      group; groups are dealt round-robin to the 8 XCDs and
 *                      a group's members run concurrently on one XCD,
 *                      sharing its L2 (NAP* -- aware workgroup placement,
 *                      default page placement).  Groups are the work items
 *                      of one input chunk (split all-reduce, split
 *                      all-gather), the copies of one token row (all-to-all
 *                      dispatch), and, for one-work-item-per-workgroup
 *                      launches whose chunks are smaller than a 4 KiB page,
 *                      the chunks of one page when NUNA_PAGE_GROUPS asks for
 *                      it (Sec. 4.2: 4 kB pages).  A group of one work item is placed
 *                      as LINEAR places it.  Chunk groups stay together only
 *                      where the members' L2 re-reads are at least a quarter
 *                      of the group's traffic and, for the split all-reduce,
 *                      the launch moves more than 256 KiB; elsewhere XCD runs
 *                      the linear map.  XCD mode needs nuna_init to have
 *                      verified the dispatch map on the current device (else
 *                      NUNA_ERR_UNSUPPORTED); LINEAR needs nothing.
 * The mode changes which workgroup computes what, never the result.
 *
 * Buffers and ownership.  All data buffers are device memory owned by the
 * caller.  `in`/`out`/`send`/`recv` are HOST arrays of P device pointers; they
 * are read during the call only (their values are copied into kernel
 * arguments, so a captured HIP graph keeps them).  The library allocates no
 * device memory inside the collective calls; only nuna_a2a_layout_upload
 * does, and the layout owns it until nuna_a2a_layout_destroy.
 *
 * Streams.  Collective calls enqueue on `stream` (NULL = the null stream),
 * return without synchronising, and make no allocation, blocking copy or
 * synchronisation, so they can be captured into a HIP graph.
 *
 * Threads.  Collective, layout and planner calls may run concurrently from
 * several host threads; each thread keeps its own error text.  A layout is
 * read-only once uploaded and may be shared by concurrent calls.  The
 * setters nuna_set_max_workgroups and nuna_set_tunable change process-wide
 * launch shapes and must not race with other calls.
 *
 * Interface additions to the plain collective calls (kept because a single
 * GPU needs them): the all-to-all calls take the receive capacity of the
 * caller's buffers (recv_capacity_rows, y_capacity_rows), so the library can
 * check them; layouts are planned on the host (nuna_a2a_layout_create) and
 * copied to the device by a separate call (nuna_a2a_layout_upload), which is
 * the only allocating step; the algorithm enum adds the destination-split
 * one-shot and the two-kernel two-shot; NUNA_ERR_NO_MEMORY reports host
 * memory exhaustion.
 *
 * Errors.  Every call returns a status and never aborts or lets an exception
 * out.  All argument checks run on the host before any HIP call.  On failure,
 * nuna_last_error_string() describes the problem (per thread).  A launch
 * failure is NUNA_ERR_HIP; host memory exhausted while building the call's
 * own tables (layouts, plans) is NUNA_ERR_NO_MEMORY, and nothing is leaked.
 */
#ifndef NUNA_H
#define NUNA_H

#include <stddef.h>
#include <stdint.h>

/* Plain C and C++ compilers other than hipcc compile this header with
 * -D__HIP_PLATFORM_AMD__ and -I/opt/rocm/include, as HIP's own headers
 * require; it is C99. */
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    NUNA_OK = 0,
    NUNA_ERR_INVALID_ARG = 1, /* null pointer, P out of [1,64], bad enum, size overflow, bad layout */
    NUNA_ERR_UNSUPPORTED = 2, /* dtype / combination not provided */
    NUNA_ERR_MISALIGNED = 3,  /* a data pointer is not 16-byte aligned */
    NUNA_ERR_OVERLAP = 4,     /* buffers overlap other than in the documented in-place forms */
    NUNA_ERR_HIP = 5,         /* the HIP runtime reported an error (no device, launch failure, ...) */
    NUNA_ERR_NO_MEMORY = 6    /* host memory for the call's own tables could not be allocated */
} nuna_status_t;

typedef enum { NUNA_F32 = 0, NUNA_BF16 = 1 } nuna_dtype_t;

typedef enum { NUNA_PLACE_LINEAR = 0, NUNA_PLACE_XCD = 1 } nuna_placement_t;

typedef enum {
    NUNA_ALGO_AUTO = 0,           /* library picks by size: NUNA_ALGO_TWO_SHOT for 8 ranks of bf16
                                     from 16 MiB per rank when a shard is whole 16-byte vectors,
                                     NUNA_ALGO_ONE_SHOT otherwise */
    NUNA_ALGO_ONE_SHOT = 1,       /* one kernel: read P inputs, write P outputs per element */
    NUNA_ALGO_TWO_SHOT = 2,       /* reduce-scatter then all-gather, both phases per chunk in one
                                     kernel: the workgroup that reduces chunk c of shard r stores
                                     it to out[r], then to every other out[d].  Runs the two
                                     kernels of NUNA_ALGO_TWO_SHOT_TWO_KERNELS when P is not 2,
                                     4, 8 or 16, a shard is not whole 16-byte vectors, or at the
                                     sizes where they measured faster (NUNA_TWO_SHOT_FORM) */
    NUNA_ALGO_ONE_SHOT_SPLIT = 3, /* one kernel, work item = (chunk, destination group): more
                                     workgroups for small messages; inputs re-read per group */
    NUNA_ALGO_TWO_SHOT_TWO_KERNELS = 4 /* reduce-scatter kernel, then all-gather kernel (stream
                                     ordered): the phase boundary is the kernel boundary */
} nuna_algo_t;

#define NUNA_MAX_RANKS 64
#define NUNA_NUM_XCD 8

/* Probe the current device and cache the result (Sec. 4.2.3 hands the
 * topology to the placement step; this is where the library learns it).
 * Checks that the device is gfx950, then launches 2048 one-wave workgroups
 * that each record the XCC they ran on, and verifies the dispatch map XCD
 * placement relies on: 256 compute units and workgroup b on XCD b mod 8 for
 * every b (nuna_check_dispatch_map).  Allocates 8 KiB of device memory for
 * the probe and frees it; synchronous, not capturable.  Idempotent and
 * thread-safe; call it once on every device before XCD-mode collectives
 * (LINEAR-mode calls work without it).  Returns NUNA_ERR_HIP without a
 * device, NUNA_ERR_UNSUPPORTED if the device is not gfx950 or the map does
 * not hold (XCD placement then stays unavailable on that device). */
nuna_status_t nuna_init(void);

/* What nuna_init found on the current device. */
typedef struct {
    int32_t device;       /* HIP device ordinal */
    int32_t cu_count;     /* compute units */
    int32_t xcd_count;    /* distinct XCC ids seen by the probe (1 + largest) */
    int32_t map_verified; /* 1: workgroup b runs on XCD b mod 8; XCD placement available */
} nuna_device_info_t;

/* Fill *info for the current device.  NUNA_ERR_INVALID_ARG if nuna_init has
 * not run on it (or info is NULL). */
nuna_status_t nuna_get_device_info(nuna_device_info_t* info);

/* Launches of the calling thread's last collective call (nuna_allreduce,
 * nuna_reduce_scatter, nuna_all_gather, nuna_all_to_all,
 * nuna_all_to_all_combine): which kernels ran and under which map.  A call
 * that launched nothing (count 0, an argument error) leaves launches == 0.
 * Lets a caller or a benchmark see whether the two placement modes ran the
 * same launches. */
#define NUNA_MAP_LINEAR 0     /* workgroup b runs work item b (grid-stride) */
#define NUNA_MAP_XCD_GROUPS 1 /* logical groups of work items sharing a chunk, one XCD each */
#define NUNA_MAP_XCD_PAGES 2  /* the chunks of each 4 KiB page on one XCD */
#define NUNA_MAP_XCD_LISTS 3  /* per-XCD work lists from the placement planner (all-to-all) */
#define NUNA_MAP_XCD_SHARDS 4 /* fused two-shot: every chunk of shard r on XCD r mod 8 */
typedef struct {
    char kernels[96];           /* kernel names, '+'-separated, in launch order */
    int32_t launches;           /* kernels launched */
    int32_t map;                /* NUNA_MAP_*: a non-linear map if any launch ran one */
    int64_t group_size;         /* work items per logical group of that map (0: variable) */
    int64_t grid;               /* workgroups of the last launch */
    int32_t threads;            /* workgroup size of the last launch */
    int32_t vectors_per_thread; /* 16-byte vectors per thread per work item of the last launch */
} nuna_launch_info_t;

nuna_status_t nuna_last_launch(nuna_launch_info_t* info);

/* Host-only check behind nuna_init (no HIP call): xcc[b] is the XCC
 * workgroup b of a G-workgroup launch ran on (HOST int32 array, G >= 64).
 * NUNA_OK if cu_count is 256 and xcc[b] == b mod 8 for every b, else
 * NUNA_ERR_UNSUPPORTED naming the first mismatch (NUNA_ERR_INVALID_ARG for a
 * NULL array or G < 64). */
nuna_status_t nuna_check_dispatch_map(const int32_t* xcc, int64_t G, int32_t cu_count);

/* Text of the last error raised on the calling thread ("" if none).  The
 * string is owned by the library and valid until the thread's next call. */
const char* nuna_last_error_string(void);

/* Library version as major*10000 + minor*100 + patch. */
int nuna_version(void);

/* Cap on workgroups per kernel launch for all later calls of the process
 * (0 restores the default, 16384).  Work beyond the cap is looped over by
 * each workgroup (persistent loop), in the same placement.  Without a cap set
 * here or through NUNA_MAX_GRID, the 8-rank all-gather and the MoE dispatch
 * run one workgroup per work item up to 2^20 workgroups; a cap that is set
 * bounds them too.  Changes the launch shape only, never results; lets a
 * caller leave compute units free for concurrent kernels.  Returns
 * NUNA_ERR_INVALID_ARG for values < 0. */
nuna_status_t nuna_set_max_workgroups(int max_workgroups);

/* Launch-shape tunables, by the name of the environment variable that also
 * sets them at load time.  They choose workgroup sizes, vectors per thread,
 * kernel variants and grid caps; they never change results.  A setting
 * applies to later calls of the process; it must not race with other calls
 * into the library.
 *   NUNA_MAX_GRID         default workgroup cap, 0..INT32_MAX (0: 16384, and see
 *                         nuna_set_max_workgroups)
 *   NUNA_WG_THREADS       0 (by size), 64, 128, 256
 *   NUNA_VPT              vectors per thread of the all-reduce, reduce-scatter and
 *                         all-gather: 0 (by size), 1, 2, 4, 8 (8: one-shot all-reduce
 *                         with 2, 4 or 8 ranks only; 4 elsewhere)
 *   NUNA_LPR_MIN_RANKS    many-rank all-reduce kernels from this many ranks, 1..65 (16)
 *   NUNA_LPR_MAX_VECTORS  lane-per-rank all-reduce up to this many input vectors in
 *                         total, 0..2^40 (0: never)
 *   NUNA_COMBINE_VPT      combine vectors per thread: 0 (default), 1, 2, 4
 *   NUNA_COMBINE_CHUNKS   combine column chunks per token, 0 (by size)..INT32_MAX; with
 *                         up to 8 ranks raised where needed so that a chunk is at most
 *                         (workgroup threads x combine vectors per thread) vectors
 *   NUNA_COMBINE_LISTS    0: the combine reads per-token records with up to 8 ranks;
 *                         1: always the offset lists
 *   NUNA_WRITE_THROUGH    stores of the 8-rank one-shot all-reduce and of the 8-rank two-shot's
 *                         all-gather phase: 0 (system-scope write-through where measured
 *                         faster: one-shot with 8 vectors per thread from 16 MiB per rank,
 *                         all-gather phase at 1-2 MiB shards; streaming elsewhere),
 *                         1 (always streaming), 2 (always write-through)
 *   NUNA_TILE_V           rank-major tile all-reduce width: 0 (16 up to 256 KiB per
 *                         rank, else off), 16, 32, 64
 *   NUNA_PAGE_GROUPS      XCD mode, one-work-item-per-workgroup launches with chunks
 *                         smaller than 4 KiB: 0 (default) runs the linear map, 1 keeps
 *                         the chunks of one page on one XCD
 *   NUNA_DIRECT_MAX_GRID  largest grid of the one-work-item-per-workgroup kernels,
 *                         0 (8192)..2^24; larger launches loop (persistent kernels)
 *   NUNA_SHARD_XCD        fused two-shot, every chunk of shard r on XCD r mod 8: 0 (in XCD
 *                         mode with 16 ranks, where it measured faster), 1 (never), 2 (in
 *                         both modes with 8 or 16 ranks)
 *   NUNA_TWO_SHOT_FORM    NUNA_ALGO_TWO_SHOT: 0 (by size: fused, except 8 ranks of bf16
 *                         at 16-40 MiB per rank, which run the two kernels), 1 (fused
 *                         wherever it applies), 2 (always the two kernels)
 *   NUNA_STORE_GAP        pause between the stores of consecutive destinations when one
 *                         result is stored to several outputs (one-shot and fused two-shot
 *                         all-reduce, all-gather), in units of 8 wait states of the wave:
 *                         -1 (by size: 1 from 32 MiB per rank, else 0), 0..32
 * Unknown names and values outside these sets: NUNA_ERR_INVALID_ARG. */
nuna_status_t nuna_set_tunable(const char* name, int64_t value);
nuna_status_t nuna_get_tunable(const char* name, int64_t* value);

/*
 * All-reduce (sum).  Sec. 2.1 (all-reduce of gradients / partial
 * activations); direct algorithm as in Sec. 5.1.
 *   in[r]   P device pointers, each `count` elements of `dtype`, rank order
 *           r = 0..P-1 is the summation order.
 *   out[d]  P device pointers, each `count` elements; every out[d] receives
 *           the same result.
 *   algo    ONE_SHOT, ONE_SHOT_SPLIT, TWO_SHOT, TWO_SHOT_TWO_KERNELS or
 *           AUTO.  The two-shot forms need count % P == 0 (rank r owns the
 *           shard [r*count/P, (r+1)*count/P)); otherwise they run one-shot
 *           (same bits).
 *           ONE_SHOT_SPLIT with in-place buffers runs ONE_SHOT (a split
 *           work item would overwrite an input another group still reads).
 * In-place: out[r] == in[r] is allowed.  Any other overlap between an input
 * and an output, or between two outputs, is NUNA_ERR_OVERLAP.  Inputs may
 * alias each other.  count == 0 returns NUNA_OK with no launch.
 * Alignment: every pointer 16-byte aligned (NUNA_ERR_MISALIGNED).
 */
nuna_status_t nuna_allreduce(const void* const* in, void* const* out, int P, size_t count,
                             nuna_dtype_t dtype, nuna_algo_t algo, nuna_placement_t place,
                             hipStream_t stream);

/*
 * Reduce-scatter (sum).  Sec. 2.1 (tensor-parallel traces).
 *   in[q]   P device pointers, each P*recvcount elements.  Rank r owns the
 *           contiguous shard [r*recvcount, (r+1)*recvcount).
 *   out[r]  P device pointers, each recvcount elements:
 *           out[r][j] = sum over q ascending of in[q][r*recvcount + j].
 * In-place: out[r] == in[r] + r*recvcount (elements) is allowed.  Other
 * overlaps are NUNA_ERR_OVERLAP.  recvcount == 0 is a no-op.
 */
nuna_status_t nuna_reduce_scatter(const void* const* in, void* const* out, int P, size_t recvcount,
                                  nuna_dtype_t dtype, nuna_placement_t place, hipStream_t stream);

/*
 * All-gather (byte copy).  Sec. 2.1; the paper's worked placement example
 * (Sec. 4.2, the two-GPU all-gather figure) is an all-gather done as local
 * load, remote store.
 *   in[r]   P device pointers, each sendcount elements.
 *   out[d]  P device pointers, each P*sendcount elements:
 *           out[d][r*sendcount + j] = in[r][j] for every d.
 * In-place: in[r] == out[r] + r*sendcount (elements) is allowed.  Other
 * overlaps are NUNA_ERR_OVERLAP.  sendcount == 0 is a no-op.
 */
nuna_status_t nuna_all_gather(const void* const* in, void* const* out, int P, size_t sendcount,
                              nuna_dtype_t dtype, nuna_placement_t place, hipStream_t stream);

/*
 * All-to-all dispatch of MoE token rows (Sec. 2.1: all-to-all routes tokens
 * to experts; Sec. 6.7: expert token routing).
 *
 * A layout is the routing plan of one dispatch.  Expert e lives on rank
 * e / (num_experts / P).  Token t of rank s is sent once to every distinct
 * rank that owns one of its top-k experts; rank d receives its rows ordered
 * by source rank, then token (both ascending).
 *
 * nuna_a2a_layout_create: host-only planning, no HIP call.
 *   topk_idx  HOST int32 array [P][tokens_per_rank][topk], read during the
 *             call; every entry in [0, num_experts).
 *   Requires 1 <= P <= 64, tokens_per_rank >= 0, P * tokens_per_rank <=
 *   INT32_MAX, 1 <= topk <= num_experts, num_experts % P == 0.  *out
 *   receives a layout owned by the caller.
 * nuna_a2a_layout_upload: copies the layout's descriptor tables to the
 *   current device (allocates device memory; synchronous; not capturable).
 *   A layout must be uploaded before nuna_all_to_all or
 *   nuna_all_to_all_combine uses it.
 * nuna_a2a_layout_recv_rows: rows_per_rank[d] = rows rank d receives (HOST
 *   int64 array of P).
 * nuna_a2a_layout_recv_map: for destination d, the source rank and token of
 *   each received row in receive order (HOST int32 arrays of
 *   rows_per_rank[d] entries each).
 * nuna_a2a_layout_destroy: frees host and device parts; NULL is a no-op.
 *   The caller must ensure no enqueued all-to-all still uses the layout.
 */
typedef struct nuna_a2a_layout nuna_a2a_layout_t;

nuna_status_t nuna_a2a_layout_create(int P, int tokens_per_rank, int topk, int num_experts,
                                     const int32_t* topk_idx, nuna_a2a_layout_t** out);
nuna_status_t nuna_a2a_layout_upload(nuna_a2a_layout_t* layout);
nuna_status_t nuna_a2a_layout_recv_rows(const nuna_a2a_layout_t* layout, int64_t* rows_per_rank);
nuna_status_t nuna_a2a_layout_recv_map(const nuna_a2a_layout_t* layout, int d, int32_t* src_rank,
                                       int32_t* src_token);
void nuna_a2a_layout_destroy(nuna_a2a_layout_t* layout);

/*
 * All-to-all dispatch: recv[d][j, :] = send[s][t, :] for the j-th row (s, t)
 * of destination d in the layout.
 *   send[s]  P device pointers, each [tokens_per_rank][row_elems] of dtype.
 *   recv[d]  P device pointers, each with room for recv_capacity_rows rows of
 *            row_elems; rows beyond rows_per_rank[d] are left untouched.
 *   Returns NUNA_ERR_INVALID_ARG if the layout is not uploaded or any
 *   rows_per_rank[d] exceeds recv_capacity_rows.  Send and receive buffers
 *   must not overlap (NUNA_ERR_OVERLAP).
 */
nuna_status_t nuna_all_to_all(const void* const* send, void* const* recv, const nuna_a2a_layout_t* layout,
                              size_t row_elems, size_t recv_capacity_rows, nuna_dtype_t dtype,
                              nuna_placement_t place, hipStream_t stream);

/*
 * All-to-all dispatch that allocates nothing, for callers that cannot call
 * hipMalloc: code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation.  Same result as nuna_all_to_all on a layout built from
 * the same top-k table, but the routing is read from DEVICE memory and the
 * receive rows are computed on the device, in the library's static scratch
 * array (8 MiB per GPU, held by each GPU the library runs on until the
 * process ends) instead of layout tables the library allocates.
 *   send[s]        P device pointers, each [tokens_per_rank][row_elems].
 *   recv[d]        P device pointers, each with room for recv_capacity_rows rows;
 *                  rows past the capacity are not written.
 *   topk_idx       DEVICE int32 [P][tokens_per_rank][topk], 4-byte aligned;
 *                  entries outside [0, num_experts) route nowhere.
 *   rows_per_rank  DEVICE int64 [P + 1], 8-byte aligned, written by the call:
 *                  [d] = rows rank d receives (compare with the capacity),
 *                  [P] = top-k entries outside [0, num_experts).
 * The routing tables need 4*P*P + 4*P + 4*P*tokens_per_rank*min(topk, P)
 * bytes of the scratch: larger calls return NUNA_ERR_INVALID_ARG, as do
 * P*tokens_per_rank >= 2^26.  Calls of at most 256 tokens over all ranks
 * (and at most 2048 top-k entries) run as one kernel that recomputes the
 * routing in every workgroup and leaves the scratch alone.  Rows must be
 * whole 16-byte vectors (NUNA_ERR_UNSUPPORTED otherwise).  Needs nuna_init
 * on the current device (it looks up the scratch array's address there;
 * NUNA_ERR_UNSUPPORTED without it).  Every call on a GPU uses that GPU's one array: calls on one
 * stream run in order, calls that overlap on one GPU (other streams, other
 * threads) race and must not be made.  One work item copies a token row to
 * one of its destinations; NUNA_PLACE_XCD runs the copies of a token row on
 * one XCD (a logical group, as nuna_all_to_all does with its layout),
 * NUNA_PLACE_LINEAR in order.  Capture-safe.
 */
nuna_status_t nuna_all_to_all_routed(const void* const* send, void* const* recv, const int32_t* topk_idx, int P,
                                     int tokens_per_rank, int topk, int num_experts, size_t row_elems,
                                     size_t recv_capacity_rows, nuna_dtype_t dtype, nuna_placement_t place,
                                     int64_t* rows_per_rank, hipStream_t stream);

/*
 * All-to-all combine: the result-collection step of MoE expert parallelism
 * (Sec. 2.1: the all-to-all that sends tokens to their experts also brings
 * the expert outputs back).  It reverses a dispatch made with the same
 * layout: row j of y[d] is the result for the j-th row rank d received, and
 *   out[s][t, :] = y[d0][j0, :] + y[d1][j1, :] + ...
 * over the distinct ranks d0 < d1 < ... that token t of rank s was sent to
 * (j_i its receive row there).  Addition runs in that rank order in fp32,
 * starting from the first row, with one rounding to dtype at the end (bf16:
 * round to nearest even; NaN stays NaN).  Every output row is written.
 * Weighted form: with weights not NULL each term is first scaled,
 *   out[s][t, :] = w[s][t][d0] * y[d0][j0, :] + w[s][t][d1] * y[d1][j1, :] + ...
 * each product an fp32 multiply rounded once (no fused multiply-add).  With
 * one expert per rank (num_experts == P) w holds the router's gate weights
 * and this is the top-k weighted sum of a MoE layer; with several experts
 * per rank, ranks usually return their local weighted sums and weights is
 * NULL.
 *   y[d]    P device pointers, each with room for y_capacity_rows rows of
 *           row_elems; rows beyond rows_per_rank[d] are not read.
 *   out[s]  P device pointers, each [tokens_per_rank][row_elems] of dtype.
 *   weights NULL, or a device fp32 array [P][tokens_per_rank][P] (source
 *           rank, token, destination rank), 4-byte aligned; entries for
 *           ranks a token was not sent to are not read.
 *   The placement argument is accepted for symmetry with the dispatch; a
 *   combine work item shares no input with any other, so both modes run the
 *   same map.
 *   Returns NUNA_ERR_INVALID_ARG if the layout is not uploaded or any
 *   rows_per_rank[d] exceeds y_capacity_rows.  Result, weight and output
 *   buffers must not overlap (NUNA_ERR_OVERLAP).  A layout with no tokens is
 *   a no-op.
 */
nuna_status_t nuna_all_to_all_combine(const void* const* y, void* const* out, const nuna_a2a_layout_t* layout,
                                      const float* weights, size_t row_elems, size_t y_capacity_rows,
                                      nuna_dtype_t dtype, nuna_placement_t place, hipStream_t stream);

/*
 * NUNA-aware placement planner: Algorithm 1 of the paper (Sec. 4.2.2,
 * logical allocation then physical placement), host-only, no HIP call.
 *
 * Workload: num_tb threadblocks in the order the plan lists them;
 * threadblock t touches the chunks chunk_ids[chunk_offsets[t] ..
 * chunk_offsets[t+1]) (any 64-bit ids; a chunk touched by several
 * threadblocks appears once per threadblock) and is charged tb_bytes[t]
 * against the CU and stack budgets.  chunk_pages (same length as chunk_ids,
 * or NULL) gives each entry's page id; a chunk must carry the same page in
 * every entry.
 *
 * Logical allocation: a threadblock none of whose chunks belongs to a group
 * starts a new group; otherwise it joins the group it shares the most chunks
 * with (ties: the group created first), and its unassigned chunks join too.
 * Groups are then ordered by decreasing number of threadblocks, creation
 * order among equals.
 * Physical placement: the i-th group of that order goes to NAR domain
 * i mod nar_max, which spans the physical domains [n*D/nar_max,
 * (n+1)*D/nar_max) (D = topo->num_domains; nar_max must divide D).  Each of
 * its threadblocks takes the first CU of the domain whose remaining budget
 * covers tb_bytes (none: the first CU with the most budget left), and the
 * first stack in its physical domain's preference order whose remaining
 * budget covers them (none: the most preferred stack); both budgets are
 * charged.  A chunk lives on the stack of the first threadblock placed that
 * touches it; with pages, a page's stack is fixed by its first chunk.
 *
 * Outputs (HOST arrays, caller-owned): tb_group[num_tb] (group index in
 * creation order), tb_domain[num_tb] (NAR domain), tb_cu[num_tb] (physical
 * domain * cus_per_domain + CU index), entry_stack[chunk_offsets[num_tb]]
 * (stack of each entry's chunk), *num_groups.  Any output pointer may be
 * NULL.  Invalid topology, nar_max, offsets or negative bytes:
 * NUNA_ERR_INVALID_ARG.
 *
 * On MI355X the kernels realise the domain part of the plan (workgroup b runs
 * on XCD b mod 8); the CU within an XCD is the hardware's choice, and stacks
 * cannot be chosen per page in NPS1, so tb_cu and entry_stack describe the
 * plan rather than what the hardware is told.
 */
#define NUNA_NAP_MAX_DOMAINS 16
#define NUNA_NAP_MAX_STACKS 16

typedef struct {
    int32_t num_domains;    /* physical domains (MI355X: 8 XCDs) */
    int32_t cus_per_domain; /* CUs per physical domain (MI355X: 32) */
    int32_t num_stacks;     /* HBM stacks (MI355X: 8) */
    int32_t reserved;
    int64_t cu_budget;      /* R_max of a CU, in the units of tb_bytes */
    int64_t stack_budget;   /* R_max of a stack */
    int32_t stack_pref[NUNA_NAP_MAX_DOMAINS][NUNA_NAP_MAX_STACKS]; /* per physical domain: all stacks,
                                                                      most preferred first */
} nuna_nap_topology_t;

/* MI355X: 8 XCDs x 32 CUs, 8 stacks; XCDs and stacks 0-3 on one I/O die,
 * 4-7 on the other; XCD x prefers stack x, then its die's other stacks, then
 * the far die's (index order); CU budget 700 x 128 B, stack budget 1 MiB. */
nuna_status_t nuna_nap_topology_mi355x(nuna_nap_topology_t* topo);

nuna_status_t nuna_nap_plan(const nuna_nap_topology_t* topo, int nar_max, int64_t num_tb,
                            const int64_t* chunk_offsets, const int64_t* chunk_ids, const int64_t* tb_bytes,
                            const int64_t* chunk_pages, int64_t* tb_group, int32_t* tb_domain, int32_t* tb_cu,
                            int32_t* entry_stack, int64_t* num_groups);

/*
 * Placement map, host mirror of what the kernels compute (for inspection and
 * tests; no HIP call).  A launch over `groups` logical groups of
 * `group_size` work items each (items numbered group-major: item =
 * group * group_size + member) with G workgroups: nuna_placement_items
 * writes to items[0..capacity) the work items workgroup b runs, in the
 * order it runs them, and sets *count to their number
 * (NUNA_ERR_INVALID_ARG if capacity is too small; *count is still set).
 * nuna_placement_grid gives the workgroup count a launch of that placement
 * uses before the nuna_set_max_workgroups cap (XCD mode sizes every XCD for
 * the longest per-XCD group list).
 */
nuna_status_t nuna_placement_items(nuna_placement_t place, int64_t b, int64_t G, int64_t groups,
                                   int64_t group_size, int64_t* items, int64_t capacity, int64_t* count);
nuna_status_t nuna_placement_grid(nuna_placement_t place, int64_t groups, int64_t group_size,
                                  int64_t* workgroups);

/*
 * Host mirror of the map of the one-work-item-per-workgroup launches (the
 * direct kernels; no HIP call): `items` work items of `chunk_bytes` each
 * (a power of two, at least 16), item i covering bytes [i*chunk_bytes,
 * (i+1)*chunk_bytes) of every rank buffer.  LINEAR: workgroup b runs item b.
 * XCD with chunks below 4 KiB and NUNA_PAGE_GROUPS set to 1: the gp = 4096 /
 * chunk_bytes items of one page form a group; group g runs on XCD g mod 8,
 * its members on consecutive workgroups of that XCD (b, b+8, ...); the grid
 * is padded to whole rounds of 8 groups.  *workgroups receives the grid;
 * item_of[b] (HOST int64 array of `capacity`) the item workgroup b runs, or
 * -1 for a padding workgroup (NUNA_ERR_INVALID_ARG if capacity is too
 * small; *workgroups is still set).  The launch-time cap and direct-grid
 * limit, under which a launch falls back to other maps, are not applied.
 */
nuna_status_t nuna_placement_direct(nuna_placement_t place, int64_t items, int64_t chunk_bytes, int64_t* item_of,
                                    int64_t capacity, int64_t* workgroups);

/*
 * Dispatch probe (verifies the workgroup -> XCD assumption behind
 * NUNA_PLACE_XCD).  Launches G workgroups; workgroup b writes the hardware
 * XCC id it ran on to xcc[b] and its raw HW_ID register to hw_id[b]
 * (hw_id may be NULL).  xcc/hw_id: device int32 arrays of G entries.
 */
nuna_status_t nuna_probe_xcc(int G, int32_t* xcc, int32_t* hw_id, hipStream_t stream);

/*
 * Load-latency probe: the one-GPU counterpart of the paper's measurement of
 * how remote-access latency varies with the CU and the target address
 * (Sec. 3.2).  A single lane on XCD `xcd` walks the nbytes / stride blocks
 * of `buf` (device memory) in order; for block i it first loads another
 * 128-byte line of the block (warming the address translation), then times
 * one load of the word at i*stride + line_offset.  cycles[i] (device
 * uint32 array, nbytes / stride entries) receives that latency in shader
 * clock cycles.  The loads should be cold: the caller evicts the caches
 * beforehand (for instance by streaming over more than the 256 MB Infinity
 * Cache).  Runs serially, about half a microsecond per block.  Requires
 * 4-byte aligned buf and cycles, stride and line_offset multiples of 4,
 * line_offset + 4 <= stride.
 */
nuna_status_t nuna_probe_load_latency(const void* buf, size_t nbytes, size_t stride, size_t line_offset, int xcd,
                                      uint32_t* cycles, hipStream_t stream);

/*
 * Per-compute-unit load-latency probe (the paper's latency profiling over
 * every CU and target address, Sec. 3.2, on one GPU).  Launches 512 one-wave
 * workgroups; each of those that run on XCD `xcd` claims the compute unit it
 * runs on if no earlier workgroup did, and the claimed compute units (at most
 * 32, in claim order: slot j) each walk the nbytes / stride blocks of `buf`
 * with one lane, timing one cold load per block.  Slot j loads lines 2j
 * (warm-up of the block's address translation) and 2j + 1 (timed) of each
 * block, so no two compute units of the XCD share a line.
 *   work    device int32 [257], zeroed by the caller before each call (claim
 *           words, then the slot counter; work[256] ends as the number of
 *           compute units found, counting any past 32).
 *   cycles  device uint32 [32][nbytes / stride]: slot j's latency of block i
 *           in shader clock cycles at [j * nblocks + i].
 *   cu_of   device int32 [32]: bits 8-15 of the HW_ID register (CU, array and
 *           shader-engine fields) of the compute unit in slot j; untouched
 *           for unused slots.
 * The loads should be cold: the caller evicts the caches beforehand, and
 * between two XCDs' calls on the same buffer.  stride: a multiple of 128 of
 * at least 8 KiB; buffers 4-byte aligned.  About half a microsecond per block.
 */
nuna_status_t nuna_probe_load_latency_cus(const void* buf, size_t nbytes, size_t stride, int xcd, int32_t* work,
                                          uint32_t* cycles, int32_t* cu_of, hipStream_t stream);

/*
 * Reference streams: the plain access patterns that bound the collectives'
 * HBM rooflines, for calibration and comparison.  Not an operation of the
 * paper and not a collective: measurement support, like nuna_copy.
 * n buffers of `bytes` bytes each, n in {1, 2, 4, 8, 16}, bytes a multiple
 * of 16 up to 2^34 (0: no launch).  Pointers 16-byte aligned; no written
 * range may overlap another or any source (NUNA_ERR_OVERLAP).  One work item
 * is 4 KiB of every buffer (one 16-byte vector per thread and buffer), one
 * item per workgroup, like the collectives' one-vector launches; loads and
 * stores are non-temporal.
 *   NUNA_REF_READ   reads src[0..n); writes only dst[0]: one 16-byte checksum
 *                   per item (the XOR of the item's vectors of all n buffers),
 *                   so that the loads are kept.  A read item is b = 8/n
 *                   consecutive 4 KiB blocks of every buffer (b = 1 for n >= 8),
 *                   so that every thread has 8 or more loads in flight; dst[0]
 *                   receives ceil(bytes / (b * 4096)) * 16 bytes.
 *   NUNA_REF_WRITE  writes dst[0..n) (src unused, may be NULL): 16-byte vector
 *                   v of buffer r holds the 32-bit words {v mod 2^32,
 *                   v div 2^32, r, 0x52454631}.
 *   NUNA_REF_COPY   dst[r] = src[r] for every r, each thread's n loads issued
 *                   before its n stores.
 * Errors: NUNA_ERR_INVALID_ARG (kind, n, bytes, NULL), NUNA_ERR_MISALIGNED,
 * NUNA_ERR_OVERLAP, NUNA_ERR_HIP.
 */
typedef enum { NUNA_REF_READ = 0, NUNA_REF_WRITE = 1, NUNA_REF_COPY = 2 } nuna_ref_t;
nuna_status_t nuna_ref_stream(nuna_ref_t kind, const void* const* src, void* const* dst, int n, size_t bytes,
                              hipStream_t stream);

/*
 * Plain device copy of `bytes` bytes (16-byte aligned pointers, no overlap):
 * the reference streaming kernel used to calibrate memory-traffic counters
 * and the copy-bandwidth ceiling.
 */
nuna_status_t nuna_copy(void* dst, const void* src, size_t bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* NUNA_H */
