// kernels.h -- launchers of the gfx950 kernels (internal to libnuna).
//
// Every launcher assumes the host API has validated its arguments: pointers
// non-null and 16-byte aligned, 1 <= P <= 64, sizes within range.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace nuna {

constexpr int kDtF32 = 0;
constexpr int kDtBf16 = 1;

inline size_t dtype_size(int dt) { return dt == kDtF32 ? 4u : 2u; }

// Tunables (read once from the environment by the host API; they change the
// launch shape only, never the arithmetic).
struct Tuning {
    int max_grid = 0;      // cap on workgroups per launch (persistent loop beyond); 0: 16384
    int wg_threads = 0;    // workgroup size for the streaming kernels (0 = by size)
    int vpt = 0;           // vectors per thread per work item (0 = by size; 8: one-shot all-reduce only)
    int lpr_min_ranks = 16;           // many-rank all-reduce kernels (tile, lane per rank) from this many ranks
    int64_t lpr_max_vectors = 0;       // lane-per-rank all-reduce up to this many input vectors in total (0: off)
    int combine_vpt = 0;               // combine vectors per thread per pass (0 = default)
    int combine_chunks = 0;            // combine column chunks per token (0 = by size)
    int tile_v = 0;                    // rank-major tile all-reduce width (16/32/64; 0 = by size)
    int combine_lists = 0;             // 1: combine reads the offset lists even where records exist
    int write_through = 0;             // 8-rank one-shot stores: 0 by size, 1 streaming, 2 write-through
    int page_groups = 0;               // XCD mode: 1 puts the chunks of a 4 KiB page on one XCD (direct kernels)
    int direct_max_grid = 0;           // largest grid of the direct kernels (0: 8192)
    int two_shot_form = 0;             // two-shot: 0 by size, 1 fused where it applies, 2 two kernels
    int shard_xcd = 0;                 // fused two-shot shard-per-XCD order: 0 in XCD mode, 1 never, 2 always
    int store_gap = -1;                // s_nop 7 pauses between a fan-out's per-destination stores: -1 by size
};
const Tuning& tuning();
// Current workgroup cap (nuna_set_max_workgroups, else the tuning default).
int max_workgroups();
// Largest grid for a kernel that runs one work item per workgroup and is
// better off without a persistent loop: the caller's cap when one is set
// (nuna_set_max_workgroups or NUNA_MAX_GRID), otherwise `dflt`.
int64_t grid_limit(int64_t dflt);

// Record of the kernel launches of the calling thread's current collective
// call (read back through nuna_last_launch): the API starts a record before
// its launches, every launcher appends to it.  map: the workgroup -> work
// item map the launch ran (placement.h); group_size: work items per logical
// group of that map.
enum MapKind { kMapLinear = 0, kMapXcdGroups = 1, kMapXcdPages = 2, kMapXcdLists = 3, kMapXcdShards = 4 };
void note_launch(const char* kernel, int map, int64_t group_size, int64_t grid, int threads, int vpt);

// One-shot all-reduce.  `dest_groups` > 1 selects the split variant: a work
// item is (chunk, destination group) and writes P/dest_groups outputs.
hipError_t launch_allreduce(const void* const* in, void* const* out, int P, size_t count, int dtype,
                            int dest_groups, int mode, hipStream_t stream);

// Fused two-shot all-reduce (reduce-scatter and all-gather phases per chunk in
// one kernel).  Needs P in {2, 4, 8, 16} and shards of whole 16-byte vectors
// (two_shot_fused_ok); otherwise the caller runs the two kernels.
bool two_shot_fused_ok(int P, size_t count, int dtype);
// The fused form applies and is the one to run (size rule, NUNA_TWO_SHOT_FORM).
bool two_shot_runs_fused(int P, size_t count, int dtype);
hipError_t launch_two_shot_fused(const void* const* in, void* const* out, int P, size_t count, int dtype, int mode,
                                 hipStream_t stream);

// Reduce-scatter: in[q] holds P*m elements; out[r][j] = sum_q in[q][r*m+j].
// keep_output: store the shards through the caches (they are read right
// after, by the all-gather phase of a two-shot all-reduce).
hipError_t launch_reduce_scatter(const void* const* in, void* const* out, int P, size_t m, int dtype,
                                 int mode, bool keep_output, hipStream_t stream);

// All-gather: out[d][r*m + j] = in[r][j]; a destination whose shard region
// is the source itself (in-place form) is skipped.  src_cached: read the
// sources through the caches (they were just written).
hipError_t launch_all_gather(const void* const* in, void* const* out, int P, size_t m, int dtype,
                             int mode, bool src_cached, hipStream_t stream);

// All-to-all row copy driven by a descriptor table (device int4 per item:
// src rank, src token, dst rank, dst row) stored in placement order.  For the
// XCD mode, xcd_start holds the 9 offsets of the per-XCD item lists.
hipError_t launch_all_to_all(const void* const* send, void* const* recv, int P, const void* desc,
                             int64_t nitems, const int64_t* xcd_start, size_t row_bytes, int esize,
                             int mode, hipStream_t stream);

// MoE combine: out[s][t] = sum over the token's entries (rank d, row j), in
// list order, of y[d][j], each scaled by weights[(s*T + t)*P + d] when
// weights is not null.  off: device int64[P*T + 1]; ent: device int32 pairs
// (rank, row).  rec: null, or (P <= kCombRecRanks) the same entries as
// kCombRecRanks words per token, (row << 3) | rank, padded with all ones.
constexpr int kCombRecRanks = 8;
hipError_t launch_combine(const void* const* y, void* const* out, int P, int T, const void* off, const void* ent,
                          const void* rec, const float* weights, size_t row_bytes, int dtype, int mode,
                          hipStream_t stream);

// Routed all-to-all dispatch (routing on the device, tables in the library's
// static scratch array, nothing allocated per call).  The scratch holds
// cnt int32[P][P], bad int32[P] and R = min(k, P) uint32 record words per token.
constexpr size_t kRoutedScratchBytes = size_t(8) << 20;
inline size_t routed_scratch_need(int P, int T, int k) {
    const size_t R = static_cast<size_t>(k < P ? k : P);
    return 4 * static_cast<size_t>(P) * P + 4 * static_cast<size_t>(P) + 4 * static_cast<size_t>(P) * T * R;
}
// Device address of the scratch array on the current device (hipGetSymbolAddress).
hipError_t routed_scratch_address(void** ptr);
hipError_t launch_routed_dispatch(const void* const* send, void* const* recv, const int32_t* topk, int P, int T,
                                  int k, int E, int64_t rowvec, int64_t cap, void* scratch_ptr, int64_t* rows_out,
                                  int mode, hipStream_t stream);

hipError_t launch_probe_xcc(int G, int32_t* xcc, int32_t* hw_id, hipStream_t stream);

hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t stream);
// Reference streams (nuna_ref_stream): kind 0 read, 1 write, 2 copy; n in {1, 2, 4, 8, 16};
// bytes a multiple of 16.  Read: dst[0] receives one 16-byte checksum per item of
// max(1, 8 / n) 4 KiB blocks.
hipError_t launch_ref_stream(int kind, const void* const* src, void* const* dst, int n, size_t bytes,
                             hipStream_t stream);

// Per-compute-unit load-latency probe on XCD `xcd` (lines 2j and 2j + 1 of each
// block for probe slot j; claimed: 257 zeroed int32 words).
constexpr int kProbeCuSlotsMax = 32;
hipError_t launch_probe_latency_cus(const void* buf, int64_t nblocks, int64_t stride, int xcd, int32_t* claimed,
                                    uint32_t* cycles, int32_t* cu_of, hipStream_t stream);

// Serial load-latency probe from XCD `xcd` (warm_off < 0: no translation warm-up).
hipError_t launch_probe_latency(const void* buf, int64_t nblocks, int64_t stride, int64_t line_off, int64_t warm_off,
                                int xcd, uint32_t* cycles, hipStream_t stream);

}  // namespace nuna
