// nuna_allreduce.hip -- gfx950 all-reduce kernels: one-shot (with the
// destination-split variant), the two-shot with both phases fused per chunk,
// rank-major tile and lane-per-rank for many ranks, and their launchers.
//
// Memory-bound streaming kernels: every lane moves 16-byte vectors
// (global_load/store_dwordx4), so one wavefront instruction touches 1 KiB of
// contiguous memory.  Reductions widen bf16 to fp32 (exact), add ranks in
// ascending order with one fp32 rounding per add, and round once to the
// buffer dtype with round-to-nearest-even.  No MFMA: there is no contraction,
// and the arithmetic intensity (P-1 adds per 2P element transfers) is far
// below any compute roof.
//
// Workgroup -> work item mapping comes from placement.h (LINEAR / XCD modes).
#include "device_common.h"
#include "shapes.h"

namespace nuna {
namespace {

// ---------------------------------------------------------------- all-reduce (one-shot, optional split)

struct ArShape {
    int64_t nvec;  // full 16-byte vectors per rank buffer
    int32_t dpi;   // destinations per work item (P / group size)
    int32_t P;
    int32_t tail;  // elements after the last full vector
    int32_t gap;   // store_gap between destinations
};

// WT: the item's stores use the system-scope cache policy (store_vecs_wt);
// `cbase` is the chunk's first vector (v0 less the lane).
template <int PT, int DT, int VPT, bool FULL, bool NT, bool WT, int MAXP>
__device__ __forceinline__ void allreduce_chunk(const Ptrs<MAXP>& p, const RankTable& tab, const ArShape& s, int P,
                                                int64_t v0, int nt, int g, bool all_dests, int64_t cbase) {
    using A = Arith<DT>;
    float acc[VPT][A::kLanes];
    reduce_ranks<PT, DT, VPT, FULL, NT>(p, tab, P, 0, v0, nt, s.nvec, acc);
    uint4 y[VPT];
#pragma unroll
    for (int j = 0; j < VPT; ++j) y[j] = A::narrow(acc[j]);
    if (PT > 0 && all_dests) {
#pragma unroll
        for (int d = 0; d < (PT > 0 ? PT : 1); ++d) {
            if (d > 0) store_gap(s.gap);
            if constexpr (WT)
                store_vecs_wt<FULL, VPT>(out_ptr<PT>(p, tab, d) + cbase, y, static_cast<int>(threadIdx.x), nt,
                                         s.nvec - cbase);
            else
                store_vecs<FULL, VPT>(out_ptr<PT>(p, tab, d), y, v0, nt, s.nvec);
        }
    } else {
        const int d0 = g * s.dpi;
        for (int d = d0; d < d0 + s.dpi; ++d) {
            if (d > d0) store_gap(s.gap);
            store_vecs<FULL, VPT>(out_ptr<PT>(p, tab, d), y, v0, nt, s.nvec);
        }
    }
}

template <int PT, int MAXP, int DT, int VPT, bool WT>
__global__ __launch_bounds__(kWG) void k_allreduce(Ptrs<MAXP> p, ArShape s, Place pl) {
    using A = Arith<DT>;
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    const int P = PT > 0 ? PT : s.P;
    __builtin_assume(pl.gsize > 0);  // the collectives always place uniform groups
    const bool all_dests = pl.gsize == 1;
    const RankTable tab = use_table<PT>() ? load_rank_table(p, P) : RankTable{0u, 0u, 0u, 0u};
    if constexpr (PT == 8) {
        // One use of every argument the item loop needs: all their loads issue together.
        asm volatile("" ::"s"(p.in[0]), "s"(p.in[1]), "s"(p.in[2]), "s"(p.in[3]), "s"(p.in[4]), "s"(p.in[5]),
                     "s"(p.in[6]), "s"(p.in[7]), "s"(p.out[0]), "s"(p.out[1]), "s"(p.out[2]), "s"(p.out[3]),
                     "s"(p.out[4]), "s"(p.out[5]), "s"(p.out[6]), "s"(p.out[7]), "s"(s.nvec), "s"(s.dpi),
                     "s"(s.tail), "s"(s.gap), "s"(pl.groups), "s"(pl.mode), "s"(pl.gsize), "s"(pl.gshift),
                     "s"(blockDim.x));
    } else {
        asm volatile("" ::"s"(s.nvec), "s"(s.dpi), "s"(s.tail), "s"(s.gap), "s"(pl.groups), "s"(pl.mode),
                     "s"(pl.gsize), "s"(pl.gshift), "s"(blockDim.x));
    }
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const int64_t w = item_at(pl, blockIdx.x, gridDim.x, i);
        int64_t c;
        int g;
        split_item(w, pl.gsize, pl.gshift, c, g);
        const int64_t v0 = c * cv + threadIdx.x;
        // A chunk read by one work item streams; a chunk shared by a group is
        // read through L2 so the group's re-reads hit.
        if (all_dests) {
            if ((c + 1) * cv <= s.nvec)
                allreduce_chunk<PT, DT, VPT, true, true, WT>(p, tab, s, P, v0, nt, g, all_dests, c * cv);
            else
                allreduce_chunk<PT, DT, VPT, false, true, WT>(p, tab, s, P, v0, nt, g, all_dests, c * cv);
        } else {
            if ((c + 1) * cv <= s.nvec)
                allreduce_chunk<PT, DT, VPT, true, false, false>(p, tab, s, P, v0, nt, g, all_dests, c * cv);
            else
                allreduce_chunk<PT, DT, VPT, false, false, false>(p, tab, s, P, v0, nt, g, all_dests, c * cv);
        }
    }
    if (s.tail > 0 && blockIdx.x == 0 && static_cast<int>(threadIdx.x) < s.tail) {
        const int64_t i = s.nvec * (16 / A::kEsize) + threadIdx.x;
        float a = A::load1(p.in[0], i);
        for (int r = 1; r < P; ++r) a = a + A::load1(p.in[r], i);
        for (int d = 0; d < P; ++d) A::store1(p.out[d], i, a);
    }
}

// Direct one-shot: one work item per workgroup (every uncapped launch whose
// groups have one item, up to the direct-grid limit).  Workgroup b reduces
// chunk page_item(b, gshift): chunk b on the linear map (gshift 0); in XCD
// mode with chunks smaller than a page, the chunks of one 4 KiB page run on
// one XCD (placement.h).  All the kernel reads from its arguments sits at
// fixed offsets (the pointers, the vector count, the tail, the map), so one
// round of scalar loads brings everything and the first vector loads follow
// at once.  The general kernel above first reads its placement state and then
// the pointers, a chain of dependent argument loads that measured about 1 us
// per launch at 1 MiB per rank on MI355X (5.3 against 4.2 us).
template <int PT, int DT, int VPT, bool WT>
__global__ __launch_bounds__(kWG) void k_allreduce_direct(Ptrs<PT> p, int64_t nvec, int32_t tail, int32_t gshift,
                                                          int64_t nitems, int32_t gap) {
    using A = Arith<DT>;
    pin_args(p, nvec, tail, gshift, nitems, gap, blockDim.x);
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    const int64_t c = page_item(blockIdx.x, gshift);
    if (c >= nitems) return;  // padding of a page-grouped grid
    const int64_t v0 = c * cv + threadIdx.x;
    ArShape s{};
    s.nvec = nvec;
    s.dpi = PT;
    s.P = PT;
    s.gap = gap;
    const RankTable tab{0u, 0u, 0u, 0u};  // compile-time rank count: pointers come from the arguments
    if ((c + 1) * cv <= nvec)
        allreduce_chunk<PT, DT, VPT, true, true, WT>(p, tab, s, PT, v0, nt, 0, true, c * cv);
    else
        allreduce_chunk<PT, DT, VPT, false, true, WT>(p, tab, s, PT, v0, nt, 0, true, c * cv);
    if (tail > 0 && blockIdx.x == 0 && static_cast<int>(threadIdx.x) < tail) {
        const int64_t i = nvec * (16 / A::kEsize) + threadIdx.x;
        float a = A::load1(p.in[0], i);
        for (int r = 1; r < PT; ++r) a = a + A::load1(p.in[r], i);
        for (int d = 0; d < PT; ++d) A::store1(p.out[d], i, a);
    }
}

// ---------------------------------------------------------------- two-shot all-reduce, fused phases
//
// The two-shot all-reduce is a reduce-scatter followed by an all-gather
// (Sec. 2.1): rank r reduces its own shard [r*m, (r+1)*m) over the P inputs,
// then copies the reduced shard into the other ranks' outputs.  Here the two
// phases run per chunk inside one kernel.  The workgroup that reduces chunk c
// of shard r stores the result to out[r] (the reduce-scatter result, held in
// the owner's output), then stores the same chunk to out[d] for every d != r
// (the all-gather).  The all-gather's source is the reduce-scatter result the
// workgroup already holds, so no chunk waits on another workgroup, and the
// phase boundary costs neither a second launch nor a grid-wide wait.  Chunks
// never cross a shard.  On one GPU this moves P reads and P writes per
// element, as the one-shot does; the per-rank kernel of a real P-GPU system
// (rank r reducing its shard from P peers, then pushing it to P-1 peers) is
// the work of the workgroups with y = r here.

// Chunk c of shard r (vector offsets relative to the shard; mv vectors per shard).
// SEL: the owner's output pointer is picked among the pinned pointers (direct
// kernel); otherwise it is loaded from the arguments, which keeps the
// persistent kernel's loop from holding every pointer in SGPRs.
template <int PT, int DT, int VPT, bool FULL, bool WT, bool SEL>
__device__ __forceinline__ void two_shot_chunk(const Ptrs<PT>& p, int64_t mv, int r, int64_t c, int nt, int gap) {
    using A = Arith<DT>;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    const int64_t base = static_cast<int64_t>(r) * mv;
    const int64_t v0 = c * cv + threadIdx.x;
    const RankTable tab{0u, 0u, 0u, 0u};  // compile-time rank count: pointers come from the arguments
    float acc[VPT][A::kLanes];
    reduce_ranks<PT, DT, VPT, FULL, true>(p, tab, PT, base, v0, nt, mv, acc);
    uint4 y[VPT];
#pragma unroll
    for (int j = 0; j < VPT; ++j) y[j] = A::narrow(acc[j]);
    // Reduce-scatter phase: the owner's shard.  All-gather phase: every other rank.
    if constexpr (WT) {
        const int lane = static_cast<int>(threadIdx.x);
        store_vecs_wt<FULL, VPT>((SEL ? out_at(p, r) : p.out[r]) + base + c * cv, y, lane, nt, mv - c * cv);
#pragma unroll
        for (int d = 0; d < PT; ++d)
            if (d != r) {
                store_gap(gap);
                store_vecs_wt<FULL, VPT>(p.out[d] + base + c * cv, y, lane, nt, mv - c * cv);
            }
    } else {
        store_vecs<FULL, VPT>((SEL ? out_at(p, r) : p.out[r]) + base, y, v0, nt, mv);
#pragma unroll
        for (int d = 0; d < PT; ++d)
            if (d != r) {
                store_gap(gap);
                store_vecs<FULL, VPT>(p.out[d] + base, y, v0, nt, mv);
            }
    }
}

// Item order.  Chunk-major (the linear map): item w is chunk (w mod wcs) of
// shard (w div wcs), so consecutive workgroups, which the hardware deals to
// consecutive XCDs, take consecutive chunks of one shard.  Shard-interleaved
// (XCD mode with a rank count that is a multiple of 8): item w is chunk
// (w div P) of shard (w mod P), so workgroup b runs shard b mod P and, with
// workgroup b on XCD b mod 8, every chunk of shard r runs on XCD r mod 8: the
// reduce-scatter and all-gather work of simulated rank r stays on one XCD, as
// a rank's own kernel would stay on its own device.

// Direct form, one item per workgroup.  Chunk-major: grid (chunks per shard,
// P), workgroup (c, r).  Shard-interleaved: grid P * wcs, workgroup b.
template <int PT, int DT, int VPT, bool WT, bool ILV>
__global__ __launch_bounds__(kWG) void k_two_shot_direct(Ptrs<PT> p, int64_t mv, int32_t gap) {
    pin_args(p, mv, gap, blockDim.x);
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    int64_t c;
    int r;
    if constexpr (ILV) {
        c = blockIdx.x / PT;
        r = static_cast<int>(blockIdx.x % PT);
    } else {
        c = blockIdx.x;
        r = static_cast<int>(blockIdx.y);
    }
    if ((c + 1) * cv <= mv)
        two_shot_chunk<PT, DT, VPT, true, WT, (PT <= 8)>(p, mv, r, c, nt, gap);
    else
        two_shot_chunk<PT, DT, VPT, false, WT, (PT <= 8)>(p, mv, r, c, nt, gap);
}

// Persistent form for grids beyond the direct limit or under a workgroup cap:
// workgroup b runs items b, b + G, ... of the P * wcs items, in chunk-major
// or (ILV) shard-interleaved order.  With ILV and G a multiple of P, each
// workgroup keeps to shard b mod P.
template <int PT, int DT, int VPT, bool WT, bool ILV>
__global__ __launch_bounds__(kWG) void k_two_shot(Ptrs<PT> p, int64_t mv, int64_t wcs, int32_t gap) {
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    asm volatile("" ::"s"(mv), "s"(wcs), "s"(gap), "s"(blockDim.x));
    const int64_t items = wcs * PT;
    for (int64_t w = blockIdx.x; w < items; w += gridDim.x) {
        int r;
        int64_t c;
        if constexpr (ILV) {
            r = static_cast<int>(w % PT);
            c = w / PT;
        } else {
            r = static_cast<int>(w / wcs);
            c = w - static_cast<int64_t>(r) * wcs;
        }
        if ((c + 1) * cv <= mv)
            two_shot_chunk<PT, DT, VPT, true, WT, false>(p, mv, r, c, nt, gap);
        else
            two_shot_chunk<PT, DT, VPT, false, WT, false>(p, mv, r, c, nt, gap);
    }
}

// ---------------------------------------------------------------- all-reduce, lane per rank (many ranks)
//
// With many ranks a thread that owns one vector position must issue P loads
// and P stores, so small messages run on few workgroups with long
// per-thread instruction streams.  Here thread t of a workgroup owns slot
// (rank t mod P, vector t div P) of a chunk of V = 256 / P vectors: it loads
// one vector of its rank with that rank's own pointer (fetched from the lane
// holding it in the rank table), writes it to an LDS tile [P][V], and after
// the barrier one thread per output dword adds the P ranks in ascending
// order (same order and rounding as every other kernel).  After a second
// barrier thread t stores the result vector to its rank's output.  A message
// of 16 KiB per rank at P=64 thus spreads over 256 workgroups.  Each lane
// reads a different rank, so its accesses are scattered 16-byte requests; the
// rank-major tile kernel below measured faster at every size, and this one
// runs only when the NUNA_LPR_MAX_VECTORS tunable asks for it.

struct LprShape {
    int64_t nvec;  // full 16-byte vectors per rank buffer
    int32_t P;
    int32_t V;     // vectors per rank per work item; P * V <= kWG
    int32_t tail;  // elements after the last full vector
    int32_t pad;
};

// Sum column `col` of the LDS tile over ranks 0..P-1 in order; the dword of
// rank r is col[r * stride].
template <int PT, int DT>
__device__ __forceinline__ uint32_t lpr_sum_column(const uint32_t* col, int stride, int P) {
    constexpr int U = 16;
    float lo, hi;
    if constexpr (DT == kDtF32) {
        lo = __uint_as_float(col[0]);
        hi = 0.0f;
    } else {
        lo = bf16_lo(col[0]);
        hi = bf16_hi(col[0]);
    }
    auto add = [&](uint32_t v) {
        if constexpr (DT == kDtF32) {
            lo = lo + __uint_as_float(v);
        } else {
            lo = lo + bf16_lo(v);
            hi = hi + bf16_hi(v);
        }
    };
    if constexpr (PT > 0) {
        uint32_t t[PT];
#pragma unroll
        for (int r = 1; r < PT; ++r) t[r] = col[r * stride];
#pragma unroll
        for (int r = 1; r < PT; ++r) add(t[r]);
    } else {
        int r = 1;
        for (; r + U <= P; r += U) {
            uint32_t t[U];
#pragma unroll
            for (int q = 0; q < U; ++q) t[q] = col[(r + q) * stride];
#pragma unroll
            for (int q = 0; q < U; ++q) add(t[q]);
        }
        for (; r < P; ++r) add(col[r * stride]);
    }
    if constexpr (DT == kDtF32)
        return __float_as_uint(lo);
    else
        return f32_to_bf16(lo) | (f32_to_bf16(hi) << 16);
}

template <int PT, int DT>
__global__ __launch_bounds__(kWG) void k_allreduce_lpr(Ptrs<64> p, LprShape s, Place pl) {
    using A = Arith<DT>;
    extern __shared__ uint4 lds[];  // [P][V] tile, then [V] results
    const int P = PT > 0 ? PT : s.P;
    const int V = s.V;
    const int t = threadIdx.x;
    const RankTable tab = load_rank_table(p, P);
    // This thread's slot and its rank's pointers, fetched from lane `rank`.
    const int rank = t % P;
    const int vec = t / P;
    const bool active = vec < V;
    const int src_lane = rank * 4;
    const uint64_t in_lo = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(src_lane, static_cast<int>(tab.in_lo)));
    const uint64_t in_hi = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(src_lane, static_cast<int>(tab.in_hi)));
    const uint64_t out_lo = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(src_lane, static_cast<int>(tab.out_lo)));
    const uint64_t out_hi = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(src_lane, static_cast<int>(tab.out_hi)));
    const uint4* my_in = global_in((in_hi << 32) | in_lo);
    uint4* my_out = global_out((out_hi << 32) | out_lo);
    uint4* res = lds + P * V;
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const int64_t c = item_at(pl, blockIdx.x, gridDim.x, i);
        const int64_t base = c * V;
        const int64_t left = s.nvec - base;
        const int lim = left < V ? static_cast<int>(left) : V;
        if (active && vec < lim) lds[rank * V + vec] = load16<true>(my_in + base + vec);
        __syncthreads();
        // 4 * lim output dwords; with fewer than 4 ranks there are more of
        // them than threads.
        for (int dw = t; dw < lim * 4; dw += kWG) {
            const uint32_t* col = reinterpret_cast<const uint32_t*>(lds) + dw;
            reinterpret_cast<uint32_t*>(res)[dw] = lpr_sum_column<PT, DT>(col, V * 4, P);
        }
        __syncthreads();
        if (active && vec < lim) store_stream(my_out + base + vec, res[vec]);
        __syncthreads();
    }
    if (s.tail > 0 && blockIdx.x == 0 && t < s.tail) {
        const int64_t e = s.nvec * (16 / A::kEsize) + t;
        float a = A::load1(p.in[0], e);
        for (int r = 1; r < P; ++r) a = a + A::load1(p.in[r], e);
        for (int d = 0; d < P; ++d) A::store1(p.out[d], e, a);
    }
}

// ---------------------------------------------------------------- all-reduce, rank-major tiles (many ranks)
//
// The lane-per-rank kernel spreads a small message over many workgroups, but
// every lane of a wave reads a different rank, so its loads and stores are
// scattered 16-byte accesses; with more data that costs more than it saves.
// Here a work item is V consecutive vectors of every rank.  The workgroup
// loads the [P][V] tile in passes, lanes walking V consecutive vectors of one
// rank (a wave reads 64 / V ranks per pass, each a contiguous V * 16-byte
// run), and parks it in LDS.  One thread per output dword then adds the P
// ranks in ascending order (same order and rounding as every other kernel);
// the results go back to the tile's first row, and the workgroup stores them
// to every rank the way it loaded.

struct TileShape {
    int64_t nvec;  // full 16-byte vectors per rank buffer
    int32_t P;
    int32_t tail;  // elements after the last full vector
};

// Pointer of rank r from the rank table, r chosen per lane (all lanes active).
__device__ __forceinline__ const uint4* lane_rank_in(const RankTable& tab, int r) {
    const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(r * 4, static_cast<int>(tab.in_lo)));
    const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(r * 4, static_cast<int>(tab.in_hi)));
    return global_in((hi << 32) | lo);
}

__device__ __forceinline__ uint4* lane_rank_out(const RankTable& tab, int r) {
    const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(r * 4, static_cast<int>(tab.out_lo)));
    const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(r * 4, static_cast<int>(tab.out_hi)));
    return global_out((hi << 32) | lo);
}

// One work item of the tile kernel: V vectors of every rank starting at `base`.
template <int PT, int DT, int V>
__device__ __forceinline__ void tile_item(const RankTable& tab, const TileShape& s, int P, int64_t base, uint4* lds) {
    constexpr int RPP = kWG / V;  // ranks per pass
    constexpr int kMaxPass = ((PT > 0 ? PT : 64) + RPP - 1) / RPP;
    const int t = threadIdx.x;
    const int rsub = t / V;
    const int vsub = t % V;
    const int npass = (P + RPP - 1) / RPP;
    const bool in_range = base + vsub < s.nvec;
    // Every pass's load is issued before the first one is waited for.
    uint4 buf[kMaxPass];
#pragma unroll
    for (int k = 0; k < kMaxPass; ++k) {
        const int r = k * RPP + rsub;
        const uint4* src = lane_rank_in(tab, r < P ? r : 0);
        if (k < npass && r < P && in_range) buf[k] = load16<true>(src + base + vsub);
    }
#pragma unroll
    for (int k = 0; k < kMaxPass; ++k) {
        const int r = k * RPP + rsub;
        if (k < npass && r < P && in_range) lds[r * V + vsub] = buf[k];
    }
    __syncthreads();
    uint32_t y = 0;
    if (t < V * 4) y = lpr_sum_column<PT, DT>(reinterpret_cast<const uint32_t*>(lds) + t, V * 4, P);
    __syncthreads();
    if (t < V * 4) reinterpret_cast<uint32_t*>(lds)[t] = y;
    __syncthreads();
    const uint4 out = lds[vsub];
#pragma unroll
    for (int k = 0; k < kMaxPass; ++k) {
        const int r = k * RPP + rsub;
        uint4* dst = lane_rank_out(tab, r < P ? r : 0);
        if (k < npass && r < P && in_range) store_stream(dst + base + vsub, out);
    }
}

// Elements after the last full vector, summed by one workgroup.
template <int DT, int MAXP>
__device__ __forceinline__ void tail_elements(const Ptrs<MAXP>& p, int P, int64_t nvec, int tail) {
    using A = Arith<DT>;
    if (tail > 0 && blockIdx.x == 0 && static_cast<int>(threadIdx.x) < tail) {
        const int64_t e = nvec * (16 / A::kEsize) + threadIdx.x;
        float a = A::load1(p.in[0], e);
        for (int r = 1; r < P; ++r) a = a + A::load1(p.in[r], e);
        for (int d = 0; d < P; ++d) A::store1(p.out[d], e, a);
    }
}

template <int PT, int DT, int V>
__global__ __launch_bounds__(kWG) void k_allreduce_tile(Ptrs<64> p, TileShape s, Place pl) {
    static_assert(kWG % V == 0 && V * 4 <= kWG, "tile width");
    extern __shared__ uint4 lds[];  // [P][V]
    __builtin_assume(pl.gsize > 0);  // the collectives always place uniform groups
    const int P = PT > 0 ? PT : s.P;
    const RankTable tab = load_rank_table(p, P);
    asm volatile("" ::"s"(s.nvec), "s"(s.tail), "s"(pl.groups), "s"(pl.mode), "s"(pl.gsize), "s"(pl.gshift));
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        tile_item<PT, DT, V>(tab, s, P, item_at(pl, blockIdx.x, gridDim.x, i) * V, lds);
        __syncthreads();
    }
    tail_elements<DT>(p, P, s.nvec, s.tail);
}

// Direct tile kernel: one item per workgroup (every uncapped launch up to the
// direct-grid limit; the tile kernel's groups have one item), item b on the
// linear map or the page-grouped XCD map (placement.h), so no placement
// state sits between the argument loads and the data loads.
template <int PT, int DT, int V>
__global__ __launch_bounds__(kWG) void k_allreduce_tile_direct(Ptrs<64> p, TileShape s, int32_t gshift,
                                                               int64_t nitems) {
    static_assert(kWG % V == 0 && V * 4 <= kWG, "tile width");
    extern __shared__ uint4 lds[];  // [P][V]
    const int64_t item = page_item(blockIdx.x, gshift);
    if (item >= nitems) return;  // padding of a page-grouped grid
    const int P = PT > 0 ? PT : s.P;
    const RankTable tab = load_rank_table(p, P);
    tile_item<PT, DT, V>(tab, s, P, item * V, lds);
    tail_elements<DT>(p, P, s.nvec, s.tail);
}

// ---------------------------------------------------------------- launch helpers

template <int PT, int MAXP, int DT, int VPT, bool WT = false>
void launch_ar_t(const void* const* in, void* const* out, int P, const ArShape& s, const Place& pl, int64_t G, int nt,
                 hipStream_t st) {
    Ptrs<MAXP> p = make_ptrs<MAXP>(in, out, P, P);
    hipLaunchKernelGGL((k_allreduce<PT, MAXP, DT, VPT, WT>), dim3(static_cast<unsigned>(G)), dim3(nt), 0, st, p, s,
                       pl);
}

// 8 ranks with or without write-through stores.
template <int DT, int VPT>
void launch_ar_8(const void* const* in, void* const* out, const ArShape& s, const Place& pl, int64_t G, int nt,
                 bool wt, hipStream_t st) {
    if (wt) launch_ar_t<8, 8, DT, VPT, true>(in, out, 8, s, pl, G, nt, st);
    else launch_ar_t<8, 8, DT, VPT, false>(in, out, 8, s, pl, G, nt, st);
}

template <int DT, int VPT>
void launch_ar_p(const void* const* in, void* const* out, int P, const ArShape& s, const Place& pl, int64_t G, int nt,
                 bool wt, hipStream_t st) {
    if constexpr (VPT == 8) {
        // Eight vectors per thread exist for 2, 4 and 8 ranks only (pick_ar_shape).
        switch (P) {
            case 2: launch_ar_t<2, 2, DT, 8>(in, out, P, s, pl, G, nt, st); break;
            case 4: launch_ar_t<4, 4, DT, 8>(in, out, P, s, pl, G, nt, st); break;
            case 8: launch_ar_8<DT, 8>(in, out, s, pl, G, nt, wt, st); break;
            default: break;  // refused by launch_allreduce
        }
        return;
    }
    switch (P) {
        case 2: launch_ar_t<2, 2, DT, VPT>(in, out, P, s, pl, G, nt, st); break;
        case 4: launch_ar_t<4, 4, DT, VPT>(in, out, P, s, pl, G, nt, st); break;
        case 8: launch_ar_8<DT, VPT>(in, out, s, pl, G, nt, wt, st); break;
        case 16: launch_ar_t<16, 16, DT, VPT>(in, out, P, s, pl, G, nt, st); break;
        default:
            if constexpr (VPT == 1) {
                if (P == 32) launch_ar_t<32, 64, DT, 1>(in, out, P, s, pl, G, nt, st);
                else if (P == 64) launch_ar_t<64, 64, DT, 1>(in, out, P, s, pl, G, nt, st);
                else launch_ar_t<0, 64, DT, 1>(in, out, P, s, pl, G, nt, st);
            } else {
                launch_ar_t<0, 64, DT, VPT>(in, out, P, s, pl, G, nt, st);  // other P up to 16 (above: VPT 1)
            }
            break;
    }
}

template <int PT, int DT, int VPT, bool WT = false>
void launch_ar_direct_t(const void* const* in, void* const* out, const ArShape& s, const DirectMap& m, int nt,
                        hipStream_t st) {
    const Ptrs<PT> p = make_ptrs<PT>(in, out, PT, PT);
    hipLaunchKernelGGL((k_allreduce_direct<PT, DT, VPT, WT>), dim3(static_cast<unsigned>(m.grid)), dim3(nt), 0, st, p,
                       s.nvec, s.tail, m.gshift, m.items, s.gap);
}

// Direct kernel for 2, 4, 8 or 16 ranks (8 vectors per thread: 2, 4 or 8 ranks);
// write-through stores with 8 ranks when `wt`.
template <int DT, int VPT>
void launch_ar_direct_p(const void* const* in, void* const* out, int P, const ArShape& s, const DirectMap& m, int nt,
                        bool wt, hipStream_t st) {
    switch (P) {
        case 2: launch_ar_direct_t<2, DT, VPT>(in, out, s, m, nt, st); break;
        case 4: launch_ar_direct_t<4, DT, VPT>(in, out, s, m, nt, st); break;
        case 8:
            if (wt) launch_ar_direct_t<8, DT, VPT, true>(in, out, s, m, nt, st);
            else launch_ar_direct_t<8, DT, VPT, false>(in, out, s, m, nt, st);
            break;
        default:
            if constexpr (VPT != 8) launch_ar_direct_t<16, DT, VPT>(in, out, s, m, nt, st);
            break;
    }
}

// Fused two-shot: the direct kernel or the persistent one, in chunk-major or
// (ilv, 8 and 16 ranks) shard-interleaved order.
template <int PT, int DT, int VPT, bool WT>
void launch_two_shot_t(const void* const* in, void* const* out, int64_t mv, int64_t wcs, int64_t G, bool direct,
                       bool ilv, int nt, hipStream_t st) {
    const Ptrs<PT> p = make_ptrs<PT>(in, out, PT, PT);
    const int32_t gap = store_gap_for(static_cast<size_t>(mv) * 16 * PT);
    if constexpr (PT % 8 == 0) {
        if (ilv) {
            if (direct)
                hipLaunchKernelGGL((k_two_shot_direct<PT, DT, VPT, WT, true>), dim3(static_cast<unsigned>(wcs * PT)),
                                   dim3(nt), 0, st, p, mv, gap);
            else
                hipLaunchKernelGGL((k_two_shot<PT, DT, VPT, WT, true>), dim3(static_cast<unsigned>(G)), dim3(nt), 0, st,
                                   p, mv, wcs, gap);
            return;
        }
    }
    if (direct)
        hipLaunchKernelGGL((k_two_shot_direct<PT, DT, VPT, WT, false>), dim3(static_cast<unsigned>(wcs), PT), dim3(nt),
                           0, st, p, mv, gap);
    else
        hipLaunchKernelGGL((k_two_shot<PT, DT, VPT, WT, false>), dim3(static_cast<unsigned>(G)), dim3(nt), 0, st, p,
                           mv, wcs, gap);
}

template <int DT, int VPT>
void launch_two_shot_p(const void* const* in, void* const* out, int P, int64_t mv, int64_t wcs, int64_t G,
                       bool direct, bool ilv, int nt, bool wt, hipStream_t st) {
    switch (P) {
        case 2: launch_two_shot_t<2, DT, VPT, false>(in, out, mv, wcs, G, direct, ilv, nt, st); break;
        case 4: launch_two_shot_t<4, DT, VPT, false>(in, out, mv, wcs, G, direct, ilv, nt, st); break;
        case 8:
            if (wt) launch_two_shot_t<8, DT, VPT, true>(in, out, mv, wcs, G, direct, ilv, nt, st);
            else launch_two_shot_t<8, DT, VPT, false>(in, out, mv, wcs, G, direct, ilv, nt, st);
            break;
        default:
            if constexpr (VPT != 8) launch_two_shot_t<16, DT, VPT, false>(in, out, mv, wcs, G, direct, ilv, nt, st);
            break;
    }
}

}  // namespace

// ---------------------------------------------------------------- launchers

template <int PT, int DT>
void launch_lpr_t(const void* const* in, void* const* out, int P, const LprShape& s, const Place& pl, int64_t G,
                  hipStream_t st) {
    Ptrs<64> p = make_ptrs<64>(in, out, P, P);
    const size_t lds = static_cast<size_t>(P + 1) * s.V * 16;
    hipLaunchKernelGGL((k_allreduce_lpr<PT, DT>), dim3(static_cast<unsigned>(G)), dim3(kWG), lds, st, p, s, pl);
}

template <int DT>
void launch_lpr_p(const void* const* in, void* const* out, int P, const LprShape& s, const Place& pl, int64_t G,
                  hipStream_t st) {
    switch (P) {
        case 16: launch_lpr_t<16, DT>(in, out, P, s, pl, G, st); break;
        case 32: launch_lpr_t<32, DT>(in, out, P, s, pl, G, st); break;
        case 64: launch_lpr_t<64, DT>(in, out, P, s, pl, G, st); break;
        default: launch_lpr_t<0, DT>(in, out, P, s, pl, G, st); break;
    }
}

// Lane-per-rank all-reduce: a work item is a chunk of V = 256 / P vectors of
// every rank.
hipError_t launch_allreduce_lpr(const void* const* in, void* const* out, int P, size_t count, int dtype, int mode,
                                hipStream_t stream) {
    const size_t es = dtype_size(dtype);
    const size_t bytes = count * es;
    LprShape s{};
    s.nvec = static_cast<int64_t>(bytes / 16);
    s.tail = static_cast<int32_t>((bytes % 16) / es);
    s.P = P;
    s.V = kWG / P;
    const int64_t groups = (s.nvec + s.V - 1) / s.V;
    const Place pl = make_place_uniform(mode, groups > 0 ? groups : 1, 1);
    const int64_t G = cap_grid(place_grid(pl));
    note_launch("k_allreduce_lpr", kMapLinear, 1, G, kWG, 1);
    if (dtype == kDtF32)
        launch_lpr_p<kDtF32>(in, out, P, s, pl, G, stream);
    else
        launch_lpr_p<kDtBf16>(in, out, P, s, pl, G, stream);
    return hipGetLastError();
}

template <int PT, int DT, int V>
void launch_tile_t(const void* const* in, void* const* out, int P, const TileShape& s, const Place& pl, int64_t G,
                   const DirectMap& m, hipStream_t st) {
    Ptrs<64> p = make_ptrs<64>(in, out, P, P);
    const size_t lds = static_cast<size_t>(P) * V * 16;
    if (m.direct)
        hipLaunchKernelGGL((k_allreduce_tile_direct<PT, DT, V>), dim3(static_cast<unsigned>(m.grid)), dim3(kWG), lds,
                           st, p, s, m.gshift, m.items);
    else
        hipLaunchKernelGGL((k_allreduce_tile<PT, DT, V>), dim3(static_cast<unsigned>(G)), dim3(kWG), lds, st, p, s,
                           pl);
}

template <int DT, int V>
void launch_tile_p(const void* const* in, void* const* out, int P, const TileShape& s, const Place& pl, int64_t G,
                   const DirectMap& m, hipStream_t st) {
    switch (P) {
        case 16: launch_tile_t<16, DT, V>(in, out, P, s, pl, G, m, st); break;
        case 32: launch_tile_t<32, DT, V>(in, out, P, s, pl, G, m, st); break;
        case 64: launch_tile_t<64, DT, V>(in, out, P, s, pl, G, m, st); break;
        default: launch_tile_t<0, DT, V>(in, out, P, s, pl, G, m, st); break;
    }
}

// Rank-major tile all-reduce with V vectors per rank per work item (16, 32 or 64).
hipError_t launch_allreduce_tile(const void* const* in, void* const* out, int P, size_t count, int dtype, int V,
                                 int mode, hipStream_t stream) {
    const size_t es = dtype_size(dtype);
    const size_t bytes = count * es;
    TileShape s{};
    s.nvec = static_cast<int64_t>(bytes / 16);
    s.tail = static_cast<int32_t>((bytes % 16) / es);
    s.P = P;
    const int64_t groups = (s.nvec + V - 1) / V;
    const Place pl = make_place_uniform(mode, groups > 0 ? groups : 1, 1);
    const int64_t G = cap_grid(place_grid(pl));
    // One item per workgroup, no placement state: the direct kernel, page-grouped in XCD mode.
    const DirectMap m = direct_map(mode, groups > 0 ? groups : 1, int64_t(V) * 16);
    if (m.direct)
        note_launch("k_allreduce_tile_direct", m.gshift > 0 ? kMapXcdPages : kMapLinear, int64_t(1) << m.gshift, m.grid,
                    kWG, V);
    else
        note_launch("k_allreduce_tile", kMapLinear, 1, G, kWG, V);
    if (dtype == kDtF32) {
        if (V == 16) launch_tile_p<kDtF32, 16>(in, out, P, s, pl, G, m, stream);
        else if (V == 32) launch_tile_p<kDtF32, 32>(in, out, P, s, pl, G, m, stream);
        else launch_tile_p<kDtF32, 64>(in, out, P, s, pl, G, m, stream);
    } else {
        if (V == 16) launch_tile_p<kDtBf16, 16>(in, out, P, s, pl, G, m, stream);
        else if (V == 32) launch_tile_p<kDtBf16, 32>(in, out, P, s, pl, G, m, stream);
        else launch_tile_p<kDtBf16, 64>(in, out, P, s, pl, G, m, stream);
    }
    return hipGetLastError();
}

hipError_t launch_allreduce(const void* const* in, void* const* out, int P, size_t count, int dtype,
                            int dest_groups, int mode, hipStream_t stream) {
    const size_t es = dtype_size(dtype);
    const size_t bytes = count * es;
    // Many ranks.  Up to 256 KiB per rank the rank-major tile kernel (16
    // vectors per rank per work item) measured fastest on MI355X, 20-47 %
    // below the one-shot kernel at 64 ranks and below the lane-per-rank kernel
    // at every size; beyond that the one-shot kernel's long per-thread streams
    // win.  The lane-per-rank kernel runs only when its tunable asks for it.
    if (dest_groups <= 1 && P >= tuning().lpr_min_ranks) {
        if (static_cast<int64_t>(bytes / 16) * P <= tuning().lpr_max_vectors)
            return launch_allreduce_lpr(in, out, P, count, dtype, mode, stream);
        int tv = tuning().tile_v;
        if (tv == 0 && bytes <= (size_t(256) << 10)) tv = 16;
        if (tv == 16 || tv == 32 || tv == 64) return launch_allreduce_tile(in, out, P, count, dtype, tv, mode, stream);
    }
    ArShape s{};
    s.nvec = static_cast<int64_t>(bytes / 16);
    s.tail = static_cast<int32_t>((bytes % 16) / es);
    s.P = P;
    s.gap = store_gap_for(bytes);
    const int gsize = dest_groups > 1 ? dest_groups : 1;
    s.dpi = P / gsize;
    int nt, vpt;
    pick_ar_shape(s.nvec, P, nt, vpt);
    if (vpt == 8 && P != 2 && P != 4 && P != 8) return hipErrorInvalidValue;
    const int64_t cv = static_cast<int64_t>(nt) * vpt;
    const int64_t groups = (s.nvec + cv - 1) / cv;
    // A split group reads the chunk of all P ranks gsize times and writes it to
    // P destinations: (gsize - 1) * P of its gsize * P + P transfers are re-reads.
    // The grouped map from launches of more than 2 MiB: up to 2 MiB it gained
    // at most 1.6 % cold on MI355X and lost up to 4.7 % with warm inputs (8
    // ranks at 64 KiB per rank; 64 ranks at 16 KiB), while from 4 MiB it was
    // 5-53 % faster cold and within 2.5 % warm.
    const int gmode = gsize > 1 ? group_mode(mode, int64_t(gsize - 1) * P, int64_t(gsize) * P + P,
                                             static_cast<int64_t>(2 * P) * static_cast<int64_t>(bytes),
                                             int64_t(2) << 20)
                                : mode;
    const Place pl = make_place_uniform(gmode, groups > 0 ? groups : 1, gsize);
    const int64_t G = cap_grid(place_grid(pl));
    // Write-through stores (store_vecs_wt): 8 ranks, 8 vectors per thread,
    // from 16 MiB per rank.  Against streaming stores on MI355X, back-to-back
    // calls: 1.3 % faster cold and 8 % warm at 16 MiB per rank, 3.4 % and
    // 13 % at 32 MiB; 1-14 % slower cold below 16 MiB (though 6-24 % faster
    // warm) and 16 % slower at 64 MiB (the one-vector general kernel).
    const int wtf = tuning().write_through;
    const bool wt = P == 8 && gsize == 1 &&
                    (wtf == 2 || (wtf == 0 && vpt == 8 && bytes >= (size_t(16) << 20)));
    // One item per workgroup: the direct kernel (page-grouped in XCD mode).
    const DirectMap m = direct_map(mode, groups > 0 ? groups : 1, cv * 16);
    if (gsize == 1 && m.direct && direct_ranks(P, vpt)) {
        note_launch("k_allreduce_direct", m.gshift > 0 ? kMapXcdPages : kMapLinear, int64_t(1) << m.gshift, m.grid, nt,
                    vpt);
        if (dtype == kDtF32) {
            if (vpt == 8) launch_ar_direct_p<kDtF32, 8>(in, out, P, s, m, nt, wt, stream);
            else if (vpt == 4) launch_ar_direct_p<kDtF32, 4>(in, out, P, s, m, nt, wt, stream);
            else if (vpt == 2) launch_ar_direct_p<kDtF32, 2>(in, out, P, s, m, nt, wt, stream);
            else launch_ar_direct_p<kDtF32, 1>(in, out, P, s, m, nt, wt, stream);
        } else {
            if (vpt == 8) launch_ar_direct_p<kDtBf16, 8>(in, out, P, s, m, nt, wt, stream);
            else if (vpt == 4) launch_ar_direct_p<kDtBf16, 4>(in, out, P, s, m, nt, wt, stream);
            else if (vpt == 2) launch_ar_direct_p<kDtBf16, 2>(in, out, P, s, m, nt, wt, stream);
            else launch_ar_direct_p<kDtBf16, 1>(in, out, P, s, m, nt, wt, stream);
        }
        return hipGetLastError();
    }
    // The kernel's vectors per thread must be the VPT the chunks were sized with.
    note_launch("k_allreduce", pl.mode == kPlaceXcd && !linear_map(pl, G) ? kMapXcdGroups : kMapLinear, pl.gsize, G,
                nt, vpt);
    if (dtype == kDtF32) {
        if (vpt == 8) launch_ar_p<kDtF32, 8>(in, out, P, s, pl, G, nt, wt, stream);
        else if (vpt == 4) launch_ar_p<kDtF32, 4>(in, out, P, s, pl, G, nt, wt, stream);
        else if (vpt == 2) launch_ar_p<kDtF32, 2>(in, out, P, s, pl, G, nt, wt, stream);
        else launch_ar_p<kDtF32, 1>(in, out, P, s, pl, G, nt, wt, stream);
    } else {
        if (vpt == 8) launch_ar_p<kDtBf16, 8>(in, out, P, s, pl, G, nt, wt, stream);
        else if (vpt == 4) launch_ar_p<kDtBf16, 4>(in, out, P, s, pl, G, nt, wt, stream);
        else if (vpt == 2) launch_ar_p<kDtBf16, 2>(in, out, P, s, pl, G, nt, wt, stream);
        else launch_ar_p<kDtBf16, 1>(in, out, P, s, pl, G, nt, wt, stream);
    }
    return hipGetLastError();
}

bool two_shot_fused_ok(int P, size_t count, int dtype) {
    if (P != 2 && P != 4 && P != 8 && P != 16) return false;
    if (count % static_cast<size_t>(P) != 0) return false;
    return ((count / P) * dtype_size(dtype)) % 16 == 0;  // shards of whole 16-byte vectors
}

// Which form of the two-shot runs (NUNA_TWO_SHOT_FORM: 0 by size, 1 fused
// wherever it applies, 2 two kernels).  By size: the fused kernel, except
// with 8 ranks of bf16 at 16-40 MiB per rank, where the two kernels measured
// 1-7 % faster on MI355X (cold, back to back: 46.8 against 48.4 us at 16 MiB,
// 58.1 against 62.4 at 20 MiB, 113.8 against 118.7 at 40 MiB), while the
// fused kernel was faster at 4-10 MiB (11.8 against 14.3 us at 4 MiB) and at
// 48-64 MiB (179.8 against 189.2 us at 64 MiB).
bool two_shot_runs_fused(int P, size_t count, int dtype) {
    if (!two_shot_fused_ok(P, count, dtype)) return false;
    const int form = tuning().two_shot_form;
    if (form == 1) return true;
    if (form == 2) return false;
    const size_t bytes = count * dtype_size(dtype);
    return !(P == 8 && dtype == kDtBf16 && bytes >= (size_t(16) << 20) && bytes <= (size_t(40) << 20));
}

// Fused two-shot all-reduce (k_two_shot_direct / k_two_shot): launch shape by
// the bytes per rank, as for the one-shot (the two move the same bytes);
// chunks are cut per shard.
hipError_t launch_two_shot_fused(const void* const* in, void* const* out, int P, size_t count, int dtype, int mode,
                                 hipStream_t stream) {
    if (!two_shot_fused_ok(P, count, dtype)) return hipErrorInvalidValue;
    const size_t es = dtype_size(dtype);
    const size_t bytes = count * es;
    const int64_t nvec = static_cast<int64_t>(bytes / 16);
    const int64_t mv = nvec / P;
    int nt, vpt;
    pick_ar_shape(nvec, P, nt, vpt);
    if (vpt == 8 && P == 16) vpt = 4;
    const int64_t cv = static_cast<int64_t>(nt) * vpt;
    const int64_t wcs = (mv + cv - 1) / cv;
    const int64_t items = wcs * P;
    const int64_t G = cap_grid(items);
    const bool direct = G == items && items <= direct_max_grid();
    const int wtf = tuning().write_through;
    const bool wt = P == 8 && (wtf == 2 || (wtf == 0 && vpt == 8 && bytes >= (size_t(16) << 20)));
    // Shard-interleaved order (each shard's work on one XCD): in XCD mode with
    // 16 ranks, where it measured faster on MI355X than the chunk-major order
    // (cold: 3.45 against 3.71 us at 64 KiB per rank, 11.71 against 11.89 at
    // 1 MiB, 51.3 against 52.0 at 4 MiB).  With 8 ranks it measured slower
    // (4.29 against 4.02 us at 1 MiB per rank, 11.87 against 11.78 at 4 MiB,
    // 184.1 against 178.6 at 64 MiB), so XCD mode keeps the chunk-major order
    // there.  NUNA_SHARD_XCD: 0 by this rule, 1 never, 2 always (8 or 16 ranks).
    const int sx = tuning().shard_xcd;
    const bool ilv = P % 8 == 0 && (sx == 2 || (sx == 0 && mode == kPlaceXcd && P == 16));
    note_launch(direct ? "k_two_shot_direct" : "k_two_shot", ilv ? kMapXcdShards : kMapLinear, ilv ? wcs : 1,
                direct ? items : G, nt, vpt);
    if (dtype == kDtF32) {
        if (vpt == 8) launch_two_shot_p<kDtF32, 8>(in, out, P, mv, wcs, G, direct, ilv, nt, wt, stream);
        else if (vpt == 4) launch_two_shot_p<kDtF32, 4>(in, out, P, mv, wcs, G, direct, ilv, nt, wt, stream);
        else if (vpt == 2) launch_two_shot_p<kDtF32, 2>(in, out, P, mv, wcs, G, direct, ilv, nt, wt, stream);
        else launch_two_shot_p<kDtF32, 1>(in, out, P, mv, wcs, G, direct, ilv, nt, wt, stream);
    } else {
        if (vpt == 8) launch_two_shot_p<kDtBf16, 8>(in, out, P, mv, wcs, G, direct, ilv, nt, wt, stream);
        else if (vpt == 4) launch_two_shot_p<kDtBf16, 4>(in, out, P, mv, wcs, G, direct, ilv, nt, wt, stream);
        else if (vpt == 2) launch_two_shot_p<kDtBf16, 2>(in, out, P, mv, wcs, G, direct, ilv, nt, wt, stream);
        else launch_two_shot_p<kDtBf16, 1>(in, out, P, mv, wcs, G, direct, ilv, nt, wt, stream);
    }
    return hipGetLastError();
}

}  // namespace nuna
