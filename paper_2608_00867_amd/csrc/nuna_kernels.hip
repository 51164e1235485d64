// nuna_kernels.hip -- gfx950 kernels of the collective copy/reduce path:
// all-reduce (one-shot, split, rank-major tile, lane-per-rank),
// reduce-scatter, all-gather, the dispatch probe and the reference copy.
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

namespace nuna {
namespace {

// ---------------------------------------------------------------- all-reduce (one-shot, optional split)

struct ArShape {
    int64_t nvec;  // full 16-byte vectors per rank buffer
    int32_t dpi;   // destinations per work item (P / group size)
    int32_t P;
    int32_t tail;  // elements after the last full vector
    int32_t pad;
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
            if constexpr (WT)
                store_vecs_wt<FULL, VPT>(out_ptr<PT>(p, tab, d) + cbase, y, static_cast<int>(threadIdx.x), nt,
                                         s.nvec - cbase);
            else
                store_vecs<FULL, VPT>(out_ptr<PT>(p, tab, d), y, v0, nt, s.nvec);
        }
    } else {
        const int d0 = g * s.dpi;
        for (int d = d0; d < d0 + s.dpi; ++d) store_vecs<FULL, VPT>(out_ptr<PT>(p, tab, d), y, v0, nt, s.nvec);
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
                     "s"(s.tail), "s"(pl.groups), "s"(pl.mode), "s"(pl.gsize), "s"(pl.gshift), "s"(blockDim.x));
    } else {
        asm volatile("" ::"s"(s.nvec), "s"(s.dpi), "s"(s.tail), "s"(pl.groups), "s"(pl.mode), "s"(pl.gsize),
                     "s"(pl.gshift), "s"(blockDim.x));
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

// Direct one-shot: one work item per workgroup on the linear map, which is
// every uncapped launch whose groups have one item (up to kDirectMaxGrid
// workgroups).  Workgroup b reduces chunk b.  All the kernel reads from its
// arguments sits at fixed offsets (the pointers, the vector count, the tail),
// so one round of scalar loads brings everything and the first vector loads
// follow at once.  The general kernel above first reads its placement state
// and then the pointers, a chain of dependent argument loads that measured
// about 1 us per launch at 1 MiB per rank on MI355X (5.3 against 4.2 us).
template <int PT, int DT, int VPT, bool WT>
__global__ __launch_bounds__(kWG) void k_allreduce_direct(Ptrs<PT> p, int64_t nvec, int32_t tail) {
    using A = Arith<DT>;
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    const int64_t c = blockIdx.x;
    const int64_t v0 = c * cv + threadIdx.x;
    ArShape s{};
    s.nvec = nvec;
    s.dpi = PT;
    s.P = PT;
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

// Direct tile kernel: workgroup b takes item b (every uncapped launch of up
// to kDirectMaxGrid workgroups; the tile kernel's groups have one item), so
// no placement state sits between the argument loads and the data loads.
template <int PT, int DT, int V>
__global__ __launch_bounds__(kWG) void k_allreduce_tile_direct(Ptrs<64> p, TileShape s) {
    static_assert(kWG % V == 0 && V * 4 <= kWG, "tile width");
    extern __shared__ uint4 lds[];  // [P][V]
    const int P = PT > 0 ? PT : s.P;
    const RankTable tab = load_rank_table(p, P);
    tile_item<PT, DT, V>(tab, s, P, static_cast<int64_t>(blockIdx.x) * V, lds);
    tail_elements<DT>(p, P, s.nvec, s.tail);
}

// ---------------------------------------------------------------- reduce-scatter

struct RsShape {
    int64_t mv;   // vectors per shard
    int64_t wcs;  // chunks per shard
    int32_t P;
    int32_t pad;
};

template <int PT, int DT, int VPT, bool FULL, bool KEEP, int MAXP>
__device__ __forceinline__ void reduce_scatter_chunk(const Ptrs<MAXP>& p, const RankTable& tab, const RsShape& s,
                                                     int P, int64_t r, int64_t v0, int nt) {
    using A = Arith<DT>;
    float acc[VPT][A::kLanes];
    reduce_ranks<PT, DT, VPT, FULL, true>(p, tab, P, r * s.mv, v0, nt, s.mv, acc);
    uint4 y[VPT];
#pragma unroll
    for (int j = 0; j < VPT; ++j) y[j] = A::narrow(acc[j]);
    store_vecs<FULL, VPT, !KEEP>(use_table<PT>() ? rank_out(tab, static_cast<int>(r)) : p.out[r], y, v0, nt, s.mv);
}

// KEEP: the shard is read again right away (the all-gather phase of a two-shot
// all-reduce), so it is stored through the caches instead of streamed.
template <int PT, int MAXP, int DT, int VPT, bool KEEP>
__global__ __launch_bounds__(kWG) void k_reduce_scatter(Ptrs<MAXP> p, RsShape s, Place pl) {
    __builtin_assume(pl.gsize > 0);  // the collectives always place uniform groups
    const int P = PT > 0 ? PT : s.P;
    const RankTable tab = use_table<PT>() ? load_rank_table(p, P) : RankTable{0u, 0u, 0u, 0u};
    // One use of every argument the item loop needs: their loads issue together.
    if constexpr (PT == 8)
        asm volatile("" ::"s"(p.in[0]), "s"(p.in[1]), "s"(p.in[2]), "s"(p.in[3]), "s"(p.in[4]), "s"(p.in[5]),
                     "s"(p.in[6]), "s"(p.in[7]), "s"(p.out[0]), "s"(p.out[1]), "s"(p.out[2]), "s"(p.out[3]),
                     "s"(p.out[4]), "s"(p.out[5]), "s"(p.out[6]), "s"(p.out[7]), "s"(s.mv), "s"(s.wcs),
                     "s"(pl.groups), "s"(pl.mode), "s"(pl.gsize), "s"(pl.gshift), "s"(blockDim.x));
    else
        asm volatile("" ::"s"(s.mv), "s"(s.wcs), "s"(pl.groups), "s"(pl.mode), "s"(pl.gsize), "s"(pl.gshift),
                     "s"(blockDim.x));
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const int64_t w = item_at(pl, blockIdx.x, gridDim.x, i);
        const int64_t r = w / s.wcs;
        const int64_t c = w - r * s.wcs;
        const int64_t v0 = c * cv + threadIdx.x;
        if ((c + 1) * cv <= s.mv)
            reduce_scatter_chunk<PT, DT, VPT, true, KEEP>(p, tab, s, P, r, v0, nt);
        else
            reduce_scatter_chunk<PT, DT, VPT, false, KEEP>(p, tab, s, P, r, v0, nt);
    }
}

// Direct reduce-scatter: grid (chunks per shard, P), workgroup (c, r) reduces
// chunk c of shard r; everything it reads from its arguments sits at fixed
// offsets (see k_allreduce_direct).
template <int PT, int DT, int VPT, bool KEEP>
__global__ __launch_bounds__(kWG) void k_reduce_scatter_direct(Ptrs<PT> p, int64_t mv) {
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    const int64_t c = blockIdx.x;
    const int64_t r = blockIdx.y;
    const int64_t v0 = c * cv + threadIdx.x;
    RsShape s{};
    s.mv = mv;
    s.P = PT;
    const RankTable tab{0u, 0u, 0u, 0u};  // compile-time rank count: pointers come from the arguments
    if ((c + 1) * cv <= mv)
        reduce_scatter_chunk<PT, DT, VPT, true, KEEP>(p, tab, s, PT, r, v0, nt);
    else
        reduce_scatter_chunk<PT, DT, VPT, false, KEEP>(p, tab, s, PT, r, v0, nt);
}

// Element-wise fallback when a shard is not a whole number of 16-byte vectors.
template <int DT>
__global__ __launch_bounds__(kWG) void k_reduce_scatter_elem(Ptrs<64> p, int P, int64_t m) {
    using A = Arith<DT>;
    const int64_t total = m * P;
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < total;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t r = i / m;
        float a = A::load1(p.in[0], i);
        for (int q = 1; q < P; ++q) a = a + A::load1(p.in[q], i);
        A::store1(p.out[r], i - r * m, a);
    }
}

// ---------------------------------------------------------------- all-gather

struct AgShape {
    int64_t mv;   // vectors per shard
    int64_t wcs;  // chunks per shard
    int32_t P;
    int32_t dpi;  // destinations per item
};

// WT: write-through stores (store_vecs_wt); `cbase` is the chunk's first
// vector within the shard (v0 less the lane).
template <int VPT, bool FULL, bool NT, bool WT>
__device__ __forceinline__ void all_gather_chunk(const RankTable& tab, const AgShape& s, int64_t r, int64_t v0, int nt,
                                                 int g, int64_t cbase) {
    const uint4* src = rank_in(tab, static_cast<int>(r));
    uint4 y[VPT];
    load_vecs<FULL, VPT, NT>(y, src, v0, nt, s.mv);
    const int d0 = g * s.dpi;
    for (int d = d0; d < d0 + s.dpi; ++d) {
        uint4* dst = rank_out(tab, d) + r * s.mv;
        if (dst == src) continue;  // in-place shard
        if constexpr (WT)
            store_vecs_wt<FULL, VPT>(dst + cbase, y, static_cast<int>(threadIdx.x), nt, s.mv - cbase);
        else
            store_vecs<FULL, VPT>(dst, y, v0, nt, s.mv);
    }
}

// CACHED: the sources were just written (two-shot all-gather phase) and may
// still sit in L2 or the Infinity Cache, so they are read through the caches.
// WT: write-through stores.
template <int MAXP, int VPT, bool CACHED, bool WT>
__global__ __launch_bounds__(kWG) void k_all_gather(Ptrs<MAXP> p, AgShape s, Place pl) {
    __builtin_assume(pl.gsize > 0);  // the collectives always place uniform groups
    const RankTable tab = load_rank_table(p, s.P);
    // One use of every scalar argument the item loop needs: their loads issue together.
    asm volatile("" ::"s"(s.mv), "s"(s.wcs), "s"(s.dpi), "s"(pl.groups), "s"(pl.mode), "s"(pl.gsize),
                 "s"(pl.gshift), "s"(blockDim.x));
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const int64_t w = item_at(pl, blockIdx.x, gridDim.x, i);
        int64_t grp;
        int g;
        split_item(w, pl.gsize, pl.gshift, grp, g);
        const int64_t r = grp / s.wcs;
        const int64_t c = grp - r * s.wcs;
        const int64_t v0 = c * cv + threadIdx.x;
        if (pl.gsize == 1 && !CACHED) {
            if ((c + 1) * cv <= s.mv)
                all_gather_chunk<VPT, true, true, WT>(tab, s, r, v0, nt, g, c * cv);
            else
                all_gather_chunk<VPT, false, true, WT>(tab, s, r, v0, nt, g, c * cv);
        } else {
            if ((c + 1) * cv <= s.mv)
                all_gather_chunk<VPT, true, false, WT>(tab, s, r, v0, nt, g, c * cv);
            else
                all_gather_chunk<VPT, false, false, WT>(tab, s, r, v0, nt, g, c * cv);
        }
    }
}

// Direct all-gather (every destination per work item): grid (chunks per
// shard, P), workgroup (c, r) copies chunk c of shard r to every destination.
// The source pointer is an argument indexed by the workgroup's y index; the
// destinations are compile-time offsets (see k_allreduce_direct).
template <int PT, int VPT, bool CACHED, bool WT>
__global__ __launch_bounds__(kWG) void k_all_gather_direct(Ptrs<PT> p, int64_t mv) {
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    const int64_t c = blockIdx.x;
    const int r = static_cast<int>(blockIdx.y);
    const int64_t v0 = c * cv + threadIdx.x;
    const uint4* src = p.in[r];
    uint4 y[VPT];
    const bool full = (c + 1) * cv <= mv;
    if (full)
        load_vecs<true, VPT, !CACHED>(y, src, v0, nt, mv);
    else
        load_vecs<false, VPT, !CACHED>(y, src, v0, nt, mv);
#pragma unroll
    for (int d = 0; d < PT; ++d) {
        uint4* dst = p.out[d] + r * mv;
        if (dst == src) continue;  // in-place shard
        if constexpr (WT) {
            if (full)
                store_vecs_wt<true, VPT>(dst + c * cv, y, static_cast<int>(threadIdx.x), nt, mv - c * cv);
            else
                store_vecs_wt<false, VPT>(dst + c * cv, y, static_cast<int>(threadIdx.x), nt, mv - c * cv);
        } else {
            if (full)
                store_vecs<true, VPT>(dst, y, v0, nt, mv);
            else
                store_vecs<false, VPT>(dst, y, v0, nt, mv);
        }
    }
}

template <int ES>
__global__ __launch_bounds__(kWG) void k_all_gather_elem(Ptrs<64> p, int P, int64_t m) {
    using E = typename std::conditional<ES == 2, uint16_t, uint32_t>::type;
    const int64_t total = m * P;
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < total;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t r = i / m;
        const int64_t j = i - r * m;
        const E* src = reinterpret_cast<const E*>(p.in[r]);
        const E v = src[j];
        for (int d = 0; d < P; ++d) {
            E* dst = reinterpret_cast<E*>(p.out[d]) + r * m;
            if (dst != src) dst[j] = v;
        }
    }
}

// ---------------------------------------------------------------- probe and copy

__global__ __launch_bounds__(64) void k_probe_xcc(int32_t* xcc, int32_t* hw_id) {
    if (threadIdx.x == 0) {
        uint32_t x, h;
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(h));
        xcc[blockIdx.x] = static_cast<int32_t>(x & 0xfu);
        if (hw_id) hw_id[blockIdx.x] = static_cast<int32_t>(h);
    }
}

// Reference copy.  It streams past the caches the way the collectives do
// (non-temporal 16-byte loads and stores), so its traffic-counter readings
// calibrate theirs and its speed is the ceiling a plain read+write reaches.
__global__ __launch_bounds__(kWG) void k_copy(uint4* __restrict__ dst, const uint4* __restrict__ src, int64_t nvec,
                                              unsigned char* __restrict__ dst_tail,
                                              const unsigned char* __restrict__ src_tail, int tail) {
    constexpr int U = 4;
    // One use of every argument: their loads issue together (as in the collectives).
    asm volatile("" ::"s"(dst), "s"(src), "s"(nvec), "s"(dst_tail), "s"(src_tail), "s"(tail));
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kWG * U;
    for (int64_t v = blockIdx.x * static_cast<int64_t>(kWG) * U + threadIdx.x; v < nvec; v += stride) {
        uint4 y[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (v + u * kWG < nvec) y[u] = load16<true>(src + v + u * kWG);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (v + u * kWG < nvec) store_stream(dst + v + u * kWG, y[u]);
    }
    if (blockIdx.x == 0 && static_cast<int>(threadIdx.x) < tail) dst_tail[threadIdx.x] = src_tail[threadIdx.x];
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
void launch_ar_direct_t(const void* const* in, void* const* out, const ArShape& s, int64_t G, int nt, hipStream_t st) {
    const Ptrs<PT> p = make_ptrs<PT>(in, out, PT, PT);
    hipLaunchKernelGGL((k_allreduce_direct<PT, DT, VPT, WT>), dim3(static_cast<unsigned>(G)), dim3(nt), 0, st, p,
                       s.nvec, s.tail);
}

// Direct kernel for 2, 4, 8 or 16 ranks (8 vectors per thread: 2, 4 or 8 ranks);
// write-through stores with 8 ranks when `wt`.
template <int DT, int VPT>
void launch_ar_direct_p(const void* const* in, void* const* out, int P, const ArShape& s, int64_t G, int nt, bool wt,
                        hipStream_t st) {
    switch (P) {
        case 2: launch_ar_direct_t<2, DT, VPT>(in, out, s, G, nt, st); break;
        case 4: launch_ar_direct_t<4, DT, VPT>(in, out, s, G, nt, st); break;
        case 8:
            if (wt) launch_ar_direct_t<8, DT, VPT, true>(in, out, s, G, nt, st);
            else launch_ar_direct_t<8, DT, VPT, false>(in, out, s, G, nt, st);
            break;
        default:
            if constexpr (VPT != 8) launch_ar_direct_t<16, DT, VPT>(in, out, s, G, nt, st);
            break;
    }
}

bool direct_ranks(int P, int vpt) { return P == 2 || P == 4 || P == 8 || (P == 16 && vpt != 8); }

// Largest grid that takes the direct kernels.  Beyond it the general kernels
// run: at 64 MiB per rank with one vector per thread (16384 workgroups) the
// general all-reduce measured 12 % faster than the direct one on MI355X (184
// against 209 us), while up to 8192 workgroups the direct kernels were as fast
// or faster at every size measured (1-64 MiB per rank, 1-4 vectors per thread).
constexpr int64_t kDirectMaxGrid = 8192;
constexpr int64_t kAgDirectMaxGrid8 = int64_t(1) << 20;  // 8-rank all-gather (launch_all_gather)

template <int PT, int MAXP, int DT, int VPT, bool KEEP>
void launch_rs_t(const void* const* in, void* const* out, int P, const RsShape& s, const Place& pl, int64_t G, int nt,
                 hipStream_t st) {
    Ptrs<MAXP> p = make_ptrs<MAXP>(in, out, P, P);
    hipLaunchKernelGGL((k_reduce_scatter<PT, MAXP, DT, VPT, KEEP>), dim3(static_cast<unsigned>(G)), dim3(nt), 0, st, p,
                       s, pl);
}

template <int DT, int VPT, bool KEEP>
void launch_rs_p(const void* const* in, void* const* out, int P, const RsShape& s, const Place& pl, int64_t G, int nt,
                 hipStream_t st) {
    switch (P) {
        case 2: launch_rs_t<2, 2, DT, VPT, KEEP>(in, out, P, s, pl, G, nt, st); break;
        case 4: launch_rs_t<4, 4, DT, VPT, KEEP>(in, out, P, s, pl, G, nt, st); break;
        case 8: launch_rs_t<8, 8, DT, VPT, KEEP>(in, out, P, s, pl, G, nt, st); break;
        case 16: launch_rs_t<16, 16, DT, VPT, KEEP>(in, out, P, s, pl, G, nt, st); break;
        default:
            if constexpr (VPT == 1) {
                if (P == 32) launch_rs_t<32, 64, DT, 1, KEEP>(in, out, P, s, pl, G, nt, st);
                else if (P == 64) launch_rs_t<64, 64, DT, 1, KEEP>(in, out, P, s, pl, G, nt, st);
                else launch_rs_t<0, 64, DT, 1, KEEP>(in, out, P, s, pl, G, nt, st);
            } else {
                launch_rs_t<0, 64, DT, VPT, KEEP>(in, out, P, s, pl, G, nt, st);  // other P up to 16 (above: VPT 1)
            }
            break;
    }
}

// Vectors per thread per work item for the all-reduce and reduce-scatter with
// up to 16 ranks, by message size (measured on MI355X with bf16, cold): 4 at
// 4 MiB per rank, 2 at 16 MiB, 1 at 64 MiB and above and for every smaller
// (latency-bound) message, where more workgroups win.
int pick_vpt(int64_t vectors_per_rank, int P) {
    if (P > 16) return 1;
    const int forced = tuning().vpt;
    if (forced == 1 || forced == 2 || forced == 4) return forced;
    if (forced == 8) return 4;  // 8 is an all-reduce-only shape
    if (vectors_per_rank >= (int64_t(1) << 22)) return 1;
    if (vectors_per_rank >= (int64_t(1) << 20)) return 2;
    if (vectors_per_rank >= (int64_t(1) << 18)) return 4;
    return 1;
}

// XCD placement keeps a logical group on one XCD so that its members'
// re-reads of the shared chunk hit that XCD's L2.  That pays only when the
// re-reads are a sizeable part of the group's traffic, and, for the split
// all-reduce (whose members all load the same P chunks at once), only once
// the message is large enough to be bandwidth-bound.  Otherwise the grouped
// map measured up to 3.5 % slower than the linear one on MI355X (split
// all-reduce at 8-16 KiB per rank with 8 ranks; all-gather with 64 ranks and
// 8 destinations per member), so the launch keeps the linear map there.
//   reread_num / reread_den: share of the group's loads and stores that are
//   re-reads; total_bytes: bytes the launch moves; min_total: the size below
//   which the grouped map is not used.
int group_mode(int mode, int64_t reread_num, int64_t reread_den, int64_t total_bytes, int64_t min_total) {
    if (mode != kPlaceXcd) return mode;
    if (reread_num * 4 < reread_den) return kPlaceLinear;
    if (total_bytes <= min_total) return kPlaceLinear;
    return mode;
}

int largest_divisor_upto(int P, int cap) {
    for (int d = cap < P ? cap : P; d > 1; --d)
        if (P % d == 0) return d;
    return 1;
}

// Workgroup size: one-wavefront workgroups spread small messages, and the
// long per-thread rank loops of many-rank reductions, over more compute
// units; 256-thread workgroups stream large few-rank messages, except at
// 4 MiB per rank where 128 threads with 4 vectors each measured best.
int pick_threads(int64_t vectors_per_rank, int P) {
    const int forced = tuning().wg_threads;
    if (forced == 64 || forced == 128 || forced == 256) return forced;
    if (P > 16) return 64;
    if (vectors_per_rank < (int64_t(1) << 14)) return 64;
    if (vectors_per_rank >= (int64_t(1) << 18) && vectors_per_rank < (int64_t(1) << 20)) return 128;
    return kWG;
}

// Reduce-scatter launch shape by the vectors each input rank holds (P
// shards), for up to 16 ranks (measured on MI355X with bf16, 8 ranks, cold):
// 4 vectors per thread from 8 MiB per input rank, where it was 7-9 % faster
// than the all-reduce's shapes; 128 threads with 2 at 4 MiB; the
// all-reduce's rule below that.  Forced tunables win.
void pick_rs_shape(int64_t in_vectors, int P, int dtype, int& nt, int& vpt) {
    nt = pick_threads(in_vectors, P);
    vpt = dtype == kDtBf16 ? pick_vpt(in_vectors, P) : 1;
    if (P > 16 || dtype != kDtBf16 || tuning().wg_threads || tuning().vpt) return;
    if (in_vectors >= (int64_t(1) << 19)) {
        nt = 256;
        vpt = 4;
    } else if (in_vectors >= (int64_t(1) << 18)) {
        nt = 128;
        vpt = 2;
    }
}

// All-gather launch shape by the vectors each output rank receives, for up
// to 16 ranks (measured on MI355X with bf16, 8 ranks, cold): one-wave
// workgroups with 1 vector per thread below 2 MiB per output, 64 threads with
// 4 vectors below 16 MiB, 5-20 % faster than the all-reduce's shapes.  From
// 16 MiB per output, 8 ranks have a rule of their own (below); other rank
// counts take 128 threads with 4 vectors below 64 MiB and 128 with 1 beyond.
// Forced tunables win.
void pick_ag_shape(int64_t out_vectors, int P, int& nt, int& vpt) {
    nt = pick_threads(out_vectors, P);
    vpt = pick_vpt(out_vectors, P);
    if (P > 16 || tuning().wg_threads || tuning().vpt) return;
    if (out_vectors < (int64_t(1) << 17)) {
        nt = 64;
        vpt = 1;
    } else if (out_vectors < (int64_t(1) << 20)) {
        nt = 64;
        vpt = 4;
    } else if (P == 8) {
        // 8 ranks from 2 MiB shards: 256 x 1, with the direct kernel at any
        // grid (launch_all_gather).  Measured on MI355X with back-to-back cold
        // calls: 3-11 % faster than 128 x 4 at 2-4 MiB shards (37.9 against
        // 42.8 us at 3 MiB), best or within 1 % of the best shape at 4-32 MiB.
        nt = 256;
        vpt = 1;
    } else if (out_vectors < (int64_t(1) << 22)) {
        nt = 128;
        vpt = 4;
    } else {
        nt = 128;
        vpt = 1;
    }
}

// One-shot all-reduce launch shape.  Starts from the shared rule above; with
// 2, 4 or 8 ranks a forced 8 vectors per thread is kept (other rank counts
// have no such kernel and get 4).
//
// 8 ranks, 8-32 MiB per rank: 8 vectors per thread in 256-thread workgroups.
// That kernel holds 256 VGPRs, so one workgroup per CU runs at a time and
// the launch proceeds in rounds of 256 workgroups, each moving 32 KiB
// contiguous per rank buffer.  Measured on MI355X (bf16, cold) it was 5-8 %
// faster than the shared rule at 8 and 16 MiB per rank, when its chunks fill
// whole rounds; with a partly empty last round it lost, so it is taken only
// when the last round is at least 90 % full.
void pick_ar_shape(int64_t vectors_per_rank, int P, int& nt, int& vpt) {
    nt = pick_threads(vectors_per_rank, P);
    vpt = pick_vpt(vectors_per_rank, P);
    const bool eight_ok = P == 2 || P == 4 || P == 8;
    if (tuning().vpt == 8 && eight_ok) {
        vpt = 8;
        return;
    }
    if (P != 8 || tuning().wg_threads || tuning().vpt) return;
    if (vectors_per_rank < (int64_t(1) << 19) || vectors_per_rank > (int64_t(1) << 21)) return;
    constexpr int64_t kChunk = 256 * 8, kRound = 256;
    const int64_t G = (vectors_per_rank + kChunk - 1) / kChunk;
    const int64_t rounds = (G + kRound - 1) / kRound;
    if (G * 10 >= rounds * kRound * 9) {
        nt = 256;
        vpt = 8;
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
    if (dtype == kDtF32)
        launch_lpr_p<kDtF32>(in, out, P, s, pl, G, stream);
    else
        launch_lpr_p<kDtBf16>(in, out, P, s, pl, G, stream);
    return hipGetLastError();
}

template <int PT, int DT, int V>
void launch_tile_t(const void* const* in, void* const* out, int P, const TileShape& s, const Place& pl, int64_t G,
                   bool direct, hipStream_t st) {
    Ptrs<64> p = make_ptrs<64>(in, out, P, P);
    const size_t lds = static_cast<size_t>(P) * V * 16;
    if (direct)
        hipLaunchKernelGGL((k_allreduce_tile_direct<PT, DT, V>), dim3(static_cast<unsigned>(G)), dim3(kWG), lds, st, p,
                           s);
    else
        hipLaunchKernelGGL((k_allreduce_tile<PT, DT, V>), dim3(static_cast<unsigned>(G)), dim3(kWG), lds, st, p, s,
                           pl);
}

template <int DT, int V>
void launch_tile_p(const void* const* in, void* const* out, int P, const TileShape& s, const Place& pl, int64_t G,
                   bool direct, hipStream_t st) {
    switch (P) {
        case 16: launch_tile_t<16, DT, V>(in, out, P, s, pl, G, direct, st); break;
        case 32: launch_tile_t<32, DT, V>(in, out, P, s, pl, G, direct, st); break;
        case 64: launch_tile_t<64, DT, V>(in, out, P, s, pl, G, direct, st); break;
        default: launch_tile_t<0, DT, V>(in, out, P, s, pl, G, direct, st); break;
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
    const bool direct = G == groups && G <= kDirectMaxGrid;  // one item per workgroup, no placement state
    if (dtype == kDtF32) {
        if (V == 16) launch_tile_p<kDtF32, 16>(in, out, P, s, pl, G, direct, stream);
        else if (V == 32) launch_tile_p<kDtF32, 32>(in, out, P, s, pl, G, direct, stream);
        else launch_tile_p<kDtF32, 64>(in, out, P, s, pl, G, direct, stream);
    } else {
        if (V == 16) launch_tile_p<kDtBf16, 16>(in, out, P, s, pl, G, direct, stream);
        else if (V == 32) launch_tile_p<kDtBf16, 32>(in, out, P, s, pl, G, direct, stream);
        else launch_tile_p<kDtBf16, 64>(in, out, P, s, pl, G, direct, stream);
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
    const int gsize = dest_groups > 1 ? dest_groups : 1;
    s.dpi = P / gsize;
    int nt, vpt;
    pick_ar_shape(s.nvec, P, nt, vpt);
    if (vpt == 8 && P != 2 && P != 4 && P != 8) return hipErrorInvalidValue;
    const int64_t cv = static_cast<int64_t>(nt) * vpt;
    const int64_t groups = (s.nvec + cv - 1) / cv;
    // A split group reads the chunk of all P ranks gsize times and writes it to
    // P destinations: (gsize - 1) * P of its gsize * P + P transfers are re-reads.
    const int gmode = gsize > 1 ? group_mode(mode, int64_t(gsize - 1) * P, int64_t(gsize) * P + P,
                                             static_cast<int64_t>(2 * P) * static_cast<int64_t>(bytes),
                                             int64_t(256) << 10)
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
    // One item per workgroup on the linear map: the direct kernel.
    if (gsize == 1 && G == groups && G <= kDirectMaxGrid && direct_ranks(P, vpt)) {
        if (dtype == kDtF32) {
            if (vpt == 8) launch_ar_direct_p<kDtF32, 8>(in, out, P, s, G, nt, wt, stream);
            else if (vpt == 4) launch_ar_direct_p<kDtF32, 4>(in, out, P, s, G, nt, wt, stream);
            else if (vpt == 2) launch_ar_direct_p<kDtF32, 2>(in, out, P, s, G, nt, wt, stream);
            else launch_ar_direct_p<kDtF32, 1>(in, out, P, s, G, nt, wt, stream);
        } else {
            if (vpt == 8) launch_ar_direct_p<kDtBf16, 8>(in, out, P, s, G, nt, wt, stream);
            else if (vpt == 4) launch_ar_direct_p<kDtBf16, 4>(in, out, P, s, G, nt, wt, stream);
            else if (vpt == 2) launch_ar_direct_p<kDtBf16, 2>(in, out, P, s, G, nt, wt, stream);
            else launch_ar_direct_p<kDtBf16, 1>(in, out, P, s, G, nt, wt, stream);
        }
        return hipGetLastError();
    }
    // The kernel's vectors per thread must be the VPT the chunks were sized with.
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

template <int PT, int DT, int VPT, bool KEEP>
void launch_rs_direct_t(const void* const* in, void* const* out, const RsShape& s, int nt, hipStream_t st) {
    const Ptrs<PT> p = make_ptrs<PT>(in, out, PT, PT);
    hipLaunchKernelGGL((k_reduce_scatter_direct<PT, DT, VPT, KEEP>),
                       dim3(static_cast<unsigned>(s.wcs), static_cast<unsigned>(PT)), dim3(nt), 0, st, p, s.mv);
}

template <int DT, int VPT, bool KEEP>
void launch_rs_direct_p(const void* const* in, void* const* out, int P, const RsShape& s, int nt, hipStream_t st) {
    switch (P) {
        case 2: launch_rs_direct_t<2, DT, VPT, KEEP>(in, out, s, nt, st); break;
        case 4: launch_rs_direct_t<4, DT, VPT, KEEP>(in, out, s, nt, st); break;
        case 8: launch_rs_direct_t<8, DT, VPT, KEEP>(in, out, s, nt, st); break;
        default: launch_rs_direct_t<16, DT, VPT, KEEP>(in, out, s, nt, st); break;
    }
}

// Every uncapped reduce-scatter of 2, 4, 8 or 16 ranks (single-item groups,
// so both placements run the linear map).
hipError_t launch_rs_direct(const void* const* in, void* const* out, int P, const RsShape& s, int dtype, int vpt,
                            int nt, bool keep, hipStream_t st) {
    if (dtype == kDtF32) {
        if (keep) launch_rs_direct_p<kDtF32, 1, true>(in, out, P, s, nt, st);
        else launch_rs_direct_p<kDtF32, 1, false>(in, out, P, s, nt, st);
    } else if (vpt == 4) {
        if (keep) launch_rs_direct_p<kDtBf16, 4, true>(in, out, P, s, nt, st);
        else launch_rs_direct_p<kDtBf16, 4, false>(in, out, P, s, nt, st);
    } else if (vpt == 2) {
        if (keep) launch_rs_direct_p<kDtBf16, 2, true>(in, out, P, s, nt, st);
        else launch_rs_direct_p<kDtBf16, 2, false>(in, out, P, s, nt, st);
    } else {
        if (keep) launch_rs_direct_p<kDtBf16, 1, true>(in, out, P, s, nt, st);
        else launch_rs_direct_p<kDtBf16, 1, false>(in, out, P, s, nt, st);
    }
    return hipGetLastError();
}

hipError_t launch_reduce_scatter(const void* const* in, void* const* out, int P, size_t m, int dtype, int mode,
                                 bool keep_output, hipStream_t stream) {
    const size_t es = dtype_size(dtype);
    if ((m * es) % 16 != 0) {
        Ptrs<64> p = make_ptrs<64>(in, out, P, P);
        const int64_t total = static_cast<int64_t>(m) * P;
        const int64_t G = cap_grid((total + kWG - 1) / kWG);
        if (dtype == kDtF32)
            hipLaunchKernelGGL((k_reduce_scatter_elem<kDtF32>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream,
                               p, P, static_cast<int64_t>(m));
        else
            hipLaunchKernelGGL((k_reduce_scatter_elem<kDtBf16>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream,
                               p, P, static_cast<int64_t>(m));
        return hipGetLastError();
    }
    RsShape s{};
    s.mv = static_cast<int64_t>(m * es / 16);
    s.P = P;
    // Shape by the vectors each input rank holds (P shards of mv vectors).
    int nt, vpt;
    pick_rs_shape(s.mv * P, P, dtype, nt, vpt);
    const int64_t cv = static_cast<int64_t>(nt) * vpt;
    s.wcs = (s.mv + cv - 1) / cv;
    const Place pl = make_place_uniform(mode, s.wcs * P, 1);
    const int64_t G = cap_grid(place_grid(pl));
    if (G == s.wcs * P && G <= kDirectMaxGrid && (P == 2 || P == 4 || P == 8 || P == 16))
        return launch_rs_direct(in, out, P, s, dtype, vpt, nt, keep_output, stream);
    if (dtype == kDtF32) {
        if (keep_output) launch_rs_p<kDtF32, 1, true>(in, out, P, s, pl, G, nt, stream);
        else launch_rs_p<kDtF32, 1, false>(in, out, P, s, pl, G, nt, stream);
    } else if (vpt == 4) {
        if (keep_output) launch_rs_p<kDtBf16, 4, true>(in, out, P, s, pl, G, nt, stream);
        else launch_rs_p<kDtBf16, 4, false>(in, out, P, s, pl, G, nt, stream);
    } else if (vpt == 2) {
        if (keep_output) launch_rs_p<kDtBf16, 2, true>(in, out, P, s, pl, G, nt, stream);
        else launch_rs_p<kDtBf16, 2, false>(in, out, P, s, pl, G, nt, stream);
    } else {
        if (keep_output) launch_rs_p<kDtBf16, 1, true>(in, out, P, s, pl, G, nt, stream);
        else launch_rs_p<kDtBf16, 1, false>(in, out, P, s, pl, G, nt, stream);
    }
    return hipGetLastError();
}

// Write-through variants exist for the cached-source (two-shot) phase with 8 ranks.
template <int PT>
void launch_ag_direct_p(const void* const* in, void* const* out, const AgShape& s, int vpt, bool cached, bool wt,
                        dim3 g, dim3 b, hipStream_t st) {
    const Ptrs<PT> p = make_ptrs<PT>(in, out, PT, PT);
    if (cached && wt && PT == 8) {
        if (vpt == 4) hipLaunchKernelGGL((k_all_gather_direct<PT, 4, true, true>), g, b, 0, st, p, s.mv);
        else if (vpt == 2) hipLaunchKernelGGL((k_all_gather_direct<PT, 2, true, true>), g, b, 0, st, p, s.mv);
        else hipLaunchKernelGGL((k_all_gather_direct<PT, 1, true, true>), g, b, 0, st, p, s.mv);
    } else if (cached) {
        if (vpt == 4) hipLaunchKernelGGL((k_all_gather_direct<PT, 4, true, false>), g, b, 0, st, p, s.mv);
        else if (vpt == 2) hipLaunchKernelGGL((k_all_gather_direct<PT, 2, true, false>), g, b, 0, st, p, s.mv);
        else hipLaunchKernelGGL((k_all_gather_direct<PT, 1, true, false>), g, b, 0, st, p, s.mv);
    } else {
        if (vpt == 4) hipLaunchKernelGGL((k_all_gather_direct<PT, 4, false, false>), g, b, 0, st, p, s.mv);
        else if (vpt == 2) hipLaunchKernelGGL((k_all_gather_direct<PT, 2, false, false>), g, b, 0, st, p, s.mv);
        else hipLaunchKernelGGL((k_all_gather_direct<PT, 1, false, false>), g, b, 0, st, p, s.mv);
    }
}

hipError_t launch_all_gather(const void* const* in, void* const* out, int P, size_t m, int dtype, int mode,
                             bool src_cached, hipStream_t stream) {
    const size_t es = dtype_size(dtype);
    if ((m * es) % 16 != 0) {
        Ptrs<64> p = make_ptrs<64>(in, out, P, P);
        const int64_t total = static_cast<int64_t>(m) * P;
        const int64_t G = cap_grid((total + kWG - 1) / kWG);
        if (es == 4)
            hipLaunchKernelGGL((k_all_gather_elem<4>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, P,
                               static_cast<int64_t>(m));
        else
            hipLaunchKernelGGL((k_all_gather_elem<2>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, P,
                               static_cast<int64_t>(m));
        return hipGetLastError();
    }
    AgShape s{};
    s.mv = static_cast<int64_t>(m * es / 16);
    s.P = P;
    // Shape by the vectors each output rank receives (P shards of mv vectors).
    int nt, vpt;
    pick_ag_shape(s.mv * P, P, nt, vpt);
    const int64_t cv = static_cast<int64_t>(nt) * vpt;
    s.wcs = (s.mv + cv - 1) / cv;
    // Split destinations when there are few chunks, so that more workgroups
    // share the stores; each member re-reads its chunk (an L2 hit when the
    // group's members sit on one XCD).
    const int gsize = (s.wcs * P < 512) ? largest_divisor_upto(P, 8) : 1;
    s.dpi = P / gsize;
    // Each member loads the chunk once and stores it dpi times: gsize - 1 of
    // the group's gsize * (1 + dpi) transfers are re-reads.
    const int gmode = gsize > 1 ? group_mode(mode, gsize - 1, int64_t(gsize) * (1 + s.dpi),
                                             static_cast<int64_t>(P + 1) * P * static_cast<int64_t>(m * es), 0)
                                : mode;
    const Place pl = make_place_uniform(gmode, s.wcs * P, gsize);
    const int64_t G = cap_grid(place_grid(pl));
    // Write-through stores in the two-shot's all-gather phase (the shards were
    // just written and are read through the caches) with 8 ranks, at 1-2 MiB
    // shards.  Against streaming stores on MI355X, whole two-shot, back-to-back
    // cold calls: 4.3 % faster at 2 MiB shards, +0.2-0.5 % at 1-1.5 MiB; the
    // gain does not grow smoothly beyond (-4.7 % at 3 MiB, +3.4 % at 4 MiB,
    // -9 % at 6-8 MiB) and is -12 % at 0.5 MiB.
    const int wtf = tuning().write_through;
    const int64_t shard = static_cast<int64_t>(m * es);
    const bool wt = P == 8 && src_cached && gsize == 1 &&
                    (wtf == 2 || (wtf == 0 && shard >= (int64_t(1) << 20) && shard <= (int64_t(2) << 20)));
    // The direct kernel when every chunk item has its own workgroup.  With 8
    // ranks it takes grids beyond kDirectMaxGrid too: against the general
    // kernel's persistent loop it measured 6-10 % faster at 6-32 MiB shards on
    // MI355X (103 against 114 us at 8 MiB, 418 against 457 us at 32 MiB).
    const int64_t items = s.wcs * P;
    const bool direct = gsize == 1 && (P == 8 ? items <= grid_limit(kAgDirectMaxGrid8)
                                              : (P == 2 || P == 4) && G == items && G <= kDirectMaxGrid);
    if (direct) {
        const dim3 g(static_cast<unsigned>(s.wcs), static_cast<unsigned>(P)), b(nt);
        switch (P) {
            case 2: launch_ag_direct_p<2>(in, out, s, vpt, src_cached, false, g, b, stream); break;
            case 4: launch_ag_direct_p<4>(in, out, s, vpt, src_cached, false, g, b, stream); break;
            default: launch_ag_direct_p<8>(in, out, s, vpt, src_cached, wt, g, b, stream); break;
        }
        return hipGetLastError();
    }
    if (P <= 8) {
        Ptrs<8> p = make_ptrs<8>(in, out, P, P);
        const dim3 g(static_cast<unsigned>(G)), b(nt);
        if (src_cached && wt) {
            if (vpt == 4) hipLaunchKernelGGL((k_all_gather<8, 4, true, true>), g, b, 0, stream, p, s, pl);
            else if (vpt == 2) hipLaunchKernelGGL((k_all_gather<8, 2, true, true>), g, b, 0, stream, p, s, pl);
            else hipLaunchKernelGGL((k_all_gather<8, 1, true, true>), g, b, 0, stream, p, s, pl);
        } else if (src_cached) {
            if (vpt == 4) hipLaunchKernelGGL((k_all_gather<8, 4, true, false>), g, b, 0, stream, p, s, pl);
            else if (vpt == 2) hipLaunchKernelGGL((k_all_gather<8, 2, true, false>), g, b, 0, stream, p, s, pl);
            else hipLaunchKernelGGL((k_all_gather<8, 1, true, false>), g, b, 0, stream, p, s, pl);
        } else {
            if (vpt == 4) hipLaunchKernelGGL((k_all_gather<8, 4, false, false>), g, b, 0, stream, p, s, pl);
            else if (vpt == 2) hipLaunchKernelGGL((k_all_gather<8, 2, false, false>), g, b, 0, stream, p, s, pl);
            else hipLaunchKernelGGL((k_all_gather<8, 1, false, false>), g, b, 0, stream, p, s, pl);
        }
    } else {
        Ptrs<64> p = make_ptrs<64>(in, out, P, P);
        const dim3 g(static_cast<unsigned>(G)), b(nt);
        if (src_cached) {
            if (vpt == 4) hipLaunchKernelGGL((k_all_gather<64, 4, true, false>), g, b, 0, stream, p, s, pl);
            else if (vpt == 2) hipLaunchKernelGGL((k_all_gather<64, 2, true, false>), g, b, 0, stream, p, s, pl);
            else hipLaunchKernelGGL((k_all_gather<64, 1, true, false>), g, b, 0, stream, p, s, pl);
        } else {
            if (vpt == 4) hipLaunchKernelGGL((k_all_gather<64, 4, false, false>), g, b, 0, stream, p, s, pl);
            else if (vpt == 2) hipLaunchKernelGGL((k_all_gather<64, 2, false, false>), g, b, 0, stream, p, s, pl);
            else hipLaunchKernelGGL((k_all_gather<64, 1, false, false>), g, b, 0, stream, p, s, pl);
        }
    }
    return hipGetLastError();
}

hipError_t launch_probe_xcc(int G, int32_t* xcc, int32_t* hw_id, hipStream_t stream) {
    hipLaunchKernelGGL(k_probe_xcc, dim3(static_cast<unsigned>(G)), dim3(64), 0, stream, xcc, hw_id);
    return hipGetLastError();
}

hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t stream) {
    const int64_t nvec = static_cast<int64_t>(bytes / 16);
    const int tail = static_cast<int>(bytes % 16);
    const int64_t per_wg = static_cast<int64_t>(kWG) * 4;
    int64_t G = (nvec + per_wg - 1) / per_wg;
    if (G > 4096) G = 4096;
    if (G < 1) G = 1;
    hipLaunchKernelGGL(k_copy, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, static_cast<uint4*>(dst),
                       static_cast<const uint4*>(src), nvec, static_cast<unsigned char*>(dst) + nvec * 16,
                       static_cast<const unsigned char*>(src) + nvec * 16, tail);
    return hipGetLastError();
}

}  // namespace nuna
