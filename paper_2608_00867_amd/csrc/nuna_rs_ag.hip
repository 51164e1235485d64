// nuna_rs_ag.hip -- gfx950 reduce-scatter and all-gather kernels (standalone,
// and the two phases of the two-kernel two-shot all-reduce), and their
// launchers.  Same numerics and 16-byte streaming accesses as the all-reduce
// kernels.
#include "device_common.h"
#include "shapes.h"

namespace nuna {
namespace {

// ---------------------------------------------------------------- reduce-scatter

struct RsShape {
    int64_t mv;   // vectors per shard
    int64_t wcs;  // chunks per shard
    int32_t P;
    int32_t pad;
};

// SEL: the output pointer of shard r is picked among the pinned pointers
// (direct kernel, up to 8 ranks) instead of loaded from the arguments.
template <int PT, int DT, int VPT, bool FULL, bool KEEP, int MAXP, bool SEL = false>
__device__ __forceinline__ void reduce_scatter_chunk(const Ptrs<MAXP>& p, const RankTable& tab, const RsShape& s,
                                                     int P, int64_t r, int64_t v0, int nt) {
    using A = Arith<DT>;
    float acc[VPT][A::kLanes];
    reduce_ranks<PT, DT, VPT, FULL, true>(p, tab, P, r * s.mv, v0, nt, s.mv, acc);
    uint4 y[VPT];
#pragma unroll
    for (int j = 0; j < VPT; ++j) y[j] = A::narrow(acc[j]);
    uint4* dst;
    if constexpr (SEL)
        dst = out_at(p, static_cast<int>(r));
    else
        dst = use_table<PT>() ? rank_out(tab, static_cast<int>(r)) : p.out[r];
    store_vecs<FULL, VPT, !KEEP>(dst, y, v0, nt, s.mv);
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
    pin_args(p, mv, blockDim.x, blockIdx.y);
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
        reduce_scatter_chunk<PT, DT, VPT, true, KEEP, PT, (PT <= 8)>(p, tab, s, PT, r, v0, nt);
    else
        reduce_scatter_chunk<PT, DT, VPT, false, KEEP, PT, (PT <= 8)>(p, tab, s, PT, r, v0, nt);
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
    int32_t gap;  // store_gap between destinations
    int32_t pad;
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
        if (d > d0) store_gap(s.gap);
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
    asm volatile("" ::"s"(s.mv), "s"(s.wcs), "s"(s.dpi), "s"(s.gap), "s"(pl.groups), "s"(pl.mode), "s"(pl.gsize),
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
__global__ __launch_bounds__(kWG) void k_all_gather_direct(Ptrs<PT> p, int64_t mv, int32_t gap) {
    pin_args(p, mv, gap, blockDim.x);
    const int nt = blockDim.x;
    const int64_t cv = static_cast<int64_t>(nt) * VPT;
    const int64_t c = blockIdx.x;
    const int r = static_cast<int>(blockIdx.y);
    const int64_t v0 = c * cv + threadIdx.x;
    const uint4* src = in_at(p, r);
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
        if (d > 0) store_gap(gap);
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

}  // namespace

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
        note_launch("k_reduce_scatter_elem", kMapLinear, 1, G, kWG, 0);
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
    // Every work item is its own group: both placements run the linear map.
    if (G == s.wcs * P && G <= direct_max_grid() && (P == 2 || P == 4 || P == 8 || P == 16)) {
        note_launch("k_reduce_scatter_direct", kMapLinear, 1, G, nt, vpt);
        return launch_rs_direct(in, out, P, s, dtype, vpt, nt, keep_output, stream);
    }
    note_launch("k_reduce_scatter", kMapLinear, 1, G, nt, vpt);
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
        if (vpt == 4) hipLaunchKernelGGL((k_all_gather_direct<PT, 4, true, true>), g, b, 0, st, p, s.mv, s.gap);
        else if (vpt == 2) hipLaunchKernelGGL((k_all_gather_direct<PT, 2, true, true>), g, b, 0, st, p, s.mv, s.gap);
        else hipLaunchKernelGGL((k_all_gather_direct<PT, 1, true, true>), g, b, 0, st, p, s.mv, s.gap);
    } else if (cached) {
        if (vpt == 4) hipLaunchKernelGGL((k_all_gather_direct<PT, 4, true, false>), g, b, 0, st, p, s.mv, s.gap);
        else if (vpt == 2) hipLaunchKernelGGL((k_all_gather_direct<PT, 2, true, false>), g, b, 0, st, p, s.mv, s.gap);
        else hipLaunchKernelGGL((k_all_gather_direct<PT, 1, true, false>), g, b, 0, st, p, s.mv, s.gap);
    } else {
        if (vpt == 4) hipLaunchKernelGGL((k_all_gather_direct<PT, 4, false, false>), g, b, 0, st, p, s.mv, s.gap);
        else if (vpt == 2) hipLaunchKernelGGL((k_all_gather_direct<PT, 2, false, false>), g, b, 0, st, p, s.mv, s.gap);
        else hipLaunchKernelGGL((k_all_gather_direct<PT, 1, false, false>), g, b, 0, st, p, s.mv, s.gap);
    }
}

hipError_t launch_all_gather(const void* const* in, void* const* out, int P, size_t m, int dtype, int mode,
                             bool src_cached, hipStream_t stream) {
    const size_t es = dtype_size(dtype);
    if ((m * es) % 16 != 0) {
        Ptrs<64> p = make_ptrs<64>(in, out, P, P);
        const int64_t total = static_cast<int64_t>(m) * P;
        const int64_t G = cap_grid((total + kWG - 1) / kWG);
        note_launch("k_all_gather_elem", kMapLinear, 1, G, kWG, 0);
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
    s.gap = store_gap_for(m * es * P);
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
    // the group's gsize * (1 + dpi) transfers are re-reads.  The grouped map
    // from launches of more than 2 MiB, as for the split all-reduce: below, with
    // 8 ranks at 2-32 KiB shards, it was within 1 % of the linear map cold and
    // up to 2 % slower with warm inputs on MI355X.
    const int gmode = gsize > 1 ? group_mode(mode, gsize - 1, int64_t(gsize) * (1 + s.dpi),
                                             static_cast<int64_t>(P + 1) * P * static_cast<int64_t>(m * es),
                                             int64_t(2) << 20)
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
    // ranks it takes grids beyond the direct-grid limit too: against the general
    // kernel's persistent loop it measured 6-10 % faster at 6-32 MiB shards on
    // MI355X (103 against 114 us at 8 MiB, 418 against 457 us at 32 MiB).
    const int64_t items = s.wcs * P;
    const bool direct = gsize == 1 && (P == 8 ? items <= grid_limit(kAgDirectMaxGrid8)
                                              : (P == 2 || P == 4) && G == items && G <= direct_max_grid());
    if (direct) {
        note_launch("k_all_gather_direct", kMapLinear, 1, items, nt, vpt);
        const dim3 g(static_cast<unsigned>(s.wcs), static_cast<unsigned>(P)), b(nt);
        switch (P) {
            case 2: launch_ag_direct_p<2>(in, out, s, vpt, src_cached, false, g, b, stream); break;
            case 4: launch_ag_direct_p<4>(in, out, s, vpt, src_cached, false, g, b, stream); break;
            default: launch_ag_direct_p<8>(in, out, s, vpt, src_cached, wt, g, b, stream); break;
        }
        return hipGetLastError();
    }
    note_launch("k_all_gather", pl.mode == kPlaceXcd && !linear_map(pl, G) ? kMapXcdGroups : kMapLinear, pl.gsize, G,
                nt, vpt);
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

}  // namespace nuna
