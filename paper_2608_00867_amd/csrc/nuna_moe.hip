// nuna_moe.hip -- gfx950 kernels of MoE expert parallelism: the all-to-all
// dispatch of token rows to the ranks of their experts, and the combine that
// sums the expert results back into each token's row.
//
// Row copies and row sums of 16-byte vectors; the dispatch is driven by a
// per-item descriptor list in placement order, the combine by per-token
// (rank, row) lists.  No MFMA: rows are moved and added, never contracted.
#include "device_common.h"

namespace nuna {
namespace {

// ---------------------------------------------------------------- all-to-all

// One descriptor per row copy, stored in placement order: source rank,
// source token, destination rank, destination row.
template <int MAXP, int UNROLL>
__global__ __launch_bounds__(kWG) void k_all_to_all(Ptrs<MAXP> p, int P, const int4* __restrict__ desc,
                                                    int64_t rowvec, Place pl) {
    const int nt = blockDim.x;
    const RankTable tab = load_rank_table(p, P);
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const int4 d = desc[i];
        const uint4* src = rank_in(tab, d.x) + static_cast<int64_t>(d.y) * rowvec;
        uint4* dst = rank_out(tab, d.z) + static_cast<int64_t>(d.w) * rowvec;
        for (int64_t v = threadIdx.x; v < rowvec; v += static_cast<int64_t>(nt) * UNROLL) {
            uint4 y[UNROLL];
#pragma unroll
            for (int u = 0; u < UNROLL; ++u)
                if (v + u * nt < rowvec) y[u] = src[v + u * nt];
#pragma unroll
            for (int u = 0; u < UNROLL; ++u)
                if (v + u * nt < rowvec) store_stream(dst + v + u * nt, y[u]);
        }
    }
}

// Element path for rows that are not a whole number of 16-byte vectors.
template <int ES>
__global__ __launch_bounds__(kWG) void k_all_to_all_elem(Ptrs<64> p, const int4* __restrict__ desc, int64_t rowelems,
                                                         Place pl) {
    using E = typename std::conditional<ES == 2, uint16_t, uint32_t>::type;
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const int4 d = desc[i];
        const E* src = reinterpret_cast<const E*>(p.in[d.x]) + static_cast<int64_t>(d.y) * rowelems;
        E* dst = reinterpret_cast<E*>(p.out[d.z]) + static_cast<int64_t>(d.w) * rowelems;
        for (int64_t v = threadIdx.x; v < rowelems; v += blockDim.x) dst[v] = src[v];
    }
}

// ---------------------------------------------------------------- all-to-all combine

// MoE result collection, the reverse of the dispatch: every token gets back
// one result row from each distinct rank it was sent to, and the rows are
// summed.  Work item w is column chunk w mod C of token w div C (C column
// chunks of `cw` vectors per row); token i = s*T + t writes output row t of
// rank s.  The token's (rank, row) entries come in ascending rank order; the
// sum follows that order in fp32 and is rounded once.  Each result row is
// read by one work item only, so the loads stream past the caches.
struct CombShape {
    int64_t rowvec;   // 16-byte vectors per row
    int64_t cw;       // vectors per column chunk
    uint32_t T;       // tokens per rank
    uint32_t chunks;  // column chunks per token (C)
    int32_t P;
    int32_t pad;
};

// WT: each term is first scaled by the fp32 weight w[tok * P + rank] (the
// product is rounded once; no fused multiply-add).
template <int MAXP, int DT, int VPT, bool WT>
__global__ __launch_bounds__(kWG) void k_combine(Ptrs<MAXP> p, const int64_t* __restrict__ off,
                                                 const int2* __restrict__ ent, const float* __restrict__ wts,
                                                 CombShape s, Place pl) {
    using A = Arith<DT>;
    constexpr int B = 8;  // result rows loaded per batch
    const int nt = blockDim.x;
    const RankTable tab = load_rank_table(p, s.P);
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const uint32_t w = static_cast<uint32_t>(item_at(pl, blockIdx.x, gridDim.x, i));
        const uint32_t tok = w / s.chunks;
        const int64_t lo = static_cast<int64_t>(w - tok * s.chunks) * s.cw;
        const int64_t hi = lo + s.cw < s.rowvec ? lo + s.cw : s.rowvec;
        const uint32_t src = tok / s.T;
        const uint32_t t = tok - src * s.T;
        const int64_t e0 = off[tok];
        const int c = static_cast<int>(off[tok + 1] - e0);
        uint4* dst = rank_out(tab, static_cast<int>(src)) + static_cast<int64_t>(t) * s.rowvec;
        // Uniform trip count (rank pointers come from v_readlane); lanes past
        // `hi` are masked inside the loads and stores.
        for (int64_t v0 = lo; v0 < hi; v0 += static_cast<int64_t>(nt) * VPT) {
            const int64_t v = v0 + threadIdx.x;
            float acc[VPT][A::kLanes];
            for (int q0 = 0; q0 < c; q0 += B) {
                uint4 buf[B][VPT];
                float wq[B];
#pragma unroll
                for (int q = 0; q < B; ++q) {
                    if (q0 + q < c) {
                        const int2 e = ent[e0 + q0 + q];
                        const uint4* row = rank_in(tab, e.x) + static_cast<int64_t>(e.y) * s.rowvec;
                        load_vecs<false, VPT, true>(buf[q], row, v, nt, hi);
                        if constexpr (WT) wq[q] = wts[static_cast<int64_t>(tok) * s.P + e.x];
                    }
                }
#pragma unroll
                for (int q = 0; q < B; ++q) {
                    if (q0 + q < c) {
#pragma unroll
                        for (int j = 0; j < VPT; ++j) {
                            if constexpr (WT) {
                                float t[A::kLanes];
                                A::init(t, buf[q][j]);
#pragma unroll
                                for (int l = 0; l < A::kLanes; ++l) {
                                    const float term = wq[q] * t[l];
                                    acc[j][l] = q0 + q == 0 ? term : acc[j][l] + term;
                                }
                            } else {
                                if (q0 + q == 0)
                                    A::init(acc[j], buf[q][j]);
                                else
                                    A::add(acc[j], buf[q][j]);
                            }
                        }
                    }
                }
            }
            uint4 y[VPT];
#pragma unroll
            for (int j = 0; j < VPT; ++j) y[j] = A::narrow(acc[j]);
            store_vecs<false, VPT>(dst, y, v, nt, hi);
        }
    }
}

// Element path for rows that are not a whole number of 16-byte vectors.
template <int DT>
__global__ __launch_bounds__(kWG) void k_combine_elem(Ptrs<64> p, const int64_t* __restrict__ off,
                                                      const int2* __restrict__ ent, const float* __restrict__ wts,
                                                      int P, int64_t rowelems, uint32_t T, Place pl) {
    using A = Arith<DT>;
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const uint32_t tok = static_cast<uint32_t>(item_at(pl, blockIdx.x, gridDim.x, i));
        const uint32_t src = tok / T;
        const int64_t obase = static_cast<int64_t>(tok - src * T) * rowelems;
        const int64_t e0 = off[tok];
        const int64_t e1 = off[tok + 1];
        for (int64_t h = threadIdx.x; h < rowelems; h += blockDim.x) {
            float acc = 0.0f;
            for (int64_t e = e0; e < e1; ++e) {
                const int2 q = ent[e];
                float v = A::load1(p.in[q.x], static_cast<int64_t>(q.y) * rowelems + h);
                if (wts) v = wts[static_cast<int64_t>(tok) * P + q.x] * v;
                acc = e == e0 ? v : acc + v;
            }
            A::store1(p.out[src], obase + h, acc);
        }
    }
}

// Column chunks per token: halve the chunks while the launch stays at or
// below 8192 work items and each chunk still gives every thread of a
// workgroup at least one vector.  At the 512-token, 8-rank, 7168-wide MoE
// shape this gives 2 chunks (8192 items of 448 vectors), measured on MI355X
// 6% faster than whole rows; more, smaller items lose to per-item overhead.
uint32_t pick_combine_chunks(int64_t ntok, int64_t rowvec, int nt) {
    // Work items are numbered in 32 bits: tokens * chunks stays below 2^32.
    const int forced = tuning().combine_chunks;
    if (forced >= 1 && forced <= rowvec && ntok * forced <= int64_t(UINT32_MAX))
        return static_cast<uint32_t>(forced);
    uint32_t c = 1;
    while (ntok * (2 * c) <= 8192 && rowvec / (2 * c) >= nt) c *= 2;
    return c;
}

template <int MAXP, int DT, bool WT>
void launch_combine_t(const void* const* y, void* const* out, int P, const int64_t* off, const int2* ent,
                      const float* w, const CombShape& s, const Place& pl, int64_t G, int nt, int vpt,
                      hipStream_t st) {
    Ptrs<MAXP> p = make_ptrs<MAXP>(y, out, P, P);
    const dim3 g(static_cast<unsigned>(G)), b(static_cast<unsigned>(nt));
    if (vpt == 4) hipLaunchKernelGGL((k_combine<MAXP, DT, 4, WT>), g, b, 0, st, p, off, ent, w, s, pl);
    else if (vpt == 1) hipLaunchKernelGGL((k_combine<MAXP, DT, 1, WT>), g, b, 0, st, p, off, ent, w, s, pl);
    else hipLaunchKernelGGL((k_combine<MAXP, DT, 2, WT>), g, b, 0, st, p, off, ent, w, s, pl);
}

template <int MAXP, int DT>
void launch_combine_w(const void* const* y, void* const* out, int P, const int64_t* off, const int2* ent,
                      const float* w, const CombShape& s, const Place& pl, int64_t G, int nt, int vpt,
                      hipStream_t st) {
    if (w) launch_combine_t<MAXP, DT, true>(y, out, P, off, ent, w, s, pl, G, nt, vpt, st);
    else launch_combine_t<MAXP, DT, false>(y, out, P, off, ent, w, s, pl, G, nt, vpt, st);
}

}  // namespace

hipError_t launch_all_to_all(const void* const* send, void* const* recv, int P, const void* desc, int64_t nitems,
                             const int64_t* xcd_start, size_t row_bytes, int esize, int mode, hipStream_t stream) {
    const bool vec = row_bytes % 16 == 0;
    const int64_t rowlen = static_cast<int64_t>(vec ? row_bytes / 16 : row_bytes / esize);
    Place pl{};
    pl.mode = mode;
    pl.gsize = 0;
    pl.gshift = -1;
    int64_t want = nitems;
    if (mode == kPlaceXcd) {
        int64_t longest = 0;
        for (int x = 0; x <= kNumXcd; ++x) pl.start[x] = xcd_start[x];
        for (int x = 0; x < kNumXcd; ++x)
            longest = xcd_start[x + 1] - xcd_start[x] > longest ? xcd_start[x + 1] - xcd_start[x] : longest;
        want = kNumXcd * longest;
    } else {
        pl.start[kNumXcd] = nitems;
    }
    const int64_t G = cap_grid(want);
    const int4* d = static_cast<const int4*>(desc);
    if (vec) {
        if (P <= 8) {
            Ptrs<8> p = make_ptrs<8>(send, recv, P, P);
            hipLaunchKernelGGL((k_all_to_all<8, 4>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, P, d,
                               rowlen, pl);
        } else {
            Ptrs<64> p = make_ptrs<64>(send, recv, P, P);
            hipLaunchKernelGGL((k_all_to_all<64, 4>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, P, d,
                               rowlen, pl);
        }
    } else {
        Ptrs<64> p = make_ptrs<64>(send, recv, P, P);
        if (esize == 4)
            hipLaunchKernelGGL((k_all_to_all_elem<4>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, d,
                               rowlen, pl);
        else
            hipLaunchKernelGGL((k_all_to_all_elem<2>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, d,
                               rowlen, pl);
    }
    return hipGetLastError();
}

hipError_t launch_combine(const void* const* y, void* const* out, int P, int T, const void* off, const void* ent,
                          const float* weights, size_t row_bytes, int dtype, int mode, hipStream_t stream) {
    const int64_t ntok = static_cast<int64_t>(P) * T;
    const int64_t* o = static_cast<const int64_t*>(off);
    const int2* e = static_cast<const int2*>(ent);
    if (row_bytes % 16 == 0) {
        CombShape s{};
        s.rowvec = static_cast<int64_t>(row_bytes / 16);
        s.T = static_cast<uint32_t>(T);
        s.P = P;
        const int forced = tuning().wg_threads;
        const int nt = forced == 64 || forced == 128 || forced == 256 ? forced : 256;
        const int fv = tuning().combine_vpt;
        const int vpt = fv == 1 || fv == 2 || fv == 4 ? fv : 2;
        s.chunks = pick_combine_chunks(ntok, s.rowvec, nt);
        s.cw = (s.rowvec + s.chunks - 1) / s.chunks;
        // A work item touches no data another item reads: groups of one.
        const Place pl = make_place_uniform(mode, ntok * s.chunks, 1);
        const int64_t G = cap_grid(place_grid(pl));
        if (P <= 8) {
            if (dtype == kDtF32) launch_combine_w<8, kDtF32>(y, out, P, o, e, weights, s, pl, G, nt, vpt, stream);
            else launch_combine_w<8, kDtBf16>(y, out, P, o, e, weights, s, pl, G, nt, vpt, stream);
        } else {
            if (dtype == kDtF32) launch_combine_w<64, kDtF32>(y, out, P, o, e, weights, s, pl, G, nt, vpt, stream);
            else launch_combine_w<64, kDtBf16>(y, out, P, o, e, weights, s, pl, G, nt, vpt, stream);
        }
    } else {
        const Place pl = make_place_uniform(mode, ntok, 1);
        const int64_t G = cap_grid(ntok);
        Ptrs<64> p = make_ptrs<64>(y, out, P, P);
        const int64_t esz = static_cast<int64_t>(dtype_size(dtype));
        const int64_t rowelems = static_cast<int64_t>(row_bytes) / esz;
        if (dtype == kDtF32)
            hipLaunchKernelGGL((k_combine_elem<kDtF32>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, o,
                               e, weights, P, rowelems, static_cast<uint32_t>(T), pl);
        else
            hipLaunchKernelGGL((k_combine_elem<kDtBf16>), dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, o,
                               e, weights, P, rowelems, static_cast<uint32_t>(T), pl);
    }
    return hipGetLastError();
}

}  // namespace nuna
