// nuna_moe.hip -- gfx950 kernels of MoE expert parallelism: the all-to-all
// dispatch of token rows to the ranks of their experts, and the combine that
// sums the expert results back into each token's row.
//
// Row copies and row sums of 16-byte vectors; the dispatch is driven by a
// per-item descriptor list in placement order, the combine by per-token
// (rank, row) lists: fixed-size records with up to 8 ranks, offset lists
// beyond.  No MFMA: rows are moved and added, never contracted.
#include "device_common.h"

namespace nuna {
namespace {

// ---------------------------------------------------------------- all-to-all

// One descriptor per row copy, stored in placement order: source rank,
// source token, destination rank, destination row.
template <int MAXP, int UNROLL>
__global__ __launch_bounds__(kWG) void k_all_to_all(Ptrs<MAXP> p, int P, const int4* __restrict__ desc,
                                                    int64_t rowvec, Place pl) {
    // The dispatch always runs per-XCD item lists (Place gsize 0).
    const int nt = blockDim.x;
    const RankTable tab = load_rank_table(p, P);
    // The scalar arguments the item loop needs go into one empty statement, so
    // their loads issue together instead of one after another.  The list
    // bounds pass through it, so the range below uses these loads and no
    // others.  It is not volatile and takes no pointer: a pointer passed to
    // it would count as escaping, and the descriptor loads through it could
    // then no longer be scalar loads.
    const int x = static_cast<int>(blockIdx.x & (kNumXcd - 1));
    int64_t lo = pl.start[x], hi = pl.start[x + 1], total = pl.start[kNumXcd];
    asm("" : "+s"(lo), "+s"(hi), "+s"(total) : "s"(rowvec), "s"(pl.mode), "s"(blockDim.x), "s"(gridDim.x));
    const bool linear = pl.mode == kPlaceLinear || gridDim.x < kNumXcd;
    const ItemRange it = list_items(linear, lo, hi, total, blockIdx.x, gridDim.x);
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

// Adds one term of a token's sum into acc (first: the term starts the sum).
// WT: the term is first scaled by its fp32 weight (the product is rounded
// once; no fused multiply-add).
template <int DT, int VPT, bool WT>
__device__ __forceinline__ void combine_term(float (&acc)[VPT][Arith<DT>::kLanes], const uint4 (&x)[VPT], float wq,
                                             bool first) {
    using A = Arith<DT>;
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
        if constexpr (WT) {
            float t[A::kLanes];
            A::init(t, x[j]);
#pragma unroll
            for (int l = 0; l < A::kLanes; ++l) {
                const float term = wq * t[l];
                acc[j][l] = first ? term : acc[j][l] + term;
            }
        } else {
            if (first)
                A::init(acc[j], x[j]);
            else
                A::add(acc[j], x[j]);
        }
    }
}

// WT: each term is first scaled by the fp32 weight w[tok * P + rank].
template <int MAXP, int DT, int VPT, bool WT>
__global__ __launch_bounds__(kWG) void k_combine(Ptrs<MAXP> p, const int64_t* __restrict__ off,
                                                 const int2* __restrict__ ent, const float* __restrict__ wts,
                                                 CombShape s, int64_t items) {
    using A = Arith<DT>;
    constexpr int B = 8;  // result rows loaded per batch
    const int nt = blockDim.x;
    const RankTable tab = load_rank_table(p, s.P);
    // Work items are independent (no item reads what another reads), so both
    // placements run them in the linear order: item b, b + G, ...  The scalar
    // arguments go into one empty statement so that their loads issue
    // together; the values the loop uses pass through it.  As in the dispatch
    // it takes no pointer, so the offset and entry loads stay scalar loads.
    uint32_t chunks = s.chunks;
    asm("" : "+s"(items), "+s"(chunks) : "s"(s.rowvec), "s"(s.cw), "s"(s.T), "s"(s.P), "s"(blockDim.x),
        "s"(gridDim.x));
    for (int64_t i = blockIdx.x; i < items; i += gridDim.x) {
        const uint32_t w = static_cast<uint32_t>(i);
        const uint32_t tok = w / chunks;
        const int64_t lo = static_cast<int64_t>(w - tok * chunks) * s.cw;
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
                for (int q = 0; q < B; ++q)
                    if (q0 + q < c) combine_term<DT, VPT, WT>(acc, buf[q], WT ? wq[q] : 0.0f, q0 + q == 0);
            }
            uint4 y[VPT];
#pragma unroll
            for (int j = 0; j < VPT; ++j) y[j] = A::narrow(acc[j]);
            store_vecs<false, VPT>(dst, y, v, nt, hi);
        }
    }
}

// The combine for up to 8 ranks, from fixed-size per-token records: record
// tok is kCombRecRanks words, word q = (receive row << 3) | rank of the
// token's q-th entry (ranks ascending), all ones after the last.  Lane q of
// each wave loads word q and the wave reads the entries back with
// v_readlane, so a token's whole list arrives with one vector load and its
// result rows are requested after a single dependent load (the offset lists
// take two: offsets, then entries).  A uniform scalar load of the record
// measured slower on MI355X (4.9 against 4.2 us per call at 16 tokens per
// rank).  The gate weights are fetched the same way, lane r holding rank r's
// weight, in parallel with the record.  Every token has at least one entry
// (top-k is never empty).
// A work item's column chunk is at most blockDim.x * VPT vectors (the host
// sizes the chunks so), so each item is one pass: nothing is carried from one
// pass to the next, and the per-entry row addresses die once their loads are
// issued.
template <int DT, int VPT, bool WT>
__global__ __launch_bounds__(kWG) void k_combine_rec(Ptrs<kCombRecRanks> p, const uint32_t* __restrict__ rec,
                                                     const float* __restrict__ wts, CombShape s, int64_t items) {
    using A = Arith<DT>;
    constexpr uint32_t kNone = ~0u;
    const int nt = blockDim.x;
    const RankTable tab = load_rank_table(p, s.P);
    // Items in the linear order; the argument loads are batched as in k_combine.
    uint32_t chunks = s.chunks;
    asm("" : "+s"(items), "+s"(chunks) : "s"(s.rowvec), "s"(s.cw), "s"(s.T), "s"(s.P), "s"(blockDim.x),
        "s"(gridDim.x));
    const int q_lane = static_cast<int>(threadIdx.x & (kCombRecRanks - 1));
    for (int64_t i = blockIdx.x; i < items; i += gridDim.x) {
        const uint32_t w = static_cast<uint32_t>(i);
        const uint32_t tok = w / chunks;
        const uint32_t word = rec[static_cast<int64_t>(tok) * kCombRecRanks + q_lane];
        float w_lane = 0.0f;
        if constexpr (WT)
            if (q_lane < s.P) w_lane = wts[static_cast<int64_t>(tok) * s.P + q_lane];
        uint32_t e[kCombRecRanks];
#pragma unroll
        for (int q = 0; q < kCombRecRanks; ++q)
            e[q] = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(word), q));
        const int64_t lo = static_cast<int64_t>(w - tok * chunks) * s.cw;
        const int64_t hi = lo + s.cw < s.rowvec ? lo + s.cw : s.rowvec;
        const uint32_t src = tok / s.T;
        const uint32_t t = tok - src * s.T;
        const int64_t v = lo + threadIdx.x;
        uint4 buf[kCombRecRanks][VPT];
        float wq[kCombRecRanks];
#pragma unroll
        for (int q = 0; q < kCombRecRanks; ++q) {
            if (e[q] != kNone) {
                const int r = static_cast<int>(e[q] & 7u);
                const uint4* row = rank_in(tab, r) + static_cast<int64_t>(e[q] >> 3) * s.rowvec;
                load_vecs<false, VPT, true>(buf[q], row, v, nt, hi);
                if constexpr (WT) wq[q] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w_lane), r));
            }
        }
        // Every token has at least one destination (the layout requires top-k >= 1 and experts in
        // range) and its records are packed from word 0, so record 0 always starts the sum.
        float acc[VPT][A::kLanes];
#pragma unroll
        for (int q = 0; q < kCombRecRanks; ++q)
            if (e[q] != kNone) combine_term<DT, VPT, WT>(acc, buf[q], WT ? wq[q] : 0.0f, q == 0);
        uint4 y[VPT];
#pragma unroll
        for (int j = 0; j < VPT; ++j) y[j] = A::narrow(acc[j]);
        store_vecs<false, VPT>(rank_out(tab, static_cast<int>(src)) + static_cast<int64_t>(t) * s.rowvec, y, v, nt,
                               hi);
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

// rec (records, up to kCombRecRanks ranks) when not null, else the offset lists.
template <int MAXP, int DT, int VPT, bool WT>
void launch_combine_v(const Ptrs<MAXP>& p, const int64_t* off, const int2* ent, const uint32_t* rec, const float* w,
                      const CombShape& s, int64_t items, dim3 g, dim3 b, hipStream_t st) {
    if constexpr (MAXP == kCombRecRanks) {
        if (rec) {
            hipLaunchKernelGGL((k_combine_rec<DT, VPT, WT>), g, b, 0, st, p, rec, w, s, items);
            return;
        }
    }
    hipLaunchKernelGGL((k_combine<MAXP, DT, VPT, WT>), g, b, 0, st, p, off, ent, w, s, items);
}

template <int MAXP, int DT, bool WT>
void launch_combine_t(const void* const* y, void* const* out, int P, const int64_t* off, const int2* ent,
                      const uint32_t* rec, const float* w, const CombShape& s, int64_t items, int64_t G, int nt,
                      int vpt, hipStream_t st) {
    Ptrs<MAXP> p = make_ptrs<MAXP>(y, out, P, P);
    const dim3 g(static_cast<unsigned>(G)), b(static_cast<unsigned>(nt));
    if (vpt == 4) launch_combine_v<MAXP, DT, 4, WT>(p, off, ent, rec, w, s, items, g, b, st);
    else if (vpt == 1) launch_combine_v<MAXP, DT, 1, WT>(p, off, ent, rec, w, s, items, g, b, st);
    else launch_combine_v<MAXP, DT, 2, WT>(p, off, ent, rec, w, s, items, g, b, st);
}

template <int MAXP, int DT>
void launch_combine_w(const void* const* y, void* const* out, int P, const int64_t* off, const int2* ent,
                      const uint32_t* rec, const float* w, const CombShape& s, int64_t items, int64_t G, int nt,
                      int vpt, hipStream_t st) {
    if (w) launch_combine_t<MAXP, DT, true>(y, out, P, off, ent, rec, w, s, items, G, nt, vpt, st);
    else launch_combine_t<MAXP, DT, false>(y, out, P, off, ent, rec, w, s, items, G, nt, vpt, st);
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
    // One workgroup per list position up to 2^20 workgroups unless the caller
    // caps the grid: at 512 tokens per rank (21,680 positions, XCD placement)
    // that measured 1.8 % faster on MI355X than a persistent loop over 16384
    // workgroups (55.2 against 56.2 us, back-to-back cold calls).
    const int64_t G = want < grid_limit(int64_t(1) << 20) ? (want > 0 ? want : 1) : grid_limit(int64_t(1) << 20);
    const int4* d = static_cast<const int4*>(desc);
    // XCD mode runs the per-XCD lists of the planner (each token row's copies on one XCD).
    note_launch(vec ? "k_all_to_all" : "k_all_to_all_elem", mode == kPlaceXcd ? kMapXcdLists : kMapLinear, 0, G, kWG,
                vec ? 4 : 0);
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
                          const void* rec, const float* weights, size_t row_bytes, int dtype, int mode,
                          hipStream_t stream) {
    const int64_t ntok = static_cast<int64_t>(P) * T;
    const int64_t* o = static_cast<const int64_t*>(off);
    const int2* e = static_cast<const int2*>(ent);
    const uint32_t* rc =
        P <= kCombRecRanks && tuning().combine_lists == 0 ? static_cast<const uint32_t*>(rec) : nullptr;
    if (row_bytes % 16 == 0) {
        CombShape s{};
        s.rowvec = static_cast<int64_t>(row_bytes / 16);
        s.T = static_cast<uint32_t>(T);
        s.P = P;
        const int forced = tuning().wg_threads;
        const int nt = forced == 64 || forced == 128 || forced == 256 ? forced : 256;
        // Default vectors per thread: 1 with the records (measured on MI355X at
        // 16, 128 and 512 tokens per rank, 8 ranks, 7168-wide rows: equal or
        // faster, up to 11 % at 16 tokens), 2 with the offset lists.
        const int fv = tuning().combine_vpt;
        const int vpt = fv == 1 || fv == 2 || fv == 4 ? fv : rc ? 1 : 2;
        s.chunks = pick_combine_chunks(ntok, s.rowvec, nt);
        s.cw = (s.rowvec + s.chunks - 1) / s.chunks;
        if (rc && s.cw > static_cast<int64_t>(nt) * vpt) {
            // The record kernel covers a chunk in one pass: at most nt * vpt
            // vectors per chunk.  Work items are numbered in 32 bits.
            const int64_t need = (s.rowvec + static_cast<int64_t>(nt) * vpt - 1) / (static_cast<int64_t>(nt) * vpt);
            if (ntok * need <= int64_t(UINT32_MAX)) {
                s.chunks = static_cast<uint32_t>(need);
                s.cw = (s.rowvec + s.chunks - 1) / s.chunks;
            } else {
                rc = nullptr;
            }
        }
        // A work item touches no data another item reads: both placements run
        // the items in the linear order.
        const int64_t items = ntok * s.chunks;
        const int64_t G = cap_grid(items);
        note_launch(rc && P <= kCombRecRanks ? "k_combine_rec" : "k_combine", kMapLinear, 1, G, nt, vpt);
        if (P <= kCombRecRanks) {
            if (dtype == kDtF32)
                launch_combine_w<kCombRecRanks, kDtF32>(y, out, P, o, e, rc, weights, s, items, G, nt, vpt, stream);
            else
                launch_combine_w<kCombRecRanks, kDtBf16>(y, out, P, o, e, rc, weights, s, items, G, nt, vpt, stream);
        } else {
            if (dtype == kDtF32)
                launch_combine_w<64, kDtF32>(y, out, P, o, e, nullptr, weights, s, items, G, nt, vpt, stream);
            else
                launch_combine_w<64, kDtBf16>(y, out, P, o, e, nullptr, weights, s, items, G, nt, vpt, stream);
        }
    } else {
        const Place pl = make_place_uniform(mode, ntok, 1);
        const int64_t G = cap_grid(ntok);
        note_launch("k_combine_elem", kMapLinear, 1, G, kWG, 0);
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
