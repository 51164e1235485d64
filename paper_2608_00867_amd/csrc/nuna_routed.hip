// nuna_routed.hip -- MoE all-to-all dispatch with the routing on the device,
// working in a fixed static scratch array (no allocation at call time).
//
// The dispatch rule is the one of nuna_all_to_all (Sec. 2.1: all-to-all routes
// tokens to experts): expert e lives on rank e / (E / P); token t of rank s
// goes once to every distinct rank owning one of its top-k experts; rank d
// receives its rows ordered by source rank, then token.  Here the top-k table
// is device memory and the receive row of every copy is computed on the
// device:
//
//   k_route_small  decode sizes (at most 256 tokens over all ranks, at most
//                  2048 top-k entries): one launch, no tables.  Every
//                  workgroup loads the whole top-k table (thread i: token i,
//                  its k entries issued together), forms each token's
//                  destination mask, and takes its copy's receive row as the
//                  number of earlier tokens (source-major order) sent to the
//                  same rank, which each wave counts from the masks in LDS.
//                  The last workgroup also reports the rows per rank.  At 16
//                  tokens per rank (8 ranks, 7168 bf16, top-8 of 256) it takes
//                  4.9 us cold on MI355X, where the two launches below took
//                  9.8 us (the layout-driven dispatch: 3.3 us).  Every
//                  workgroup repeats the routing, so its cost is paid 1024
//                  times there: 4-byte loads of the entries instead of 16-byte
//                  ones cost 1.5 us, integer divisions 0.9 us.
//   k_route_count  one workgroup per source rank s (64 threads per 64
//                  tokens, up to 1024 per pass), 64 tokens per wave.  Each
//                  lane forms its token's destination mask (its k entries
//                  loaded together, as in k_route_small); a wave ballot per
//                  destination d counts the wave's
//                  tokens sent to d, and a scan of those counts over the waves
//                  in LDS gives every token its rank among the tokens of s
//                  sent to d.  Each token's record lists its destinations in
//                  ascending order as (rank within s << 6) | d, padded with
//                  all ones; cnt[s][d] is the total.  (A first form, one wave
//                  per source walking 64 tokens at a time, took 21 us at 512
//                  tokens per rank on MI355X: one DRAM round trip per step.)
//   k_route_copy   one work item per (token (s, t), destination slot j),
//                  j < R: it copies the token's row to the j-th destination of
//                  its record (an empty slot does nothing).  The receive row of
//                  copy d is sum over s' < s of cnt[s'][d] plus the rank within
//                  s; up to 8 ranks every lane holds one cnt entry, loaded
//                  beside the first record, and a wave sum adds the column
//                  (beyond, the lanes q < s load cnt[q][d] together).  The R
//                  items of a token read the same row: they are the logical
//                  group of Sec. 4.2.1, and XCD placement runs them on
//                  consecutive slots of one XCD (placement.h), so the row is
//                  fetched from HBM once and re-read from that XCD's L2, as the
//                  layout-driven dispatch does.  LINEAR runs the items in order.
//                  A first form with one workgroup per token, storing the row
//                  it had read to every destination, took 95 us at 512 tokens
//                  per rank on MI355X, against 55 us for the layout-driven
//                  dispatch with XCD placement.
//
// Scratch layout (device bytes from the start of the array):
//   cnt  int32 [P][P]           tokens of source s routed to d
//   bad  int32 [P]              top-k entries of source s outside [0, E)
//   rec  uint32 [P*T][R]        per-token destination records, R = min(k, P)
// cnt and bad are written whole by k_route_count, and every token writes its
// R record words, so nothing needs clearing between calls.  The decode path
// (k_route_small) uses no scratch.
#include "device_common.h"
#include "fastdiv.h"

namespace nuna {

// The library's scratch for the routed dispatch: one copy per GPU, kept until
// the process ends.  Host code must use the address from
// hipGetSymbolAddress (routed_scratch_address), never this name.
static __device__ __align__(256) unsigned char scratch[kRoutedScratchBytes];

namespace {

constexpr int kRouteCountThreads = 1024;  // most tokens of one source per pass: 16 waves of 64
constexpr int kRouteCountWaves = kRouteCountThreads / 64;
constexpr int kRouteBatch = 8;            // top-k entries (or counts) loaded per round
constexpr int kRouteSmallTokens = kWG;    // decode path: one token per thread
constexpr int kRouteSmallEntries = 2048;  // decode path: top-k entries every workgroup reads
constexpr int kRouteVpt = 4;              // 16-byte vectors per thread per column pass

// Destination mask of one token: bit d set when one of its k experts lives on
// rank d (expert e on rank e / per); entries outside [0, E) are counted in
// nbad.  The entries come in rounds of kRouteBatch, all loads of a round
// issued before the first is used.  With vec (k a multiple of 4 and the table
// 16-byte aligned) a round is two 16-byte loads per lane; otherwise eight
// 4-byte loads whose lanes lie k entries apart, four times the requests.
// Entries past k repeat loaded ones and are ignored; no branch depends on an
// entry.
__device__ __forceinline__ void load_round(const int32_t* __restrict__ row, int k, int j0, bool vec,
                                           int (&e)[kRouteBatch]) {
    if (vec) {
        const uint4* r4 = reinterpret_cast<const uint4*>(row + j0);
        const uint4 a = r4[0];
        const uint4 b = r4[j0 + 4 < k ? 1 : 0];
        e[0] = static_cast<int>(a.x), e[1] = static_cast<int>(a.y), e[2] = static_cast<int>(a.z);
        e[3] = static_cast<int>(a.w), e[4] = static_cast<int>(b.x), e[5] = static_cast<int>(b.y);
        e[6] = static_cast<int>(b.z), e[7] = static_cast<int>(b.w);
    } else {
#pragma unroll
        for (int u = 0; u < kRouteBatch; ++u) e[u] = row[j0 + u < k ? j0 + u : k - 1];
    }
}

__device__ __forceinline__ void fold_round(const int (&e)[kRouteBatch], int k, int j0, int E, const Magic& per,
                                           int& nbad, uint64_t& mask) {
#pragma unroll
    for (int u = 0; u < kRouteBatch; ++u) {
        const bool in = j0 + u < k;
        const bool ok = in && e[u] >= 0 && e[u] < E;
        nbad += in && !ok ? 1 : 0;
        const uint32_t d = udiv(ok ? static_cast<uint32_t>(e[u]) : 0u, per);
        mask |= ok ? uint64_t(1) << d : uint64_t(0);
    }
}

__device__ __forceinline__ uint64_t token_mask(const int32_t* __restrict__ row, int k, int E, const Magic& per,
                                               bool vec, int& nbad) {
    uint64_t mask = 0;
    for (int j0 = 0; j0 < k; j0 += kRouteBatch) {
        int e[kRouteBatch];
        load_round(row, k, j0, vec, e);
        fold_round(e, k, j0, E, per, nbad, mask);
    }
    return mask;
}

// Sum of the n ints at base[0], base[stride], ..., loads issued kRouteBatch at a time.
__device__ __forceinline__ int64_t strided_sum(const int32_t* base, int stride, int n) {
    int64_t sum = 0;
    for (int q0 = 0; q0 < n; q0 += kRouteBatch) {
        int v[kRouteBatch];
#pragma unroll
        for (int u = 0; u < kRouteBatch; ++u) v[u] = base[static_cast<int64_t>(q0 + u < n ? q0 + u : n - 1) * stride];
#pragma unroll
        for (int u = 0; u < kRouteBatch; ++u)
            if (q0 + u < n) sum += v[u];
    }
    return sum;
}

__device__ __forceinline__ int wave_sum(int v) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// One token row to one destination row: the R items of a token read the same
// row, so loads go through the caches; stores stream.
__device__ __forceinline__ void copy_row(const uint4* src, uint4* dst, int64_t rowvec, int tid) {
    for (int64_t v = tid; v < rowvec; v += int64_t(kWG) * kRouteVpt) {
        uint4 y[kRouteVpt];
#pragma unroll
        for (int u = 0; u < kRouteVpt; ++u)
            if (v + u * kWG < rowvec) y[u] = src[v + u * kWG];
#pragma unroll
        for (int u = 0; u < kRouteVpt; ++u)
            if (v + u * kWG < rowvec) store_stream(dst + v + u * kWG, y[u]);
    }
}

// Decode path: P*T <= kRouteSmallTokens tokens, one per thread.  Every
// workgroup forms all destination masks and keeps them in LDS, then runs its
// items: item (w, j) copies token w = s*T + t to the j-th rank d of its mask,
// at receive row = tokens w' < w (source-major, the receive order) whose mask
// holds d, which each wave counts from the masks in LDS.
template <int MAXP>
__global__ __launch_bounds__(kWG) void k_route_small(Ptrs<MAXP> p, const int32_t* __restrict__ topk, int P, int T,
                                                     int k, int E, int R, Magic per, Magic byR, Magic byT, int vec,
                                                     int64_t rowvec, int64_t cap, int64_t* rows_out, Place pl) {
    __shared__ uint64_t masks[kRouteSmallTokens];
    __shared__ int total[kWG / 64][64];      // reporter: per wave, tokens sent to d
    __shared__ int wave_bad[kWG / 64];
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int ntok = P * T;
    // The top-k entries are loaded first: the routing waits on them.  (Loading
    // the first item's row beside them, which does not depend on the routing,
    // was 0.3 us slower at 16 tokens per rank on MI355X.)
    const int32_t* my_row = topk + static_cast<int64_t>(tid) * k;
    int e0[kRouteBatch] = {};
    if (tid < ntok) load_round(my_row, k, 0, vec != 0, e0);
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    const RankTable tab = load_rank_table(p, P);
    int nbad = 0;
    uint64_t mask = 0;
    if (tid < ntok) {
        fold_round(e0, k, 0, E, per, nbad, mask);
        for (int j0 = kRouteBatch; j0 < k; j0 += kRouteBatch) {
            int e[kRouteBatch];
            load_round(my_row, k, j0, vec != 0, e);
            fold_round(e, k, j0, E, per, nbad, mask);
        }
    }
    masks[tid] = mask;
    // The last workgroup reports the totals: its item is the last slot of a
    // token, empty for most, so the extra work stays off the critical path.
    const bool reporter = blockIdx.x == gridDim.x - 1;
    if (reporter) {
        int mine = 0;  // lane d: tokens of this wave sent to d
        for (int d = 0; d < P; ++d) {
            const int c = __popcll(__ballot((mask >> d) & 1u));
            if (lane == d) mine = c;
        }
        total[wave][lane] = mine;
        nbad = wave_sum(nbad);
        if (lane == 0) wave_bad[wave] = nbad;
    }
    __syncthreads();
    if (reporter && tid <= P) {
        // Rows each rank receives (the caller compares them with its capacity)
        // and the count of invalid top-k entries.
        int64_t sum = 0;
        for (int w = 0; w < kWG / 64; ++w) sum += tid < P ? total[w][tid] : wave_bad[w];
        rows_out[tid] = sum;
    }
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const uint32_t item = static_cast<uint32_t>(item_at(pl, blockIdx.x, gridDim.x, i));  // < 256 * 64
        const int w = static_cast<int>(udiv(item, byR));
        const int j = static_cast<int>(item) - w * R;
        uint64_t m = masks[w];
        for (int q = 0; q < j; ++q) m &= m - 1;
        if (m == 0) continue;  // the token has fewer than j + 1 destinations
        const int d = __builtin_ctzll(m);
        // Every wave counts the earlier tokens itself, lane l looking at tokens l, l + 64, ...: no
        // barrier per item.
        int64_t row = 0;
#pragma unroll
        for (int q = 0; q < kRouteSmallTokens / 64; ++q) {
            const int x = lane + 64 * q;
            row += __popcll(__ballot(x < w && ((masks[x] >> d) & 1u)));
        }
        if (row >= cap) continue;  // beyond the caller's capacity: reported through rows_out
        const int s = static_cast<int>(udiv(static_cast<uint32_t>(w), byT));
        const uint4* src = rank_in(tab, s) + static_cast<int64_t>(w - s * T) * rowvec;
        uint4* dst = rank_out(tab, d) + row * rowvec;
        copy_row(src, dst, rowvec, tid);
    }
}

// One workgroup per source rank s, of 64 threads per 64 tokens up to 1024
// (a small launch keeps its scan and barriers short); each pass takes
// blockDim.x tokens, wave w the 64 from t0 + 64 w.  Every lane loads its
// token's k experts (one round of loads per pass), forms the token's
// destination mask, and a wave ballot per destination d gives the token's
// rank among the wave's tokens sent to d.
// The waves' counts go through LDS, where an exclusive scan per destination
// over the waves (and the passes before) gives each wave's offset; a second
// ballot pass then writes the records.  The rank of a token is the number of
// earlier tokens of s sent to d, whichever wave or pass counts them.
__global__ __launch_bounds__(kRouteCountThreads) void k_route_count(const int32_t* __restrict__ topk, int P, int T,
                                                                    int k, int E, int R, Magic per, int vec,
                                                                    unsigned char* scr) {
    int32_t* cnt = reinterpret_cast<int32_t*>(scr);
    int32_t* bad = cnt + P * P;
    uint32_t* rec = reinterpret_cast<uint32_t*>(bad + P);
    __shared__ int wave_cnt[kRouteCountWaves][64];  // tokens of wave w sent to d (this pass)
    __shared__ int offset[kRouteCountWaves][64];    // tokens of s sent to d before wave w's first token
    __shared__ int carry[64];                       // tokens of s sent to d in earlier passes
    __shared__ int wave_bad[kRouteCountWaves];
    const int s = blockIdx.x;
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const uint64_t below = (uint64_t(1) << lane) - 1;
    if (tid < 64) carry[tid] = 0;
    int nbad = 0;  // this lane's invalid entries
    const int nw = static_cast<int>(blockDim.x) >> 6;
    for (int t0 = 0; t0 < T; t0 += static_cast<int>(blockDim.x)) {
        const int t = t0 + tid;
        const uint64_t mask =
            t < T ? token_mask(topk + (static_cast<int64_t>(s) * T + t) * k, k, E, per, vec != 0, nbad) : 0;
        int mine = 0;  // lane d: tokens of this wave sent to d
        for (int d = 0; d < P; ++d) {
            const int c = __popcll(__ballot((mask >> d) & 1u));
            if (lane == d) mine = c;
        }
        if (lane < P) wave_cnt[wave][lane] = mine;
        __syncthreads();
        if (tid < P) {
            int run = carry[tid];
            for (int w = 0; w < nw; ++w) {
                offset[w][tid] = run;
                run += wave_cnt[w][tid];
            }
            carry[tid] = run;
        }
        __syncthreads();
        if (t < T) {
            uint32_t* my = rec + (static_cast<int64_t>(s) * T + t) * R;
            int j = 0;
            for (int d = 0; d < P; ++d) {
                const bool on = (mask >> d) & 1u;
                const uint64_t bal = __ballot(on);
                if (on) my[j++] = (static_cast<uint32_t>(offset[wave][d] + __popcll(bal & below)) << 6) |
                                  static_cast<uint32_t>(d);
            }
            // Lanes past T hold no token and are the wave's last: left out of the ballots, they change
            // no rank.
            for (; j < R; ++j) my[j] = ~0u;
        }
        __syncthreads();  // offset and carry are rewritten by the next pass
    }
    if (tid < P) cnt[s * P + tid] = carry[tid];
    nbad = wave_sum(nbad);
    if (lane == 0) wave_bad[wave] = nbad;
    __syncthreads();
    if (tid == 0) {
        int total = 0;
        for (int w = 0; w < nw; ++w) total += wave_bad[w];
        bad[s] = total;
    }
}

template <int MAXP>
__global__ __launch_bounds__(kWG) void k_route_copy(Ptrs<MAXP> p, int P, int T, int R, Magic byR, Magic byT,
                                                    int64_t rowvec, int64_t cap, const unsigned char* scr,
                                                    int64_t* rows_out, Place pl) {
    const int32_t* cnt = reinterpret_cast<const int32_t*>(scr);
    const int32_t* bad = cnt + P * P;
    const uint32_t* rec = reinterpret_cast<const uint32_t*>(bad + P);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // Up to 8 ranks, lane l holds cnt[l / P][l mod P] for the whole launch.
    const bool lane_table = P * P <= 64;
    const int held = lane_table && lane < P * P ? cnt[lane] : 0;
    const int held_s = lane_table ? lane / P : 0;
    const int held_d = lane_table ? lane - held_s * P : 0;
    if (blockIdx.x == 0 && tid <= P) {
        // Rows each rank receives (the caller compares them with its capacity)
        // and the count of invalid top-k entries.
        rows_out[tid] = tid < P ? strided_sum(cnt + tid, P, P) : strided_sum(bad, 1, P);
    }
    const RankTable tab = load_rank_table(p, P);
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const int64_t item = item_at(pl, blockIdx.x, gridDim.x, i);  // < 2^21: the records fit the scratch
        const uint32_t word = rec[item];
        if (word == ~0u) continue;   // the token has fewer destinations than R
        const int64_t w = udiv(static_cast<uint32_t>(item), byR);  // token (s, t) = w
        const int d = static_cast<int>(word & 63u);
        const int s = static_cast<int>(udiv(static_cast<uint32_t>(w), byT));
        int part;
        if (lane_table)
            part = lane < P * P && held_d == d && held_s < s ? held : 0;
        else
            part = lane < s ? cnt[lane * P + d] : 0;  // s < P <= 64
        const int64_t row = static_cast<int64_t>(word >> 6) + wave_sum(part);
        if (row >= cap) continue;    // beyond the caller's capacity: reported through rows_out
        copy_row(rank_in(tab, s) + (w - static_cast<int64_t>(s) * T) * rowvec, rank_out(tab, d) + row * rowvec, rowvec,
                 tid);
    }
}

}  // namespace

hipError_t routed_scratch_address(void** ptr) { return hipGetSymbolAddress(ptr, HIP_SYMBOL(scratch)); }

hipError_t launch_routed_dispatch(const void* const* send, void* const* recv, const int32_t* topk, int P, int T,
                                  int k, int E, int64_t rowvec, int64_t cap, void* scratch_ptr, int64_t* rows_out,
                                  int mode, hipStream_t stream) {
    const int R = k < P ? k : P;
    const int64_t ntok = static_cast<int64_t>(P) * T;
    const Place pl = make_place_uniform(mode, ntok, R);
    // One workgroup per item up to 2^20 workgroups unless the caller caps the
    // grid, as for the layout-driven dispatch.
    const int64_t want = place_grid(pl);
    const int64_t lim = grid_limit(int64_t(1) << 20);
    const int64_t G = want < 1 ? 1 : (want < lim ? want : lim);
    const int map = pl.mode == kPlaceXcd && !linear_map(pl, G) ? kMapXcdGroups : kMapLinear;
    const Magic per = make_magic(static_cast<uint32_t>(E / P));
    const Magic byR = make_magic(static_cast<uint32_t>(R));
    const Magic byT = make_magic(static_cast<uint32_t>(T > 0 ? T : 1));
    const int vec = (k % 4 == 0 && (reinterpret_cast<uintptr_t>(topk) & 15u) == 0) ? 1 : 0;
    if (ntok <= kRouteSmallTokens && ntok * k <= kRouteSmallEntries) {
        note_launch("k_route_small", map, R, G, kWG, kRouteVpt);
        if (P <= 8) {
            const Ptrs<8> p = make_ptrs<8>(send, recv, P, P);
            hipLaunchKernelGGL(k_route_small<8>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, topk, P, T,
                               k, E, R, per, byR, byT, vec, rowvec, cap, rows_out, pl);
        } else {
            const Ptrs<64> p = make_ptrs<64>(send, recv, P, P);
            hipLaunchKernelGGL(k_route_small<64>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, topk, P,
                               T, k, E, R, per, byR, byT, vec, rowvec, cap, rows_out, pl);
        }
        return hipGetLastError();
    }
    unsigned char* scr = static_cast<unsigned char*>(scratch_ptr);
    const int nt = T >= kRouteCountThreads ? kRouteCountThreads : (T < 64 ? 64 : (T + 63) / 64 * 64);
    hipLaunchKernelGGL(k_route_count, dim3(static_cast<unsigned>(P)), dim3(static_cast<unsigned>(nt)), 0, stream, topk,
                       P, T, k, E, R, per, vec, scr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    note_launch("k_route_count+k_route_copy", map, R, G, kWG, kRouteVpt);
    const unsigned char* cs = static_cast<const unsigned char*>(scratch_ptr);
    if (P <= 8) {
        const Ptrs<8> p = make_ptrs<8>(send, recv, P, P);
        hipLaunchKernelGGL(k_route_copy<8>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, P, T, R, byR,
                           byT, rowvec, cap, cs, rows_out, pl);
    } else {
        const Ptrs<64> p = make_ptrs<64>(send, recv, P, P);
        hipLaunchKernelGGL(k_route_copy<64>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, P, T, R, byR,
                           byT, rowvec, cap, cs, rows_out, pl);
    }
    return hipGetLastError();
}

}  // namespace nuna
