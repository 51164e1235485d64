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
//   k_route_count  one workgroup per source rank s (64 threads per 64
//                  tokens, up to 1024 per pass), 64 tokens per wave.  Each
//                  lane forms its token's destination mask; a wave ballot per
//                  destination d counts
//                  the wave's tokens sent to d, and a scan of those counts over
//                  the waves in LDS gives every token its rank among the
//                  tokens of s sent to d.  Each token's record lists its
//                  destinations in ascending order as (rank within s << 6) | d,
//                  padded with all ones; cnt[s][d] is the total.  (A first form,
//                  one wave per source walking 64 tokens at a time, took 21 us at
//                  512 tokens per rank on MI355X: one DRAM round trip per step.)
//   k_route_copy   one work item per (token (s, t), destination slot j),
//                  j < R: it copies the token's row to the j-th destination of
//                  its record (an empty slot does nothing).  The receive row of
//                  copy d is sum over s' < s of cnt[s'][d] plus the rank within
//                  s.  The R items of a token read the same row: they are the
//                  logical group of Sec. 4.2.1, and XCD placement runs them on
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
// R record words, so nothing needs clearing between calls.
#include "device_common.h"

namespace nuna {

// The library's scratch for the routed dispatch: one copy per GPU, kept until
// the process ends.  Host code must use the address from
// hipGetSymbolAddress (routed_scratch_address), never this name.
static __device__ __align__(256) unsigned char scratch[kRoutedScratchBytes];

namespace {

constexpr int kRouteCountThreads = 1024;  // most tokens of one source per pass: 16 waves of 64
constexpr int kRouteCountWaves = kRouteCountThreads / 64;

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
                                                                    int k, int E, int R, unsigned char* scr) {
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
    const int per = E / P;
    const uint64_t below = (uint64_t(1) << lane) - 1;
    if (tid < 64) carry[tid] = 0;
    int nbad = 0;  // this lane's invalid entries
    const int nw = static_cast<int>(blockDim.x) >> 6;
    for (int t0 = 0; t0 < T; t0 += static_cast<int>(blockDim.x)) {
        const int t = t0 + tid;
        uint64_t mask = 0;
        if (t < T) {
            const int32_t* row = topk + (static_cast<int64_t>(s) * T + t) * k;
            for (int j = 0; j < k; ++j) {
                const int e = row[j];
                if (e >= 0 && e < E)
                    mask |= uint64_t(1) << (e / per);
                else
                    ++nbad;
            }
        }
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
    for (int off = 32; off > 0; off >>= 1) nbad += __shfl_down(nbad, off);
    if (lane == 0) wave_bad[wave] = nbad;
    __syncthreads();
    if (tid == 0) {
        int total = 0;
        for (int w = 0; w < nw; ++w) total += wave_bad[w];
        bad[s] = total;
    }
}

constexpr int kRouteVpt = 4;  // 16-byte vectors per thread per column pass

template <int MAXP>
__global__ __launch_bounds__(kWG) void k_route_copy(Ptrs<MAXP> p, int P, int T, int R, int64_t rowvec, int64_t cap,
                                                    const unsigned char* scr, int64_t* rows_out, Place pl) {
    const int32_t* cnt = reinterpret_cast<const int32_t*>(scr);
    const int32_t* bad = cnt + P * P;
    const uint32_t* rec = reinterpret_cast<const uint32_t*>(bad + P);
    const int tid = threadIdx.x;
    if (blockIdx.x == 0 && tid <= P) {
        // Rows each rank receives (the caller compares them with its capacity)
        // and the count of invalid top-k entries.
        int64_t sum = 0;
        if (tid < P)
            for (int q = 0; q < P; ++q) sum += cnt[q * P + tid];
        else
            for (int q = 0; q < P; ++q) sum += bad[q];
        rows_out[tid] = sum;
    }
    const RankTable tab = load_rank_table(p, P);
    const ItemRange it = items_of(pl, blockIdx.x, gridDim.x);
    for (int64_t i = it.first; i < it.end; i += it.stride) {
        const int64_t item = item_at(pl, blockIdx.x, gridDim.x, i);
        const int64_t w = item / R;  // token (s, t) = w
        const uint32_t word = rec[item];
        if (word == ~0u) continue;   // the token has fewer destinations than R
        const int d = static_cast<int>(word & 63u);
        const int s = static_cast<int>(w / T);
        int64_t row = word >> 6;
        for (int q = 0; q < s; ++q) row += cnt[q * P + d];
        if (row >= cap) continue;    // beyond the caller's capacity: reported through rows_out
        const uint4* src = rank_in(tab, s) + (w - static_cast<int64_t>(s) * T) * rowvec;
        uint4* dst = rank_out(tab, d) + row * rowvec;
        // The group's other items read the same row: loads go through the caches.
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
}

}  // namespace

hipError_t routed_scratch_address(void** ptr) { return hipGetSymbolAddress(ptr, HIP_SYMBOL(scratch)); }

hipError_t launch_routed_dispatch(const void* const* send, void* const* recv, const int32_t* topk, int P, int T,
                                  int k, int E, int64_t rowvec, int64_t cap, void* scratch_ptr, int64_t* rows_out,
                                  int mode, hipStream_t stream) {
    const int R = k < P ? k : P;
    unsigned char* scr = static_cast<unsigned char*>(scratch_ptr);
    const int nt = T >= kRouteCountThreads ? kRouteCountThreads : (T < 64 ? 64 : (T + 63) / 64 * 64);
    hipLaunchKernelGGL(k_route_count, dim3(static_cast<unsigned>(P)), dim3(static_cast<unsigned>(nt)), 0, stream, topk,
                       P, T, k, E, R, scr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t ntok = static_cast<int64_t>(P) * T;
    const Place pl = make_place_uniform(mode, ntok, R);
    // One workgroup per item up to 2^20 workgroups unless the caller caps the
    // grid, as for the layout-driven dispatch.
    const int64_t want = place_grid(pl);
    const int64_t lim = grid_limit(int64_t(1) << 20);
    const int64_t G = want < 1 ? 1 : (want < lim ? want : lim);
    note_launch("k_route_count+k_route_copy", pl.mode == kPlaceXcd && !linear_map(pl, G) ? kMapXcdGroups : kMapLinear,
                R, G, kWG, kRouteVpt);
    const unsigned char* cs = static_cast<const unsigned char*>(scratch_ptr);
    if (P <= 8) {
        const Ptrs<8> p = make_ptrs<8>(send, recv, P, P);
        hipLaunchKernelGGL(k_route_copy<8>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, P, T, R, rowvec,
                           cap, cs, rows_out, pl);
    } else {
        const Ptrs<64> p = make_ptrs<64>(send, recv, P, P);
        hipLaunchKernelGGL(k_route_copy<64>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, P, T, R,
                           rowvec, cap, cs, rows_out, pl);
    }
    return hipGetLastError();
}

}  // namespace nuna
