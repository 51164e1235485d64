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
//   k_route_count  one wave per source rank s.  Walking its tokens 64 at a
//                  time, each lane forms its token's destination mask; for
//                  each destination d a wave ballot of the mask bit gives the
//                  token's rank among the tokens of s sent to d so far.  Each
//                  token's record lists its destinations in ascending order as
//                  (rank within s << 6) | d, padded with all ones; lane d
//                  finally stores cnt[s][d], the tokens of s sent to d.
//   k_route_copy   one workgroup per token (s, t).  The receive row of copy d
//                  is sum over s' < s of cnt[s'][d] plus the rank within s.
//                  The source row is read once into registers and stored to
//                  every destination row, column pass by column pass, so the
//                  copies of a token row (the logical group of Sec. 4.2.1)
//                  share one read and no L2 re-read is needed.
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

__global__ __launch_bounds__(64) void k_route_count(const int32_t* __restrict__ topk, int P, int T, int k, int E,
                                                    int R, unsigned char* scr) {
    int32_t* cnt = reinterpret_cast<int32_t*>(scr);
    int32_t* bad = cnt + P * P;
    uint32_t* rec = reinterpret_cast<uint32_t*>(bad + P);
    const int s = blockIdx.x;
    const int lane = threadIdx.x;
    const int per = E / P;
    const uint64_t below = (uint64_t(1) << lane) - 1;
    int run = 0;   // lane d: tokens of s routed to d so far
    int nbad = 0;  // this lane's invalid entries
    for (int t0 = 0; t0 < T; t0 += 64) {
        const int t = t0 + lane;
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
        uint32_t* my = rec + (static_cast<int64_t>(s) * T + t) * R;
        int j = 0;
        for (int d = 0; d < P; ++d) {
            const bool on = (mask >> d) & 1u;
            const uint64_t bal = __ballot(on);
            const int before = __builtin_amdgcn_readlane(run, d);
            if (on) my[j++] = (static_cast<uint32_t>(before + __popcll(bal & below)) << 6) | static_cast<uint32_t>(d);
            if (lane == d) run += __popcll(bal);
        }
        if (t < T)
            for (; j < R; ++j) my[j] = ~0u;
    }
    if (lane < P) cnt[s * P + lane] = run;
    for (int off = 32; off > 0; off >>= 1) nbad += __shfl_down(nbad, off);
    if (lane == 0) bad[s] = nbad;
}

constexpr int kRouteVpt = 4;  // 16-byte vectors per thread per column pass

__global__ __launch_bounds__(kWG) void k_route_copy(Ptrs<64> p, int P, int T, int R, int64_t rowvec, int64_t cap,
                                                    const unsigned char* scr, int64_t* rows_out) {
    const int32_t* cnt = reinterpret_cast<const int32_t*>(scr);
    const int32_t* bad = cnt + P * P;
    const uint32_t* rec = reinterpret_cast<const uint32_t*>(bad + P);
    __shared__ int64_t s_row[64];
    __shared__ int s_dst[64];
    const int tid = threadIdx.x;
    const int64_t w = blockIdx.x;
    const int64_t ntok = static_cast<int64_t>(P) * T;
    if (w == 0 && tid <= P) {
        // Rows each rank receives (the caller compares them with its capacity)
        // and the count of invalid top-k entries.
        int64_t sum = 0;
        if (tid < P)
            for (int q = 0; q < P; ++q) sum += cnt[q * P + tid];
        else
            for (int q = 0; q < P; ++q) sum += bad[q];
        rows_out[tid] = sum;
    }
    if (w >= ntok) return;
    const int s = static_cast<int>(w / T);
    const RankTable tab = load_rank_table(p, P);
    if (tid < R) {
        const uint32_t word = rec[w * R + tid];
        int d = -1;
        int64_t row = 0;
        if (word != ~0u) {
            d = static_cast<int>(word & 63u);
            row = word >> 6;
            for (int q = 0; q < s; ++q) row += cnt[q * P + d];
        }
        s_dst[tid] = d;
        s_row[tid] = row;
    }
    __syncthreads();
    const uint4* src = rank_in(tab, s) + static_cast<int64_t>(w - static_cast<int64_t>(s) * T) * rowvec;
    for (int64_t c0 = 0; c0 < rowvec; c0 += int64_t(kWG) * kRouteVpt) {
        uint4 y[kRouteVpt];
#pragma unroll
        for (int u = 0; u < kRouteVpt; ++u) {
            const int64_t v = c0 + u * kWG + tid;
            if (v < rowvec) y[u] = load16<true>(src + v);
        }
        for (int j = 0; j < R; ++j) {
            const int d = __builtin_amdgcn_readfirstlane(s_dst[j]);
            if (d < 0) break;
            const int64_t row = s_row[j];
            if (row >= cap) continue;  // beyond the caller's capacity: reported through rows_out
            uint4* dst = rank_out(tab, d) + row * rowvec;
#pragma unroll
            for (int u = 0; u < kRouteVpt; ++u) {
                const int64_t v = c0 + u * kWG + tid;
                if (v < rowvec) store_stream(dst + v, y[u]);
            }
        }
    }
}

}  // namespace

hipError_t routed_scratch_address(void** ptr) { return hipGetSymbolAddress(ptr, HIP_SYMBOL(scratch)); }

hipError_t launch_routed_dispatch(const void* const* send, void* const* recv, const int32_t* topk, int P, int T,
                                  int k, int E, int64_t rowvec, int64_t cap, void* scratch_ptr, int64_t* rows_out,
                                  hipStream_t stream) {
    const int R = k < P ? k : P;
    unsigned char* scr = static_cast<unsigned char*>(scratch_ptr);
    hipLaunchKernelGGL(k_route_count, dim3(static_cast<unsigned>(P)), dim3(64), 0, stream, topk, P, T, k, E, R, scr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    Ptrs<64> p = make_ptrs<64>(send, recv, P, P);
    const int64_t ntok = static_cast<int64_t>(P) * T;
    const int64_t G = ntok > 0 ? ntok : 1;
    note_launch("k_route_count+k_route_copy", kMapLinear, 1, G, kWG, kRouteVpt);
    hipLaunchKernelGGL(k_route_copy, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, p, P, T, R, rowvec, cap,
                       static_cast<const unsigned char*>(scratch_ptr), rows_out);
    return hipGetLastError();
}

}  // namespace nuna
