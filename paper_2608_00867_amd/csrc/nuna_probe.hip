// nuna_probe.hip -- diagnostic kernels: the workgroup -> XCD dispatch probe,
// the memory load-latency probe and the reference streaming copy.
//
// Kept apart from the collective kernels: it measures the machine, it does
// not move collective data.
#include "device_common.h"

namespace nuna {
namespace {

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


// Load-latency probe.  One lane of the workgroup that runs on XCD `xcd`
// walks the blocks of a buffer in order; for each it first loads another
// 128-byte line of the block (so the block's address translation is warm),
// then times one load of the probed line with s_memtime around the load and
// its wait.  Vector loads (nt) go the way the collective kernels' loads go.
__global__ __launch_bounds__(64) void k_probe_latency(const unsigned char* buf, int64_t nblocks, int64_t stride,
                                                      int64_t line_off, int64_t warm_off, int xcd,
                                                      uint32_t* cycles) {
    uint32_t me;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(me));
    if ((me & 0xfu) != static_cast<uint32_t>(xcd) || threadIdx.x != 0 || (blockIdx.x >> 3) != 0) return;
    uint32_t sink = 0;
    for (int64_t i = 0; i < nblocks; ++i) {
        const unsigned char* blk = buf + i * stride;
        uint32_t v;
        if (warm_off >= 0) {
            const uint32_t* w = reinterpret_cast<const uint32_t*>(blk + warm_off);
            asm volatile("global_load_dword %0, %1, off nt\n s_waitcnt vmcnt(0)" : "=v"(v) : "v"(w) : "memory");
            sink += v;
        }
        const uint32_t* q = reinterpret_cast<const uint32_t*>(blk + line_off);
        uint64_t t0, t1;
        asm volatile(
            "s_waitcnt vmcnt(0) lgkmcnt(0)\n"
            "s_memtime %0\n"
            "s_waitcnt lgkmcnt(0)\n"
            "global_load_dword %2, %3, off nt\n"
            "s_waitcnt vmcnt(0)\n"
            "s_memtime %1\n"
            "s_waitcnt lgkmcnt(0)\n"
            : "=s"(t0), "=s"(t1), "=v"(v)
            : "v"(q)
            : "memory");
        sink += v;
        cycles[i] = static_cast<uint32_t>(t1 - t0) | (sink & 0u);
    }
}

// Per-compute-unit load-latency probe on XCD `xcd`.  Many one-wave workgroups
// are launched; those that land on `xcd` read the compute unit they run on
// (shader engine, array and CU fields of HW_ID), and the first workgroup on
// each compute unit claims it (claimed[hw cu], zeroed by the caller) and takes
// the next probe slot j (slot counter after the 256 claim words).  Slot j
// walks every block of the buffer with one lane, as k_probe_latency does, but
// on lines 2j (warm-up) and 2j + 1 (timed) of each block, so the compute units
// of one XCD never touch each other's lines and each timed load misses its
// XCD's L2.  cycles[j * nblocks + i] is slot j's latency for block i and
// cu_of[j] the HW_ID CU key (bits 8-15) of the compute unit in slot j.  Up to
// kProbeCuSlots slots; workgroups past them exit.
constexpr int kProbeCuSlots = 32;

__global__ __launch_bounds__(64) void k_probe_latency_cus(const unsigned char* buf, int64_t nblocks, int64_t stride,
                                                          int xcd, int32_t* claimed, uint32_t* cycles,
                                                          int32_t* cu_of) {
    uint32_t me, hw;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(me));
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
    if ((me & 0xfu) != static_cast<uint32_t>(xcd) || threadIdx.x != 0) return;
    const int key = static_cast<int>((hw >> 8) & 0xffu);
    if (atomicCAS(&claimed[key], 0, 1) != 0) return;
    const int j = atomicAdd(&claimed[256], 1);
    if (j >= kProbeCuSlots) return;
    cu_of[j] = key;
    const int64_t line = static_cast<int64_t>(2 * j + 1) * 128;
    const int64_t warm = static_cast<int64_t>(2 * j) * 128;
    uint32_t sink = 0;
    for (int64_t i = 0; i < nblocks; ++i) {
        const unsigned char* blk = buf + i * stride;
        uint32_t v;
        const uint32_t* w = reinterpret_cast<const uint32_t*>(blk + warm);
        asm volatile("global_load_dword %0, %1, off nt\n s_waitcnt vmcnt(0)" : "=v"(v) : "v"(w) : "memory");
        sink += v;
        const uint32_t* q = reinterpret_cast<const uint32_t*>(blk + line);
        uint64_t t0, t1;
        asm volatile(
            "s_waitcnt vmcnt(0) lgkmcnt(0)\n"
            "s_memtime %0\n"
            "s_waitcnt lgkmcnt(0)\n"
            "global_load_dword %2, %3, off nt\n"
            "s_waitcnt vmcnt(0)\n"
            "s_memtime %1\n"
            "s_waitcnt lgkmcnt(0)\n"
            : "=s"(t0), "=s"(t1), "=v"(v)
            : "v"(q)
            : "memory");
        sink += v;
        cycles[j * nblocks + i] = static_cast<uint32_t>(t1 - t0) | (sink & 0u);
    }
}

}  // namespace

hipError_t launch_probe_latency_cus(const void* buf, int64_t nblocks, int64_t stride, int xcd, int32_t* claimed,
                                    uint32_t* cycles, int32_t* cu_of, hipStream_t stream) {
    // 64 workgroups per XCD: the first to reach each of its compute units claims it.
    hipLaunchKernelGGL(k_probe_latency_cus, dim3(kNumXcd * 64), dim3(64), 0, stream,
                       static_cast<const unsigned char*>(buf), nblocks, stride, xcd, claimed, cycles, cu_of);
    return hipGetLastError();
}

hipError_t launch_probe_latency(const void* buf, int64_t nblocks, int64_t stride, int64_t line_off, int64_t warm_off,
                                int xcd, uint32_t* cycles, hipStream_t stream) {
    hipLaunchKernelGGL(k_probe_latency, dim3(kNumXcd), dim3(64), 0, stream, static_cast<const unsigned char*>(buf),
                       nblocks, stride, line_off, warm_off, xcd, cycles);
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
