// nuna_probe.hip -- diagnostic kernels: memory load-latency probe.
//
// Kept apart from the collective kernels: it measures the machine, it does
// not move collective data.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "placement.h"

namespace nuna {
namespace {

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

}  // namespace

hipError_t launch_probe_latency(const void* buf, int64_t nblocks, int64_t stride, int64_t line_off, int64_t warm_off,
                                int xcd, uint32_t* cycles, hipStream_t stream) {
    hipLaunchKernelGGL(k_probe_latency, dim3(kNumXcd), dim3(64), 0, stream, static_cast<const unsigned char*>(buf),
                       nblocks, stride, line_off, warm_off, xcd, cycles);
    return hipGetLastError();
}

}  // namespace nuna
