// nuna_probe.hip -- diagnostic kernels: the workgroup -> XCD dispatch probe,
// the memory load-latency probes, the reference streaming copy and the
// reference read / write / N-buffer copy streams.
//
// Kept apart from the collective kernels: it measures the machine, it does
// not move collective data.
#include "device_common.h"
#include "shapes.h"

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
// U vectors per thread per pass of a grid-stride loop.  From 32 MiB: U = 1,
// one 4 KiB item per workgroup (2^22 workgroups at most), which copied
// 128-512 MiB, cold, on MI355X at 6.3-6.5 TB/s against 6.1-6.2 TB/s for a
// persistent grid of 4096 workgroups with U = 4.  Below 32 MiB the persistent
// U = 4 grid was faster (16 MiB: 5.8 against 6.9 us) and runs.
template <int U>
__global__ __launch_bounds__(kWG) void k_copy(uint4* __restrict__ dst, const uint4* __restrict__ src, int64_t nvec,
                                              unsigned char* __restrict__ dst_tail,
                                              const unsigned char* __restrict__ src_tail, int tail) {
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


// Reference streams (nuna_ref_stream): the plain access patterns that bound
// the collectives' HBM rooflines.  Workgroup b handles vectors
// [256 b, 256 b + 256) of each of the N buffers, one per thread, as the
// collectives' one-vector items do; loads and stores are non-temporal.
constexpr uint32_t kRefTag = 0x52454631u;  // word 3 of every vector k_ref_write stores

// Reads: a work item is ref_read_blocks(N) consecutive 4 KiB blocks of every
// buffer, so that each thread has 8 loads in flight (16 with 16 buffers).
// The loads of a thread are XOR-folded, then across the workgroup in LDS: 16
// lanes fold 16 vectors each and lane 0 folds their 16 results; one 16-byte
// checksum per item is stored, so the loads cannot be dropped and the writes
// stay below 1/256 of the reads.  Both fold levels issue their 16 LDS reads
// together.  The fold lengthens a workgroup's life; with one load per thread
// in flight it cut the one-buffer read rate on MI355X to 3.8 TB/s (six
// dependent cross-lane shuffles) or 5.3 TB/s (this fold), against 6.9 TB/s
// for loads that feed no fold.
template <int N>
constexpr int ref_read_blocks() {
    return N >= 8 ? 1 : 8 / N;
}

template <int N>
__global__ __launch_bounds__(kWG) void k_ref_read(Ptrs<16> p, int64_t nvec) {
    constexpr int B = ref_read_blocks<N>();
    const int tid = static_cast<int>(threadIdx.x);
    const int64_t v0 = blockIdx.x * static_cast<int64_t>(kWG) * B + tid;
    uint4 x = make_uint4(0u, 0u, 0u, 0u);
    uint4 y[N][B];
#pragma unroll
    for (int r = 0; r < N; ++r)
#pragma unroll
        for (int j = 0; j < B; ++j)
            y[r][j] = v0 + j * kWG < nvec ? load16<true>(p.in[r] + v0 + j * kWG) : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int r = 0; r < N; ++r)
#pragma unroll
        for (int j = 0; j < B; ++j) {
            x.x ^= y[r][j].x;
            x.y ^= y[r][j].y;
            x.z ^= y[r][j].z;
            x.w ^= y[r][j].w;
        }
    __shared__ uint4 tile[kWG];
    tile[tid] = x;
    __syncthreads();
    if (tid < kWG / 16) {
        uint4 t[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) t[j] = tile[tid * 16 + j];
#pragma unroll
        for (int j = 1; j < 16; ++j) {
            t[0].x ^= t[j].x;
            t[0].y ^= t[j].y;
            t[0].z ^= t[j].z;
            t[0].w ^= t[j].w;
        }
        tile[tid * 16] = t[0];  // only this lane reads its segment
    }
    __syncthreads();
    if (tid == 0) {
        uint4 t[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) t[j] = tile[j * 16];
#pragma unroll
        for (int j = 1; j < 16; ++j) {
            t[0].x ^= t[j].x;
            t[0].y ^= t[j].y;
            t[0].z ^= t[j].z;
            t[0].w ^= t[j].w;
        }
        store_stream(p.out[0] + blockIdx.x, t[0]);
    }
}

// Writes: vector v of buffer r becomes {v mod 2^32, v div 2^32, r, kRefTag}.
template <int N>
__global__ __launch_bounds__(kWG) void k_ref_write(Ptrs<16> p, int64_t nvec, int32_t gap) {
    const int64_t v = blockIdx.x * static_cast<int64_t>(kWG) + threadIdx.x;
    if (v >= nvec) return;
#pragma unroll
    for (int r = 0; r < N; ++r) {
        if (r > 0) store_gap(gap);
        store_stream(p.out[r] + v, make_uint4(static_cast<uint32_t>(v), static_cast<uint32_t>(v >> 32),
                                              static_cast<uint32_t>(r), kRefTag));
    }
}

// N copies at once: out[r] = in[r], the N loads issued together, then the N
// stores (paced like the collectives' fan-out).
template <int N>
__global__ __launch_bounds__(kWG) void k_ref_copy(Ptrs<16> p, int64_t nvec, int32_t gap) {
    const int64_t v = blockIdx.x * static_cast<int64_t>(kWG) + threadIdx.x;
    if (v >= nvec) return;
    uint4 y[N];
#pragma unroll
    for (int r = 0; r < N; ++r) y[r] = load16<true>(p.in[r] + v);
#pragma unroll
    for (int r = 0; r < N; ++r) {
        if (r > 0) store_gap(gap);
        store_stream(p.out[r] + v, y[r]);
    }
}

template <int N>
void launch_ref_t(int kind, const Ptrs<16>& p, int64_t nvec, int64_t G, int gap, hipStream_t st) {
    if (kind == 0) {
        constexpr int64_t B = ref_read_blocks<N>();
        hipLaunchKernelGGL(k_ref_read<N>, dim3(static_cast<unsigned>((G + B - 1) / B)), dim3(kWG), 0, st, p, nvec);
    } else if (kind == 1)
        hipLaunchKernelGGL(k_ref_write<N>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, st, p, nvec, gap);
    else
        hipLaunchKernelGGL(k_ref_copy<N>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, st, p, nvec, gap);
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

hipError_t launch_ref_stream(int kind, const void* const* src, void* const* dst, int n, size_t bytes,
                             hipStream_t stream) {
    const int64_t nvec = static_cast<int64_t>(bytes / 16);
    const int64_t G = (nvec + kWG - 1) / kWG;
    const Ptrs<16> p = make_ptrs<16>(kind == 1 ? nullptr : src, dst, kind == 1 ? 0 : n, kind == 0 ? 1 : n);
    const int gap = store_gap_for(bytes * static_cast<size_t>(n));
    static const char* const names[3] = {"k_ref_read", "k_ref_write", "k_ref_copy"};
    const int64_t blocks = kind == 0 ? (n >= 8 ? 1 : 8 / n) : 1;  // 4 KiB blocks per item (ref_read_blocks)
    note_launch(names[kind], kMapLinear, 1, (G + blocks - 1) / blocks, kWG, static_cast<int>(blocks));
    switch (n) {
        case 1: launch_ref_t<1>(kind, p, nvec, G, gap, stream); break;
        case 2: launch_ref_t<2>(kind, p, nvec, G, gap, stream); break;
        case 4: launch_ref_t<4>(kind, p, nvec, G, gap, stream); break;
        case 8: launch_ref_t<8>(kind, p, nvec, G, gap, stream); break;
        case 16: launch_ref_t<16>(kind, p, nvec, G, gap, stream); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t stream) {
    const int64_t nvec = static_cast<int64_t>(bytes / 16);
    const int tail = static_cast<int>(bytes % 16);
    uint4* d = static_cast<uint4*>(dst);
    const uint4* s = static_cast<const uint4*>(src);
    unsigned char* dt = static_cast<unsigned char*>(dst) + nvec * 16;
    const unsigned char* st = static_cast<const unsigned char*>(src) + nvec * 16;
    if (bytes >= (size_t(32) << 20)) {
        int64_t G = (nvec + kWG - 1) / kWG;
        if (G > (int64_t(1) << 22)) G = int64_t(1) << 22;
        hipLaunchKernelGGL(k_copy<1>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, d, s, nvec, dt, st, tail);
    } else {
        int64_t G = (nvec + kWG * 4 - 1) / (kWG * 4);
        if (G > 4096) G = 4096;
        if (G < 1) G = 1;
        hipLaunchKernelGGL(k_copy<4>, dim3(static_cast<unsigned>(G)), dim3(kWG), 0, stream, d, s, nvec, dt, st, tail);
    }
    return hipGetLastError();
}

}  // namespace nuna
