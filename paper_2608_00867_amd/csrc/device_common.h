// device_common.h -- device helpers shared by the gfx950 kernel sources:
// bf16/fp32 numerics, 16-byte streaming and write-through loads and stores,
// the pauses between a fan-out's per-destination stores, the rank pointer
// table, the pinning of kernel arguments and the scalar selects of a run-time
// rank's pointer, and the launch-grid cap.
//
// Everything sits in an unnamed namespace: each kernel source gets its own
// copy and no symbol leaves the library.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"
#include "placement.h"

namespace nuna {
namespace {

constexpr int kWG = 256;  // 4 wavefronts of 64 lanes

// ---------------------------------------------------------------- numerics

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// fp32 -> bf16 round-to-nearest-even.  NaN keeps its sign and upper payload
// and is made quiet; overflow rounds to infinity.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

template <int DT>
struct Arith;

template <>
struct Arith<kDtF32> {
    static constexpr int kLanes = 4;
    static constexpr int kEsize = 4;
    __device__ static __forceinline__ void init(float (&a)[4], const uint4& v) {
        a[0] = __uint_as_float(v.x);
        a[1] = __uint_as_float(v.y);
        a[2] = __uint_as_float(v.z);
        a[3] = __uint_as_float(v.w);
    }
    __device__ static __forceinline__ void add(float (&a)[4], const uint4& v) {
        a[0] = a[0] + __uint_as_float(v.x);
        a[1] = a[1] + __uint_as_float(v.y);
        a[2] = a[2] + __uint_as_float(v.z);
        a[3] = a[3] + __uint_as_float(v.w);
    }
    __device__ static __forceinline__ uint4 narrow(const float (&a)[4]) {
        return make_uint4(__float_as_uint(a[0]), __float_as_uint(a[1]), __float_as_uint(a[2]),
                          __float_as_uint(a[3]));
    }
    __device__ static __forceinline__ float load1(const void* p, int64_t i) {
        return static_cast<const float*>(p)[i];
    }
    __device__ static __forceinline__ void store1(void* p, int64_t i, float v) { static_cast<float*>(p)[i] = v; }
};

template <>
struct Arith<kDtBf16> {
    static constexpr int kLanes = 8;
    static constexpr int kEsize = 2;
    __device__ static __forceinline__ void init(float (&a)[8], const uint4& v) {
        a[0] = bf16_lo(v.x);
        a[1] = bf16_hi(v.x);
        a[2] = bf16_lo(v.y);
        a[3] = bf16_hi(v.y);
        a[4] = bf16_lo(v.z);
        a[5] = bf16_hi(v.z);
        a[6] = bf16_lo(v.w);
        a[7] = bf16_hi(v.w);
    }
    __device__ static __forceinline__ void add(float (&a)[8], const uint4& v) {
        a[0] = a[0] + bf16_lo(v.x);
        a[1] = a[1] + bf16_hi(v.x);
        a[2] = a[2] + bf16_lo(v.y);
        a[3] = a[3] + bf16_hi(v.y);
        a[4] = a[4] + bf16_lo(v.z);
        a[5] = a[5] + bf16_hi(v.z);
        a[6] = a[6] + bf16_lo(v.w);
        a[7] = a[7] + bf16_hi(v.w);
    }
    __device__ static __forceinline__ uint4 narrow(const float (&a)[8]) {
        return make_uint4(f32_to_bf16(a[0]) | (f32_to_bf16(a[1]) << 16), f32_to_bf16(a[2]) | (f32_to_bf16(a[3]) << 16),
                          f32_to_bf16(a[4]) | (f32_to_bf16(a[5]) << 16), f32_to_bf16(a[6]) | (f32_to_bf16(a[7]) << 16));
    }
    __device__ static __forceinline__ float load1(const void* p, int64_t i) {
        return bf16_lo(static_cast<const uint16_t*>(p)[i]);
    }
    __device__ static __forceinline__ void store1(void* p, int64_t i, float v) {
        static_cast<uint16_t*>(p)[i] = static_cast<uint16_t>(f32_to_bf16(v));
    }
};

// ---------------------------------------------------------------- memory access

// Non-temporal (streaming) 16-byte accesses.  Stores: every output byte is
// written once and consumed by a later kernel, so the writes stream towards
// memory instead of piling up as dirty L2 lines that the end-of-kernel
// release must write back.  Loads: used where a work item is the only reader
// of its input chunk; work items that re-read a chunk shared by their group
// use ordinary cached loads so the re-reads hit L2.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void store_stream(uint4* p, const uint4& v) {
    const u32x4_t t = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(t, reinterpret_cast<u32x4_t*>(p));
}

template <bool NT>
__device__ __forceinline__ uint4 load16(const uint4* p) {
    if constexpr (NT) {
        const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
        return make_uint4(t.x, t.y, t.z, t.w);
    } else {
        return *p;
    }
}

// ---------------------------------------------------------------- kernel arguments

template <int MAXP>
struct Ptrs {
    const uint4* in[MAXP];
    uint4* out[MAXP];
};

template <int MAXP>
Ptrs<MAXP> make_ptrs(const void* const* in, void* const* out, int nin, int nout) {
    Ptrs<MAXP> p{};
    for (int r = 0; r < nin; ++r) p.in[r] = static_cast<const uint4*>(in[r]);
    for (int r = 0; r < nout; ++r) p.out[r] = static_cast<uint4*>(out[r]);
    return p;
}

// Direct kernels with 2, 4 or 8 ranks: one use of every rank pointer and of
// the given scalar arguments in a single statement, so that the kernel's
// first round of scalar loads brings all of them.  Without it the compiler
// loads a pointer where it is first used: a chain of argument loads behind
// the kernel's early tests, and a load and wait before a store to each
// output, each a round trip a short launch pays (0.12-0.15 us per call of
// the 8-rank one-shot at 16-256 KiB per rank on MI355X).
#define NUNA_PIN_PTRS8(p)                                                                                  \
    "s"(p.in[0]), "s"(p.in[1]), "s"(p.in[2]), "s"(p.in[3]), "s"(p.in[4]), "s"(p.in[5]), "s"(p.in[6]),         \
        "s"(p.in[7]), "s"(p.out[0]), "s"(p.out[1]), "s"(p.out[2]), "s"(p.out[3]), "s"(p.out[4]), "s"(p.out[5]), \
        "s"(p.out[6]), "s"(p.out[7])
#define NUNA_PIN_PTRS4(p) \
    "s"(p.in[0]), "s"(p.in[1]), "s"(p.in[2]), "s"(p.in[3]), "s"(p.out[0]), "s"(p.out[1]), "s"(p.out[2]), "s"(p.out[3])
#define NUNA_PIN_PTRS2(p) "s"(p.in[0]), "s"(p.in[1]), "s"(p.out[0]), "s"(p.out[1])

template <int PT, class A, class B, class C>
__device__ __forceinline__ void pin_args(const Ptrs<PT>& p, A a, B b, C c) {
    if constexpr (PT == 8)
        asm volatile("" ::NUNA_PIN_PTRS8(p), "s"(a), "s"(b), "s"(c));
    else if constexpr (PT == 4)
        asm volatile("" ::NUNA_PIN_PTRS4(p), "s"(a), "s"(b), "s"(c));
    else if constexpr (PT == 2)
        asm volatile("" ::NUNA_PIN_PTRS2(p), "s"(a), "s"(b), "s"(c));
    else
        asm volatile("" ::"s"(a), "s"(b), "s"(c));
}

template <int PT, class A, class B, class C, class D, class E, class F>
__device__ __forceinline__ void pin_args(const Ptrs<PT>& p, A a, B b, C c, D d, E e, F f) {
    if constexpr (PT == 8)
        asm volatile("" ::NUNA_PIN_PTRS8(p), "s"(a), "s"(b), "s"(c), "s"(d), "s"(e), "s"(f));
    else if constexpr (PT == 4)
        asm volatile("" ::NUNA_PIN_PTRS4(p), "s"(a), "s"(b), "s"(c), "s"(d), "s"(e), "s"(f));
    else if constexpr (PT == 2)
        asm volatile("" ::NUNA_PIN_PTRS2(p), "s"(a), "s"(b), "s"(c), "s"(d), "s"(e), "s"(f));
    else
        asm volatile("" ::"s"(a), "s"(b), "s"(c), "s"(d), "s"(e), "s"(f));
}

// Rank r's pointer for a uniform run-time r, chosen among the pointers
// already in SGPRs (a chain of scalar selects) instead of a scalar load from
// the argument segment.
template <int PT>
__device__ __forceinline__ const uint4* in_at(const Ptrs<PT>& p, int r) {
    const uint4* x = p.in[0];
#pragma unroll
    for (int q = 1; q < PT; ++q) x = r == q ? p.in[q] : x;
    return x;
}

template <int PT>
__device__ __forceinline__ uint4* out_at(const Ptrs<PT>& p, int r) {
    uint4* x = p.out[0];
#pragma unroll
    for (int q = 1; q < PT; ++q) x = r == q ? p.out[q] : x;
    return x;
}

// Rank pointer table.  With a handful of ranks the kernels index the
// kernel-argument pointer array with compile-time offsets, and the pointers
// arrive in SGPRs with the first scalar loads.  With many ranks, or a rank
// chosen at run time, each pointer would be a separate scalar load that the
// dependent vector load must wait for.  Instead every wave loads the table
// once, lane r holding rank r's input and output pointers (one vector load
// each), and v_readlane hands any rank's pointer to the wave as a uniform
// value with no memory round trip.  The table is loaded with all lanes
// active, at kernel start.
struct RankTable {
    uint32_t in_lo, in_hi, out_lo, out_hi;
};

template <int MAXP>
__device__ __forceinline__ RankTable load_rank_table(const Ptrs<MAXP>& p, int P) {
    const int lane = threadIdx.x & 63;
    RankTable t{0u, 0u, 0u, 0u};
    (void)P;  // entries past P are null pointers and never used
    if (lane < MAXP) {
        const uint64_t a = reinterpret_cast<uint64_t>(p.in[lane]);
        const uint64_t b = reinterpret_cast<uint64_t>(p.out[lane]);
        t.in_lo = static_cast<uint32_t>(a);
        t.in_hi = static_cast<uint32_t>(a >> 32);
        t.out_lo = static_cast<uint32_t>(b);
        t.out_hi = static_cast<uint32_t>(b >> 32);
    }
    return t;
}

// The table holds global-memory addresses.  A pointer rebuilt from an
// integer is a generic (flat) pointer, and flat instructions count in both
// the vector-memory and the scalar/LDS wait counters: a wait for a scalar
// load would then also wait for every flat load or store in flight.  The
// pointers are therefore formed in the global address space and converted to
// generic; the compiler carries the global space through to every access.
typedef __attribute__((address_space(1))) const uint4 global_cvec;
typedef __attribute__((address_space(1))) uint4 global_vec;

__device__ __forceinline__ const uint4* global_in(uint64_t addr) { return (const uint4*)((global_cvec*)addr); }
__device__ __forceinline__ uint4* global_out(uint64_t addr) { return (uint4*)((global_vec*)addr); }

__device__ __forceinline__ const uint4* rank_in(const RankTable& t, int r) {
    const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(t.in_lo), r));
    const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(t.in_hi), r));
    return global_in((hi << 32) | lo);
}

__device__ __forceinline__ uint4* rank_out(const RankTable& t, int r) {
    const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(t.out_lo), r));
    const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(t.out_hi), r));
    return global_out((hi << 32) | lo);
}

// Pointer access: compile-time offsets for up to 16 ranks, the table beyond.
template <int PT>
constexpr bool use_table() {
    return PT == 0 || PT > 16;
}

template <int PT, int MAXP>
__device__ __forceinline__ const uint4* in_ptr(const Ptrs<MAXP>& p, const RankTable& t, int r) {
    if constexpr (use_table<PT>())
        return rank_in(t, r);
    else
        return p.in[r];
}

template <int PT, int MAXP>
__device__ __forceinline__ uint4* out_ptr(const Ptrs<MAXP>& p, const RankTable& t, int r) {
    if constexpr (use_table<PT>())
        return rank_out(t, r);
    else
        return p.out[r];
}

// Ranks loaded per batch: all loads of a batch are issued before its adds.
// Compile-time rank counts load every rank at once; a run-time count goes in
// batches of 16.
template <int PT>
constexpr int rank_batch() {
    return PT == 0 ? 16 : PT;
}

// A thread's vectors within a chunk are v0 + j*nt, j < VPT, where nt is the
// workgroup size.  FULL: every index is in range (a uniform property of the
// chunk), so no per-lane guard is emitted.
template <bool FULL, int VPT, bool NT = false>
__device__ __forceinline__ void load_vecs(uint4 (&dst)[VPT], const uint4* src, int64_t v0, int nt, int64_t limit) {
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
        if (FULL || v0 + j * nt < limit)
            dst[j] = load16<NT>(src + v0 + j * nt);
        else
            dst[j] = make_uint4(0u, 0u, 0u, 0u);
    }
}

// Stores of one work item's chunk with the system-scope cache policy (sc0
// sc1): the lines are written through towards memory instead of staying as
// dirty lines in L2 and the Infinity Cache.  The accesses go through a buffer
// resource based at the chunk (`chunk`, uniform), so the lane offsets are
// chunk-relative bytes and the resource stays in scalar registers; the
// resource's size is the chunk's bytes, so the hardware drops any store past
// it.  In pass j the thread `lane` stores vector lane + j*nt of the chunk
// when that is below `limit` (chunk-relative).
constexpr int kCpolSystem = 17;  // sc0 | sc1 in the buffer-store cache-policy operand

template <bool FULL, int VPT>
__device__ __forceinline__ void store_vecs_wt(uint4* chunk, const uint4 (&y)[VPT], int lane, int nt, int64_t limit) {
    const int bytes = VPT * nt * 16;
    // Resource word 3: data format 32 (bits 15-18 = 4), no swizzle.
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(chunk, 0, bytes, 0x00020000);
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
        if (FULL || lane + j * nt < limit) {
            const u32x4_t t = {y[j].x, y[j].y, y[j].z, y[j].w};
            __builtin_amdgcn_raw_buffer_store_b128(t, r, (lane + j * nt) * 16, 0, kCpolSystem);
        }
    }
}

// Pause between the stores of consecutive destinations in a fan-out (one
// result stored to several outputs): `gap` (uniform) times s_nop 7, i.e. at
// least 8 * gap wait states of this wave.  Once its loads have landed, a
// wave would otherwise issue its P output stores back to back, and across
// the chip these store bursts cost HBM throughput on MI355X.  A plain
// 8-in/8-out kernel at 64 MiB per rank took 200 us with back-to-back stores
// and 179-182 us with any pause of 1-8 s_nop 7 or 1-3 s_sleep 1.  The
// library's one-shot went from 184-196 us to 181-182 us with one pause.
// Pauses cost latency on short launches (decode, 1 MiB per rank: 3.94 us
// with none, 4.09 with two, 4.45 with four), so the launchers pause only
// from 32 MiB per rank (store_gap_for).
__device__ __forceinline__ void store_gap(int gap) {
    for (int n = 0; n < gap; ++n) asm volatile("s_nop 7");
}

template <bool FULL, int VPT, bool NT = true>
__device__ __forceinline__ void store_vecs(uint4* dst, const uint4 (&y)[VPT], int64_t v0, int nt, int64_t limit) {
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
        if (FULL || v0 + j * nt < limit) {
            if constexpr (NT)
                store_stream(dst + v0 + j * nt, y[j]);
            else
                dst[v0 + j * nt] = y[j];
        }
    }
}

// acc[j] = sum over ranks r = 0, 1, ..., P-1 (in that order) of
// in[r][base + v0 + j*nt], for vectors below `limit` (relative to base).
// Lanes past the limit add zeros and are never stored.
template <int PT, int DT, int VPT, bool FULL, bool NT, int MAXP>
__device__ __forceinline__ void reduce_ranks(const Ptrs<MAXP>& p, const RankTable& tab, int P, int64_t base, int64_t v0,
                                             int nt, int64_t limit, float (&acc)[VPT][Arith<DT>::kLanes]) {
    using A = Arith<DT>;
    constexpr int B = rank_batch<PT>();
    if constexpr (PT > 0) {
#pragma unroll
        for (int r0 = 0; r0 < PT; r0 += B) {
            uint4 buf[B][VPT];
#pragma unroll
            for (int q = 0; q < B; ++q)
                load_vecs<FULL, VPT, NT>(buf[q], in_ptr<PT>(p, tab, r0 + q) + base, v0, nt, limit);
#pragma unroll
            for (int q = 0; q < B; ++q)
#pragma unroll
                for (int j = 0; j < VPT; ++j) {
                    if (r0 + q == 0)
                        A::init(acc[j], buf[q][j]);
                    else
                        A::add(acc[j], buf[q][j]);
                }
        }
    } else {
        // Runtime P: batches of B ranks; the last batch may be partial.
        for (int r0 = 0; r0 < P; r0 += B) {
            uint4 buf[B][VPT];
#pragma unroll
            for (int q = 0; q < B; ++q)
                if (r0 + q < P) load_vecs<FULL, VPT, NT>(buf[q], rank_in(tab, r0 + q) + base, v0, nt, limit);
#pragma unroll
            for (int q = 0; q < B; ++q)
                if (r0 + q < P) {
#pragma unroll
                    for (int j = 0; j < VPT; ++j) {
                        if (r0 + q == 0)
                            A::init(acc[j], buf[q][j]);
                        else
                            A::add(acc[j], buf[q][j]);
                    }
                }
        }
    }
}

// Split a work item into (group, member): shift when the group size is a
// power of two, divide otherwise.
__device__ __forceinline__ void split_item(int64_t w, int32_t gsize, int32_t gshift, int64_t& grp, int& member) {
    if (gshift >= 0) {
        grp = w >> gshift;
        member = static_cast<int>(w & ((int64_t(1) << gshift) - 1));
    } else {
        grp = w / gsize;
        member = static_cast<int>(w - grp * gsize);
    }
}

// Host: workgroups of a launch, at least 1 and at most the current cap.
inline int64_t cap_grid(int64_t wgs) {
    const int64_t cap = max_workgroups();
    return wgs < cap ? (wgs > 0 ? wgs : 1) : cap;
}

}  // namespace
}  // namespace nuna
