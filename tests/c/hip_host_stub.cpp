// hip_host_stub.cpp -- host-only stand-in for the HIP runtime and the kernel
// launchers, so that libnuna's host code (argument checks, launch choice, the
// all-to-all layout builder, the placement planner, the tunables) can be built
// with AddressSanitizer and UndefinedBehaviorSanitizer and run on a machine
// without a GPU.
//
// "Device" memory here is host memory: hipMalloc is malloc.  The launch stubs
// never touch the collectives' data buffers (their pointers may be made up);
// they read the tables the host code built for the kernels (all-to-all
// descriptors, combine offsets, entries and records) end to end, so a table
// shorter than the launch believes is an out-of-bounds read the sanitizer
// reports, and they check every entry against the sizes the launch was given.
// The dispatch probe writes the MI355X map (workgroup b on XCD b mod 8), so
// nuna_init verifies it and XCD-mode calls reach their launchers.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "kernels.h"

namespace {

int g_fail = 0;

void check(bool ok, const char* what) {
    if (!ok) {
        std::fprintf(stderr, "launch stub: %s\n", what);
        ++g_fail;
    }
}

}  // namespace

extern "C" int stub_failures(void) { return g_fail; }

// ---------------------------------------------------------------- runtime

extern "C" {

hipError_t hipGetDeviceCount(int* n) {
    *n = 1;
    return hipSuccess;
}

hipError_t hipGetDevice(int* d) {
    *d = 0;
    return hipSuccess;
}

hipError_t hipGetDevicePropertiesR0600(hipDeviceProp_t* prop, int) {
    std::memset(prop, 0, sizeof *prop);
    std::snprintf(prop->gcnArchName, sizeof prop->gcnArchName, "gfx950:sramecc+:xnack-");
    prop->multiProcessorCount = 256;
    return hipSuccess;
}

hipError_t hipMalloc(void** p, size_t n) {
    *p = std::malloc(n ? n : 1);
    return *p ? hipSuccess : hipErrorOutOfMemory;
}

hipError_t hipFree(void* p) {
    std::free(p);
    return hipSuccess;
}

hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind) {
    std::memcpy(dst, src, n);
    return hipSuccess;
}

const char* hipGetErrorString(hipError_t) { return "stub error"; }

}  // extern "C"

// ---------------------------------------------------------------- launchers

namespace nuna {

hipError_t launch_allreduce(const void* const* in, void* const* out, int P, size_t count, int dtype, int dest_groups,
                            int mode, hipStream_t) {
    check(in && out && P >= 1 && P <= 64 && count > 0, "allreduce arguments");
    check(dtype == kDtF32 || dtype == kDtBf16, "allreduce dtype");
    check(dest_groups >= 1 && P % dest_groups == 0, "allreduce destination groups");
    check(mode == 0 || mode == 1, "allreduce mode");
    for (int r = 0; r < P; ++r) check(in[r] && out[r], "allreduce rank pointer");
    note_launch("stub_allreduce", kMapLinear, 1, 1, 256, 1);
    return hipSuccess;
}

bool two_shot_fused_ok(int P, size_t count, int dtype) {
    if (P != 2 && P != 4 && P != 8 && P != 16) return false;
    if (count % static_cast<size_t>(P) != 0) return false;
    return ((count / P) * dtype_size(dtype)) % 16 == 0;
}

bool two_shot_runs_fused(int P, size_t count, int dtype) { return two_shot_fused_ok(P, count, dtype); }

hipError_t launch_two_shot_fused(const void* const* in, void* const* out, int P, size_t count, int dtype, int,
                                 hipStream_t) {
    check(two_shot_fused_ok(P, count, dtype), "fused two-shot launched where it does not apply");
    for (int r = 0; r < P; ++r) check(in[r] && out[r], "two-shot rank pointer");
    note_launch("stub_two_shot", kMapLinear, 1, 1, 256, 1);
    return hipSuccess;
}

hipError_t launch_reduce_scatter(const void* const* in, void* const* out, int P, size_t m, int dtype, int mode,
                                 bool, hipStream_t) {
    check(in && out && P >= 1 && P <= 64 && m > 0 && (dtype == 0 || dtype == 1) && (mode == 0 || mode == 1),
          "reduce-scatter arguments");
    for (int r = 0; r < P; ++r) check(in[r] && out[r], "reduce-scatter rank pointer");
    note_launch("stub_reduce_scatter", kMapLinear, 1, 1, 256, 1);
    return hipSuccess;
}

hipError_t launch_all_gather(const void* const* in, void* const* out, int P, size_t m, int dtype, int mode, bool,
                             hipStream_t) {
    check(in && out && P >= 1 && P <= 64 && m > 0 && (dtype == 0 || dtype == 1) && (mode == 0 || mode == 1),
          "all-gather arguments");
    for (int r = 0; r < P; ++r) check(in[r] && out[r], "all-gather rank pointer");
    note_launch("stub_all_gather", kMapLinear, 1, 1, 256, 1);
    return hipSuccess;
}

hipError_t launch_all_to_all(const void* const* send, void* const* recv, int P, const void* desc, int64_t nitems,
                             const int64_t* xcd_start, size_t row_bytes, int esize, int mode, hipStream_t) {
    check(send && recv && desc && nitems > 0 && row_bytes > 0 && (esize == 2 || esize == 4), "a2a arguments");
    // Every descriptor (src rank, src token, dst rank, dst row), read end to end.
    const int32_t* d = static_cast<const int32_t*>(desc);
    for (int64_t i = 0; i < nitems; ++i) {
        check(d[4 * i] >= 0 && d[4 * i] < P && d[4 * i + 1] >= 0 && d[4 * i + 2] >= 0 && d[4 * i + 2] < P &&
                  d[4 * i + 3] >= 0,
              "a2a descriptor out of range");
    }
    check(xcd_start[0] == 0 && xcd_start[8] == nitems, "a2a per-XCD list bounds");
    for (int x = 0; x < 8; ++x) check(xcd_start[x] <= xcd_start[x + 1], "a2a per-XCD lists out of order");
    note_launch("stub_all_to_all", mode == 1 ? kMapXcdLists : kMapLinear, 0, nitems, 256, 4);
    return hipSuccess;
}

hipError_t launch_combine(const void* const* y, void* const* out, int P, int T, const void* off, const void* ent,
                          const void* rec, const float*, size_t row_bytes, int dtype, int, hipStream_t) {
    check(y && out && off && ent && P >= 1 && T >= 0 && row_bytes > 0 && (dtype == 0 || dtype == 1),
          "combine arguments");
    const int64_t ntok = static_cast<int64_t>(P) * T;
    const int64_t* o = static_cast<const int64_t*>(off);
    const int32_t* e = static_cast<const int32_t*>(ent);
    check(o[0] == 0, "combine offsets start");
    for (int64_t i = 0; i < ntok; ++i) {
        check(o[i + 1] >= o[i] && o[i + 1] - o[i] <= P, "combine offsets");
        for (int64_t j = o[i]; j < o[i + 1]; ++j)
            check(e[2 * j] >= 0 && e[2 * j] < P && e[2 * j + 1] >= 0, "combine entry out of range");
    }
    if (rec) {
        const uint32_t* r = static_cast<const uint32_t*>(rec);
        for (int64_t i = 0; i < ntok * kCombRecRanks; ++i)
            check(r[i] == ~uint32_t(0) || static_cast<int>(r[i] & 7u) < P, "combine record out of range");
    }
    note_launch("stub_combine", kMapLinear, 1, ntok, 256, 1);
    return hipSuccess;
}

hipError_t launch_probe_xcc(int G, int32_t* xcc, int32_t* hw_id, hipStream_t) {
    for (int b = 0; b < G; ++b) {
        xcc[b] = b % 8;
        if (hw_id) hw_id[b] = 0;
    }
    return hipSuccess;
}

hipError_t routed_scratch_address(void** ptr) {
    static unsigned char* scr = static_cast<unsigned char*>(std::malloc(kRoutedScratchBytes));
    *ptr = scr;
    return scr ? hipSuccess : hipErrorOutOfMemory;
}

hipError_t launch_routed_dispatch(const void* const* send, void* const* recv, const int32_t* topk, int P, int T, int k,
                                  int E, int64_t rowvec, int64_t cap, void* scratch_ptr, int64_t*, int mode, hipStream_t) {
    check(mode == 0 || mode == 1, "routed dispatch placement mode");
    check(send && recv && P >= 1 && P <= 64 && T >= 0 && k >= 1 && E % P == 0 && rowvec > 0 && cap >= 0,
          "routed dispatch arguments");
    check(scratch_ptr != nullptr && routed_scratch_need(P, T, k) <= kRoutedScratchBytes, "routed dispatch scratch");
    // The routing tables cover the whole scratch need: touch its last byte.
    if (T > 0) {
        check(topk != nullptr, "routed dispatch top-k");
        static_cast<unsigned char*>(scratch_ptr)[routed_scratch_need(P, T, k) - 1] = 0;
    }
    note_launch("stub_routed", kMapLinear, 1, static_cast<int64_t>(P) * T, 256, 4);
    return hipSuccess;
}

hipError_t launch_copy(void*, const void*, size_t, hipStream_t) { return hipSuccess; }

hipError_t launch_ref_stream(int kind, const void* const* src, void* const* dst, int n, size_t bytes, hipStream_t) {
    check(kind >= 0 && kind <= 2 && (n == 1 || n == 2 || n == 4 || n == 8 || n == 16) && bytes % 16 == 0 && bytes > 0,
          "reference stream arguments");
    for (int r = 0; r < n; ++r) {
        if (kind != 1) check(src[r] != nullptr, "reference stream source");
        if (kind != 0 || r == 0) check(dst[r] != nullptr, "reference stream destination");
    }
    return hipSuccess;
}

hipError_t launch_probe_latency_cus(const void*, int64_t nblocks, int64_t stride, int xcd, int32_t* claimed,
                                    uint32_t*, int32_t*, hipStream_t) {
    check(nblocks > 0 && stride >= 2 * kProbeCuSlotsMax * 128 && xcd >= 0 && xcd < 8 && claimed,
          "per-CU probe arguments");
    return hipSuccess;
}

hipError_t launch_probe_latency(const void*, int64_t nblocks, int64_t stride, int64_t line_off, int64_t, int xcd,
                                uint32_t*, hipStream_t) {
    check(nblocks > 0 && line_off + 4 <= stride && xcd >= 0 && xcd < 8, "latency probe arguments");
    return hipSuccess;
}

}  // namespace nuna
