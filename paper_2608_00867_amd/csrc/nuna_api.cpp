// nuna_api.cpp -- host side of libnuna: argument validation, algorithm and
// launch-shape choice, the all-to-all routing planner, and the C ABI.
//
// Every argument check runs before the first HIP call, so invalid calls are
// rejected identically on machines without a GPU.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <exception>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "kernels.h"
#include "nap_planner.h"
#include "nuna.h"
#include "placement.h"

namespace {

thread_local std::string t_err;

nuna_status_t fail(nuna_status_t st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_err = buf;
    return st;
}

nuna_status_t ok() {
    t_err.clear();
    return NUNA_OK;
}

// Called from a catch handler: turns the exception in flight into a status,
// so that no exception crosses the C ABI.
nuna_status_t host_exception() {
    try {
        throw;
    } catch (const std::bad_alloc&) {
        return fail(NUNA_ERR_NO_MEMORY, "host memory allocation failed");
    } catch (const std::exception& e) {
        return fail(NUNA_ERR_INVALID_ARG, "host exception: %s", e.what());
    } catch (...) {
        return fail(NUNA_ERR_INVALID_ARG, "unknown host exception");
    }
}

nuna_status_t hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(NUNA_ERR_HIP, "%s: HIP error %d (%s)", what, static_cast<int>(e), hipGetErrorString(e));
}

// Largest byte count a single rank buffer may have (2^48 B keeps every
// index computation far from int64 overflow).
constexpr size_t kMaxBytes = size_t(1) << 48;
// Reference streams: one 4 KiB item per workgroup, and a grid of at most 2^22
// workgroups.
constexpr size_t kRefMaxBytes = size_t(1) << 34;

bool valid_dtype(int dt) { return dt == NUNA_F32 || dt == NUNA_BF16; }
bool valid_place(int p) { return p == NUNA_PLACE_LINEAR || p == NUNA_PLACE_XCD; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Span {
    uintptr_t lo, hi;  // [lo, hi)
    int rank;
};

bool spans_overlap(const Span& a, const Span& b) { return a.lo < b.hi && b.lo < a.hi; }

// The spans of one call: at most one per rank plus one extra buffer (the
// combine's weights), held on the stack so a call allocates nothing.
struct SpanSet {
    Span v[NUNA_MAX_RANKS + 1];
    int n = 0;
    void add(const void* p, size_t bytes, int rank) {
        const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
        v[n++] = {lo, lo + bytes, rank};
    }
};

// Outputs must be pairwise disjoint.  An input may overlap an output only
// when it is the documented in-place alias of that rank: input span equal to
// `alias(rank)` exactly.  Sorting the outputs (in place) keeps the check
// O(P log P).
template <class AllowFn>
nuna_status_t check_overlaps(const SpanSet& ins, SpanSet& outs, AllowFn allowed) {
    Span* ob = outs.v;
    Span* oe = outs.v + outs.n;
    if (ob == oe) return NUNA_OK;
    const auto by_lo = [](const Span& a, const Span& b) { return a.lo < b.lo; };
    if (!std::is_sorted(ob, oe, by_lo)) std::sort(ob, oe, by_lo);  // callers usually pass them in order
    for (const Span* o = ob + 1; o < oe; ++o)
        if (o->lo < (o - 1)->hi)
            return fail(NUNA_ERR_OVERLAP, "output buffers of ranks %d and %d overlap", (o - 1)->rank, o->rank);
    // Sorted and disjoint: the outputs lie within [ob->lo, last->hi).
    const uintptr_t hull_lo = ob->lo, hull_hi = (oe - 1)->hi;
    for (int k = 0; k < ins.n; ++k) {
        const Span& s = ins.v[k];
        if (s.hi <= hull_lo || s.lo >= hull_hi) continue;
        // first output whose end is above s.lo
        const Span* it = std::lower_bound(static_cast<const Span*>(ob), static_cast<const Span*>(oe), s.lo,
                                          [](const Span& o, uintptr_t lo) { return o.hi <= lo; });
        for (; it != oe && it->lo < s.hi; ++it) {
            if (!spans_overlap(s, *it)) continue;
            if (!allowed(s, *it))
                return fail(NUNA_ERR_OVERLAP, "input of rank %d overlaps output of rank %d outside the in-place form",
                            s.rank, it->rank);
        }
    }
    return NUNA_OK;
}

nuna_status_t check_ptr_array(const void* const* a, int P, const char* name) {
    if (!a) return fail(NUNA_ERR_INVALID_ARG, "%s is NULL", name);
    for (int r = 0; r < P; ++r) {
        if (!a[r]) return fail(NUNA_ERR_INVALID_ARG, "%s[%d] is NULL", name, r);
        if (!aligned16(a[r])) return fail(NUNA_ERR_MISALIGNED, "%s[%d] is not 16-byte aligned", name, r);
    }
    return NUNA_OK;
}

nuna_status_t check_common(int P, int dtype, int place) {
    if (P < 1 || P > NUNA_MAX_RANKS) return fail(NUNA_ERR_INVALID_ARG, "P=%d outside [1, %d]", P, NUNA_MAX_RANKS);
    if (!valid_dtype(dtype)) return fail(NUNA_ERR_UNSUPPORTED, "unsupported dtype %d", dtype);
    if (!valid_place(place)) return fail(NUNA_ERR_INVALID_ARG, "invalid placement mode %d", place);
    return NUNA_OK;
}

nuna::Tuning g_tuning;
std::once_flag g_tuning_once;

// Launches of the calling thread's last collective call (nuna_last_launch).
thread_local nuna_launch_info_t t_launch;

// Start the record of a call's launches (after its argument checks).
void begin_launches() { std::memset(&t_launch, 0, sizeof t_launch); }


}  // namespace

namespace {

// Launch-shape tunables: the environment variable's name (read once at first
// use, and also the name nuna_set_tunable takes), the field it sets, and the
// values it accepts (an explicit list, or the range [lo, hi] when the list is
// empty).  Values outside the accepted set are ignored in the environment and
// rejected by nuna_set_tunable.
struct TunableDef {
    const char* name;
    int64_t nuna::Tuning::*wide;  // int64 field, or null
    int nuna::Tuning::*narrow;    // int field, or null
    int64_t lo, hi;
    int nvals;
    int64_t vals[5];
    int64_t get(const nuna::Tuning& t) const { return wide ? t.*wide : t.*narrow; }
    void set(nuna::Tuning& t, int64_t v) const {
        if (wide)
            t.*wide = v;
        else
            t.*narrow = static_cast<int>(v);
    }
    bool accepts(int64_t v) const {
        if (nvals == 0) return v >= lo && v <= hi;
        for (int i = 0; i < nvals; ++i)
            if (vals[i] == v) return true;
        return false;
    }
};

const TunableDef kTunables[] = {
    {"NUNA_MAX_GRID", nullptr, &nuna::Tuning::max_grid, 0, INT32_MAX, 0, {}},
    {"NUNA_WG_THREADS", nullptr, &nuna::Tuning::wg_threads, 0, 0, 4, {0, 64, 128, 256}},
    {"NUNA_VPT", nullptr, &nuna::Tuning::vpt, 0, 0, 5, {0, 1, 2, 4, 8}},
    {"NUNA_LPR_MIN_RANKS", nullptr, &nuna::Tuning::lpr_min_ranks, 1, NUNA_MAX_RANKS + 1, 0, {}},
    {"NUNA_LPR_MAX_VECTORS", &nuna::Tuning::lpr_max_vectors, nullptr, 0, int64_t(1) << 40, 0, {}},
    {"NUNA_COMBINE_VPT", nullptr, &nuna::Tuning::combine_vpt, 0, 0, 4, {0, 1, 2, 4}},
    {"NUNA_COMBINE_CHUNKS", nullptr, &nuna::Tuning::combine_chunks, 0, INT32_MAX, 0, {}},
    {"NUNA_TILE_V", nullptr, &nuna::Tuning::tile_v, 0, 0, 4, {0, 16, 32, 64}},
    {"NUNA_COMBINE_LISTS", nullptr, &nuna::Tuning::combine_lists, 0, 1, 0, {}},
    {"NUNA_WRITE_THROUGH", nullptr, &nuna::Tuning::write_through, 0, 2, 0, {}},
    {"NUNA_PAGE_GROUPS", nullptr, &nuna::Tuning::page_groups, 0, 1, 0, {}},
    {"NUNA_DIRECT_MAX_GRID", nullptr, &nuna::Tuning::direct_max_grid, 0, 1 << 24, 0, {}},
    {"NUNA_TWO_SHOT_FORM", nullptr, &nuna::Tuning::two_shot_form, 0, 2, 0, {}},
    {"NUNA_SHARD_XCD", nullptr, &nuna::Tuning::shard_xcd, 0, 2, 0, {}},
    {"NUNA_STORE_GAP", nullptr, &nuna::Tuning::store_gap, -1, 32, 0, {}},
};

const TunableDef* find_tunable(const char* name) {
    if (!name) return nullptr;
    for (const TunableDef& d : kTunables)
        if (std::strcmp(d.name, name) == 0) return &d;
    return nullptr;
}

}  // namespace

namespace nuna {
void note_launch(const char* kernel, int map, int64_t group_size, int64_t grid, int threads, int vpt) {
    nuna_launch_info_t& r = t_launch;
    const size_t used = std::strlen(r.kernels);
    std::snprintf(r.kernels + used, sizeof r.kernels - used, "%s%s", used ? "+" : "", kernel);
    ++r.launches;
    if (map != kMapLinear) {
        r.map = map;
        r.group_size = group_size;
    } else if (r.launches == 1) {
        r.group_size = group_size;
    }
    r.grid = grid;
    r.threads = threads;
    r.vectors_per_thread = vpt;
}

const Tuning& tuning() {
    std::call_once(g_tuning_once, [] {
        for (const TunableDef& d : kTunables) {
            const char* v = std::getenv(d.name);
            if (!v || !*v) continue;
            char* end = nullptr;
            const long long x = std::strtoll(v, &end, 10);
            if (end && *end == '\0' && d.accepts(x)) d.set(g_tuning, x);
        }
    });
    return g_tuning;
}

std::atomic<int> g_max_workgroups{0};

int max_workgroups() {
    const int v = g_max_workgroups.load(std::memory_order_relaxed);
    if (v > 0) return v;
    return tuning().max_grid > 0 ? tuning().max_grid : 16384;
}

int64_t grid_limit(int64_t dflt) {
    const int v = g_max_workgroups.load(std::memory_order_relaxed);
    if (v > 0) return v;
    return tuning().max_grid > 0 ? tuning().max_grid : dflt;
}
}  // namespace nuna

// ============================================================== device probe

namespace {

// Per-device result of nuna_init's dispatch-map probe.
constexpr int kMaxDevices = 64;
enum MapState { kMapUnknown = 0, kMapVerified = 1, kMapFailed = 2 };
std::atomic<int> g_map_state[kMaxDevices];
std::atomic<int> g_cu_count[kMaxDevices];
std::atomic<int> g_xcd_count[kMaxDevices];
// Device address of the routed dispatch's static scratch array, per device
// (set by nuna_init with that device current).
std::atomic<void*> g_scratch[kMaxDevices];

// Workgroups the init probe launches: a few per compute unit, in many rounds of 8.
constexpr int kProbeGrid = 2048;

// XCD placement relies on the hardware running workgroup b on XCD b mod 8
// (placement.h).  Before the first XCD-mode call on a device, nuna_init must
// have verified that map there; a device where it does not hold (another
// partition mode, another chip) gets NUNA_ERR_UNSUPPORTED for XCD mode rather
// than a placement the kernels do not intend.  LINEAR needs no map.
nuna_status_t check_placement_ready(int place) {
    if (place != NUNA_PLACE_XCD) return NUNA_OK;
    int dev = 0;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e, "hipGetDevice");
    const int st = (dev >= 0 && dev < kMaxDevices) ? g_map_state[dev].load(std::memory_order_acquire) : kMapUnknown;
    if (st == kMapVerified) return NUNA_OK;
    if (st == kMapFailed)
        return fail(NUNA_ERR_UNSUPPORTED,
                    "XCD placement is unavailable on device %d: nuna_init found that workgroup b does not run on "
                    "XCD b mod %d there",
                    dev, NUNA_NUM_XCD);
    return fail(NUNA_ERR_UNSUPPORTED,
                "XCD placement needs nuna_init() on device %d first (it verifies the workgroup -> XCD dispatch map)",
                dev);
}

}  // namespace

// ============================================================== C ABI

extern "C" {

const char* nuna_last_error_string(void) { return t_err.c_str(); }

int nuna_version(void) { return 200; }

nuna_status_t nuna_set_max_workgroups(int max_workgroups) {
    if (max_workgroups < 0) return fail(NUNA_ERR_INVALID_ARG, "max_workgroups=%d < 0", max_workgroups);
    nuna::g_max_workgroups.store(max_workgroups, std::memory_order_relaxed);
    return ok();
}

nuna_status_t nuna_set_tunable(const char* name, int64_t value) {
    const TunableDef* d = find_tunable(name);
    if (!d) return fail(NUNA_ERR_INVALID_ARG, "unknown tunable %s", name ? name : "(null)");
    if (!d->accepts(value))
        return fail(NUNA_ERR_INVALID_ARG, "%s does not accept %lld", d->name, static_cast<long long>(value));
    (void)nuna::tuning();  // environment read first, so a later read cannot undo this setting
    d->set(g_tuning, value);
    return ok();
}

nuna_status_t nuna_get_tunable(const char* name, int64_t* value) {
    const TunableDef* d = find_tunable(name);
    if (!d) return fail(NUNA_ERR_INVALID_ARG, "unknown tunable %s", name ? name : "(null)");
    if (!value) return fail(NUNA_ERR_INVALID_ARG, "value is NULL");
    *value = d->get(nuna::tuning());
    return ok();
}

nuna_status_t nuna_check_dispatch_map(const int32_t* xcc, int64_t G, int32_t cu_count) {
    if (!xcc) return fail(NUNA_ERR_INVALID_ARG, "xcc is NULL");
    if (G < 8 * NUNA_NUM_XCD) return fail(NUNA_ERR_INVALID_ARG, "G=%lld: need at least %d workgroups", (long long)G,
                                          8 * NUNA_NUM_XCD);
    if (cu_count != NUNA_NUM_XCD * 32)
        return fail(NUNA_ERR_UNSUPPORTED, "%d compute units, expected %d (%d XCDs of 32)", cu_count,
                    NUNA_NUM_XCD * 32, NUNA_NUM_XCD);
    for (int64_t b = 0; b < G; ++b)
        if (xcc[b] != static_cast<int32_t>(b % NUNA_NUM_XCD))
            return fail(NUNA_ERR_UNSUPPORTED, "workgroup %lld ran on XCD %d, not %lld (b mod %d)", (long long)b, xcc[b],
                        (long long)(b % NUNA_NUM_XCD), NUNA_NUM_XCD);
    return ok();
}

nuna_status_t nuna_init(void) try {
    static std::mutex mu;
    std::lock_guard<std::mutex> lock(mu);
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess || n < 1) return fail(NUNA_ERR_HIP, "no HIP device (%s)", hipGetErrorString(e));
    int dev = 0;
    e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(NUNA_ERR_UNSUPPORTED, "device ordinal %d >= %d", dev, kMaxDevices);
    if (g_map_state[dev].load(std::memory_order_acquire) == kMapVerified) return ok();
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return hip_status(e, "hipGetDeviceProperties");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(NUNA_ERR_UNSUPPORTED, "device %d is %s, libnuna is built for gfx950", dev, prop.gcnArchName);
    (void)nuna::tuning();
    // Dispatch-map probe: every workgroup records the XCC it ran on.
    int32_t* d_xcc = nullptr;
    if ((e = hipMalloc(&d_xcc, sizeof(int32_t) * kProbeGrid)) != hipSuccess) return hip_status(e, "hipMalloc (probe)");
    std::vector<int32_t> xcc(kProbeGrid, -1);
    e = nuna::launch_probe_xcc(kProbeGrid, d_xcc, nullptr, nullptr);
    if (e == hipSuccess) e = hipMemcpy(xcc.data(), d_xcc, sizeof(int32_t) * kProbeGrid, hipMemcpyDeviceToHost);
    (void)hipFree(d_xcc);
    if (e != hipSuccess) return hip_status(e, "dispatch-map probe");
    int xcds = 0;
    for (int32_t x : xcc) xcds = std::max(xcds, x + 1);
    g_cu_count[dev].store(prop.multiProcessorCount, std::memory_order_relaxed);
    g_xcd_count[dev].store(xcds, std::memory_order_relaxed);
    // The routed dispatch's scratch array: each device holds its own copy at its own address.
    void* scr = nullptr;
    if ((e = nuna::routed_scratch_address(&scr)) != hipSuccess || !scr)
        return hip_status(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress (scratch)");
    g_scratch[dev].store(scr, std::memory_order_release);
    const nuna_status_t st = nuna_check_dispatch_map(xcc.data(), kProbeGrid, prop.multiProcessorCount);
    g_map_state[dev].store(st == NUNA_OK ? kMapVerified : kMapFailed, std::memory_order_release);
    if (st != NUNA_OK) {
        // LINEAR placement still works; XCD placement on this device reports why it is unavailable.
        const std::string why = t_err;
        return fail(NUNA_ERR_UNSUPPORTED, "device %d: dispatch map check failed (%s); XCD placement is unavailable",
                    dev, why.c_str());
    }
    return ok();
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_last_launch(nuna_launch_info_t* info) {
    if (!info) return fail(NUNA_ERR_INVALID_ARG, "info is NULL");
    *info = t_launch;
    return ok();
}

nuna_status_t nuna_get_device_info(nuna_device_info_t* info) {
    if (!info) return fail(NUNA_ERR_INVALID_ARG, "info is NULL");
    std::memset(info, 0, sizeof *info);
    int dev = 0;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e, "hipGetDevice");
    info->device = dev;
    if (dev < 0 || dev >= kMaxDevices) return fail(NUNA_ERR_INVALID_ARG, "device ordinal %d >= %d", dev, kMaxDevices);
    const int st = g_map_state[dev].load(std::memory_order_acquire);
    if (st == kMapUnknown) return fail(NUNA_ERR_INVALID_ARG, "nuna_init() has not run on device %d", dev);
    info->cu_count = g_cu_count[dev].load(std::memory_order_relaxed);
    info->xcd_count = g_xcd_count[dev].load(std::memory_order_relaxed);
    info->map_verified = st == kMapVerified ? 1 : 0;
    return ok();
}

namespace {

// NUNA_ALGO_AUTO: the two-shot for 8 ranks of bf16 from 16 MiB per rank
// (fused or two kernels, two_shot_runs_fused), the one-shot elsewhere.
// Measured on MI355X, cold, per call: 46.2-46.6 against 47.9-48.2 us at
// 16 MiB per rank, 177-179 against 179-181 at 64 MiB, 380-390 against
// 386-421 at 128 MiB; at 4 MiB the one-shot leads (11.4-11.6 against
// 11.6-11.7 us), as at every smaller size.
bool auto_two_shot(int P, size_t count, int dtype) {
    return P == 8 && dtype == nuna::kDtBf16 && count * nuna::dtype_size(dtype) >= (size_t(16) << 20) &&
           nuna::two_shot_fused_ok(P, count, dtype);
}

}  // namespace

nuna_status_t nuna_allreduce(const void* const* in, void* const* out, int P, size_t count, nuna_dtype_t dtype,
                             nuna_algo_t algo, nuna_placement_t place, hipStream_t stream) try {
    begin_launches();
    nuna_status_t st = check_common(P, dtype, place);
    if (st) return st;
    if (algo < NUNA_ALGO_AUTO || algo > NUNA_ALGO_TWO_SHOT_TWO_KERNELS)
        return fail(NUNA_ERR_INVALID_ARG, "invalid algorithm %d", static_cast<int>(algo));
    if ((st = check_ptr_array(in, P, "in"))) return st;
    if ((st = check_ptr_array(const_cast<const void* const*>(out), P, "out"))) return st;
    const size_t es = nuna::dtype_size(dtype);
    if (count > kMaxBytes / es) return fail(NUNA_ERR_INVALID_ARG, "count %zu too large", count);
    const size_t bytes = count * es;
    if (count == 0) return ok();
    SpanSet is, os;
    bool in_place = false;
    for (int r = 0; r < P; ++r) {
        is.add(in[r], bytes, r);
        os.add(out[r], bytes, r);
        in_place = in_place || in[r] == out[r];
    }
    st = check_overlaps(is, os, [](const Span& i, const Span& o) { return i.rank == o.rank && i.lo == o.lo; });
    if (st) return st;

    if ((st = check_placement_ready(place))) return st;

    int a = algo;
    if (a == NUNA_ALGO_AUTO) a = auto_two_shot(P, count, dtype) ? NUNA_ALGO_TWO_SHOT : NUNA_ALGO_ONE_SHOT;
    if ((a == NUNA_ALGO_TWO_SHOT || a == NUNA_ALGO_TWO_SHOT_TWO_KERNELS) && count % static_cast<size_t>(P) != 0)
        a = NUNA_ALGO_ONE_SHOT;
    if (a == NUNA_ALGO_ONE_SHOT_SPLIT && in_place) a = NUNA_ALGO_ONE_SHOT;
    if (a == NUNA_ALGO_TWO_SHOT) {
        // Both phases in one kernel, or two kernels where the shapes need it or
        // they measured faster (two_shot_runs_fused).
        if (nuna::two_shot_runs_fused(P, count, dtype))
            return hip_status(nuna::launch_two_shot_fused(in, out, P, count, dtype, place, stream),
                              "two-shot launch");
        a = NUNA_ALGO_TWO_SHOT_TWO_KERNELS;
    }

    hipError_t e;
    if (a == NUNA_ALGO_TWO_SHOT_TWO_KERNELS) {
        const size_t m = count / P;
        const void* shard_in[NUNA_MAX_RANKS];
        void* shard_out[NUNA_MAX_RANKS];
        for (int r = 0; r < P; ++r) {
            shard_out[r] = static_cast<char*>(out[r]) + static_cast<size_t>(r) * m * es;
            shard_in[r] = shard_out[r];
        }
        e = nuna::launch_reduce_scatter(in, shard_out, P, m, dtype, place, true, stream);
        if (e != hipSuccess) return hip_status(e, "reduce-scatter phase launch");
        e = nuna::launch_all_gather(shard_in, out, P, m, dtype, place, true, stream);
        return hip_status(e, "all-gather phase launch");
    }
    int groups = 1;
    if (a == NUNA_ALGO_ONE_SHOT_SPLIT) {
        for (int d = P < 8 ? P : 8; d > 1; --d)
            if (P % d == 0) {
                groups = d;
                break;
            }
    }
    e = nuna::launch_allreduce(in, out, P, count, dtype, groups, place, stream);
    return hip_status(e, "all-reduce launch");
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_reduce_scatter(const void* const* in, void* const* out, int P, size_t recvcount,
                                  nuna_dtype_t dtype, nuna_placement_t place, hipStream_t stream) try {
    begin_launches();
    nuna_status_t st = check_common(P, dtype, place);
    if (st) return st;
    if ((st = check_ptr_array(in, P, "in"))) return st;
    if ((st = check_ptr_array(const_cast<const void* const*>(out), P, "out"))) return st;
    const size_t es = nuna::dtype_size(dtype);
    if (recvcount > kMaxBytes / es / static_cast<size_t>(P))
        return fail(NUNA_ERR_INVALID_ARG, "recvcount %zu too large", recvcount);
    if (recvcount == 0) return ok();
    const size_t mb = recvcount * es;
    SpanSet is, os;
    for (int r = 0; r < P; ++r) {
        is.add(in[r], mb * P, r);
        os.add(out[r], mb, r);
    }
    st = check_overlaps(is, os, [mb](const Span& i, const Span& o) {
        return i.rank == o.rank && o.lo == i.lo + static_cast<uintptr_t>(o.rank) * mb;
    });
    if (st) return st;
    if ((st = check_placement_ready(place))) return st;
    return hip_status(nuna::launch_reduce_scatter(in, out, P, recvcount, dtype, place, false, stream),
                      "reduce-scatter launch");
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_all_gather(const void* const* in, void* const* out, int P, size_t sendcount, nuna_dtype_t dtype,
                              nuna_placement_t place, hipStream_t stream) try {
    begin_launches();
    nuna_status_t st = check_common(P, dtype, place);
    if (st) return st;
    if ((st = check_ptr_array(in, P, "in"))) return st;
    if ((st = check_ptr_array(const_cast<const void* const*>(out), P, "out"))) return st;
    const size_t es = nuna::dtype_size(dtype);
    if (sendcount > kMaxBytes / es / static_cast<size_t>(P))
        return fail(NUNA_ERR_INVALID_ARG, "sendcount %zu too large", sendcount);
    if (sendcount == 0) return ok();
    const size_t mb = sendcount * es;
    SpanSet is, os;
    for (int r = 0; r < P; ++r) {
        is.add(in[r], mb, r);
        os.add(out[r], mb * P, r);
    }
    st = check_overlaps(is, os, [mb](const Span& i, const Span& o) {
        return i.rank == o.rank && i.lo == o.lo + static_cast<uintptr_t>(i.rank) * mb;
    });
    if (st) return st;
    if ((st = check_placement_ready(place))) return st;
    return hip_status(nuna::launch_all_gather(in, out, P, sendcount, dtype, place, false, stream), "all-gather launch");
} catch (...) {
    return host_exception();
}

// ------------------------------------------------------------ all-to-all layout

struct nuna_a2a_layout {
    int P = 0, T = 0, k = 0, E = 0;
    std::vector<int64_t> rows;        // rows received per destination
    std::vector<int64_t> dst_off;     // P+1 offsets into the per-destination maps
    std::vector<int32_t> map_src;     // source rank of each received row, destination-major
    std::vector<int32_t> map_tok;     // source token of each received row
    std::vector<int32_t> desc_linear; // 4 ints per item, ordered by (dst, row)
    std::vector<int32_t> desc_group;  // 4 ints per item, XCD-major: each source-row group on its planned XCD
    int64_t xcd_start[NUNA_NUM_XCD + 1] = {};  // per-XCD list offsets into desc_group
    int64_t nitems = 0;
    // Combine tables: token i = s*T + t owns entries [comb_off[i], comb_off[i+1]),
    // each a (destination rank, receive row) pair, destinations ascending.
    std::vector<int64_t> comb_off;
    std::vector<int32_t> comb_ent;
    // The same lists as fixed-size records, for up to 8 ranks: 8 words per
    // token, word q = (receive row << 3) | rank for the token's q-th entry,
    // all ones after its last.  Empty when P > 8 or a row index needs more
    // than 29 bits.
    std::vector<uint32_t> comb_rec;
    void* dev_base = nullptr;  // one allocation holding every device table
    void* dev_linear = nullptr;
    void* dev_group = nullptr;
    void* dev_comb_off = nullptr;
    void* dev_comb_ent = nullptr;
    void* dev_comb_rec = nullptr;
    int device = -1;
};

nuna_status_t nuna_a2a_layout_create(int P, int tokens_per_rank, int topk, int num_experts, const int32_t* topk_idx,
                                     nuna_a2a_layout_t** out) try {
    if (!out) return fail(NUNA_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (P < 1 || P > NUNA_MAX_RANKS) return fail(NUNA_ERR_INVALID_ARG, "P=%d outside [1, %d]", P, NUNA_MAX_RANKS);
    if (tokens_per_rank < 0) return fail(NUNA_ERR_INVALID_ARG, "tokens_per_rank=%d < 0", tokens_per_rank);
    if (num_experts < P || num_experts % P != 0)
        return fail(NUNA_ERR_INVALID_ARG, "num_experts=%d is not a positive multiple of P=%d", num_experts, P);
    if (topk < 1 || topk > num_experts)
        return fail(NUNA_ERR_INVALID_ARG, "topk=%d outside [1, num_experts=%d]", topk, num_experts);
    if (tokens_per_rank > 0 && !topk_idx) return fail(NUNA_ERR_INVALID_ARG, "topk_idx is NULL");
    const int per = num_experts / P;
    const int64_t ntok = static_cast<int64_t>(P) * tokens_per_rank;
    // Receive rows and token indices are stored as int32.
    if (ntok > INT32_MAX)
        return fail(NUNA_ERR_INVALID_ARG, "P*tokens_per_rank=%lld exceeds %d", static_cast<long long>(ntok), INT32_MAX);
    for (int64_t i = 0; i < ntok * topk; ++i)
        if (topk_idx[i] < 0 || topk_idx[i] >= num_experts)
            return fail(NUNA_ERR_INVALID_ARG, "topk_idx[%lld]=%d outside [0, %d)", static_cast<long long>(i),
                        topk_idx[i], num_experts);

    std::unique_ptr<nuna_a2a_layout> L(new nuna_a2a_layout());
    L->P = P;
    L->T = tokens_per_rank;
    L->k = topk;
    L->E = num_experts;
    L->rows.assign(P, 0);
    // Pass 1: destination mask per token, rows per destination.
    std::vector<uint64_t> mask(static_cast<size_t>(ntok));
    for (int64_t i = 0; i < ntok; ++i) {
        uint64_t m = 0;
        for (int j = 0; j < topk; ++j) m |= uint64_t(1) << (topk_idx[i * topk + j] / per);
        mask[i] = m;
        for (int d = 0; d < P; ++d)
            if (m >> d & 1u) ++L->rows[d];
    }
    L->dst_off.assign(P + 1, 0);
    for (int d = 0; d < P; ++d) L->dst_off[d + 1] = L->dst_off[d] + L->rows[d];
    L->nitems = L->dst_off[P];
    L->map_src.resize(L->nitems);
    L->map_tok.resize(L->nitems);
    L->desc_linear.resize(4 * L->nitems);
    // Pass 2: walk tokens in (source, token) order; each destination's row
    // counter therefore advances in receive order.  The same walk lists, per
    // token, the (destination, receive row) pairs the combine reads back,
    // destinations ascending.
    std::vector<int64_t> next(P, 0);
    L->comb_off.assign(static_cast<size_t>(ntok) + 1, 0);
    L->comb_ent.reserve(2 * L->nitems);
    // Row indices stay below ntok < 2^29, so no entry is all ones.
    const bool records = P <= nuna::kCombRecRanks && ntok < (int64_t(1) << 29);
    if (records) L->comb_rec.assign(static_cast<size_t>(ntok) * nuna::kCombRecRanks, ~uint32_t(0));
    // Placement workload for the XCD mode: one threadblock per row copy, in
    // walk order, touching its source row and its destination row.
    std::vector<int64_t> tb_off(static_cast<size_t>(L->nitems) + 1, 0);
    std::vector<int64_t> tb_chunk(2 * static_cast<size_t>(L->nitems));
    std::vector<int32_t> walk_desc(4 * static_cast<size_t>(L->nitems));
    int64_t w = 0;
    for (int s = 0; s < P; ++s) {
        for (int t = 0; t < tokens_per_rank; ++t) {
            const size_t tok = static_cast<size_t>(s) * tokens_per_rank + t;
            const uint64_t m = mask[tok];
            L->comb_off[tok + 1] = L->comb_off[tok] + __builtin_popcountll(m);
            size_t q_rec = tok * nuna::kCombRecRanks;  // the token's next record word
            for (int d = 0; d < P; ++d) {
                if (!(m >> d & 1u)) continue;
                const int64_t j = next[d]++;
                const int64_t pos = L->dst_off[d] + j;
                L->map_src[pos] = s;
                L->map_tok[pos] = t;
                const int32_t q[4] = {s, t, d, static_cast<int32_t>(j)};
                std::memcpy(&L->desc_linear[4 * pos], q, sizeof q);
                std::memcpy(&walk_desc[4 * static_cast<size_t>(w)], q, sizeof q);
                tb_chunk[2 * static_cast<size_t>(w)] = static_cast<int64_t>(tok);        // source row
                tb_chunk[2 * static_cast<size_t>(w) + 1] = ntok + pos;                    // destination row
                tb_off[static_cast<size_t>(w) + 1] = 2 * (w + 1);
                ++w;
                if (records) L->comb_rec[q_rec++] = static_cast<uint32_t>(j) << 3 | static_cast<uint32_t>(d);
                L->comb_ent.push_back(d);
                L->comb_ent.push_back(static_cast<int32_t>(j));
            }
        }
    }
    // XCD assignment from the placement planner (Algorithm 1): the copies of
    // one token share its source row and form one logical group; groups go to
    // the 8 XCDs round-robin in decreasing size order, which evens out the
    // copies per XCD.  Every copy is charged the same, so the budgets never
    // bind and only the domain choice matters.  The algorithm fixes where a
    // group runs, not when: each XCD runs its groups in token order, which
    // keeps its source-row reads in address order (dealing them in size order
    // measured 4 % slower on MI355X).
    const std::vector<int64_t> unit(static_cast<size_t>(L->nitems), 1);
    const nuna::NapPlan plan = nuna::nap_plan(nuna::nap_topology_mi355x(), NUNA_NUM_XCD, L->nitems, tb_off.data(),
                                              tb_chunk.data(), unit.data(), nullptr);
    std::vector<std::vector<int32_t>> per_xcd(NUNA_NUM_XCD);
    for (size_t g = 0; g < plan.groups.size(); ++g) {
        const std::vector<int64_t>& members = plan.groups[g];
        std::vector<int32_t>& lst = per_xcd[static_cast<size_t>(plan.tb_domain[static_cast<size_t>(members[0])])];
        for (int64_t tb : members)
            lst.insert(lst.end(), &walk_desc[4 * static_cast<size_t>(tb)], &walk_desc[4 * static_cast<size_t>(tb)] + 4);
    }
    L->desc_group.reserve(4 * L->nitems);
    for (int x = 0; x < NUNA_NUM_XCD; ++x) {
        L->xcd_start[x] = static_cast<int64_t>(L->desc_group.size() / 4);
        L->desc_group.insert(L->desc_group.end(), per_xcd[x].begin(), per_xcd[x].end());
    }
    L->xcd_start[NUNA_NUM_XCD] = L->nitems;
    *out = L.release();
    return ok();
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_a2a_layout_upload(nuna_a2a_layout_t* L) {
    if (!L) return fail(NUNA_ERR_INVALID_ARG, "layout is NULL");
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e, "hipGetDevice");
    if (L->device >= 0) {
        if (L->device == dev) return ok();
        return fail(NUNA_ERR_INVALID_ARG, "layout already uploaded to device %d (current %d)", L->device, dev);
    }
    if (L->nitems == 0) {  // nothing routed: no tables, every collective on it is a no-op
        L->device = dev;
        return ok();
    }
    // One allocation: dispatch descriptors (linear, then XCD-major), combine
    // offsets, combine entries, combine records.  Every part starts 16-byte
    // aligned; the records start 32-byte aligned (one record per 32 bytes).
    const size_t n_desc = static_cast<size_t>(L->nitems) * 16;
    const size_t n_off = (L->comb_off.size() * sizeof(int64_t) + 15) & ~size_t(15);
    const size_t n_ent = (L->comb_ent.size() * sizeof(int32_t) + 31) & ~size_t(31);
    const size_t at_rec = (2 * n_desc + n_off + n_ent + 31) & ~size_t(31);
    const size_t n_rec = L->comb_rec.size() * sizeof(uint32_t);
    const size_t bytes = at_rec + n_rec;
    void* base = nullptr;
    if ((e = hipMalloc(&base, bytes)) != hipSuccess) return hip_status(e, "hipMalloc (a2a tables)");
    char* b = static_cast<char*>(base);
    const struct {
        size_t at;
        const void* src;
        size_t n;
    } parts[5] = {{0, L->desc_linear.data(), n_desc},
                  {n_desc, L->desc_group.data(), n_desc},
                  {2 * n_desc, L->comb_off.data(), L->comb_off.size() * sizeof(int64_t)},
                  {2 * n_desc + n_off, L->comb_ent.data(), L->comb_ent.size() * sizeof(int32_t)},
                  {at_rec, L->comb_rec.data(), n_rec}};
    for (const auto& q : parts) {
        if (q.n == 0) continue;
        if ((e = hipMemcpy(b + q.at, q.src, q.n, hipMemcpyHostToDevice)) != hipSuccess) {
            (void)hipFree(base);
            return hip_status(e, "hipMemcpy (a2a tables)");
        }
    }
    L->dev_base = base;
    L->dev_linear = b;
    L->dev_group = b + n_desc;
    L->dev_comb_off = b + 2 * n_desc;
    L->dev_comb_ent = b + 2 * n_desc + n_off;
    L->dev_comb_rec = n_rec ? b + at_rec : nullptr;
    L->device = dev;
    return ok();
}

nuna_status_t nuna_a2a_layout_recv_rows(const nuna_a2a_layout_t* L, int64_t* rows_per_rank) {
    if (!L || !rows_per_rank) return fail(NUNA_ERR_INVALID_ARG, "NULL argument");
    for (int d = 0; d < L->P; ++d) rows_per_rank[d] = L->rows[d];
    return ok();
}

nuna_status_t nuna_a2a_layout_recv_map(const nuna_a2a_layout_t* L, int d, int32_t* src_rank, int32_t* src_token) {
    if (!L || !src_rank || !src_token) return fail(NUNA_ERR_INVALID_ARG, "NULL argument");
    if (d < 0 || d >= L->P) return fail(NUNA_ERR_INVALID_ARG, "destination %d outside [0, %d)", d, L->P);
    for (int64_t j = 0; j < L->rows[d]; ++j) {
        src_rank[j] = L->map_src[L->dst_off[d] + j];
        src_token[j] = L->map_tok[L->dst_off[d] + j];
    }
    return ok();
}

void nuna_a2a_layout_destroy(nuna_a2a_layout_t* L) {
    if (!L) return;
    if (L->dev_base) (void)hipFree(L->dev_base);
    delete L;
}

nuna_status_t nuna_all_to_all(const void* const* send, void* const* recv, const nuna_a2a_layout_t* L,
                              size_t row_elems, size_t recv_capacity_rows, nuna_dtype_t dtype,
                              nuna_placement_t place, hipStream_t stream) try {
    begin_launches();
    if (!L) return fail(NUNA_ERR_INVALID_ARG, "layout is NULL");
    const int P = L->P;
    nuna_status_t st = check_common(P, dtype, place);
    if (st) return st;
    if ((st = check_ptr_array(send, P, "send"))) return st;
    if ((st = check_ptr_array(const_cast<const void* const*>(recv), P, "recv"))) return st;
    const size_t es = nuna::dtype_size(dtype);
    if (row_elems == 0) return fail(NUNA_ERR_INVALID_ARG, "row_elems is 0");
    if (row_elems > kMaxBytes / es) return fail(NUNA_ERR_INVALID_ARG, "row_elems %zu too large", row_elems);
    const size_t row_bytes = row_elems * es;
    for (int d = 0; d < P; ++d)
        if (static_cast<size_t>(L->rows[d]) > recv_capacity_rows)
            return fail(NUNA_ERR_INVALID_ARG, "rank %d receives %lld rows, capacity is %zu", d,
                        static_cast<long long>(L->rows[d]), recv_capacity_rows);
    if (static_cast<size_t>(L->T) > kMaxBytes / row_bytes || recv_capacity_rows > kMaxBytes / row_bytes)
        return fail(NUNA_ERR_INVALID_ARG, "buffer sizes too large");
    SpanSet ss, rs;
    for (int r = 0; r < P; ++r) {
        ss.add(send[r], row_bytes * L->T, r);
        rs.add(recv[r], row_bytes * recv_capacity_rows, r);
    }
    st = check_overlaps(ss, rs, [](const Span&, const Span&) { return false; });
    if (st) return st;
    if (L->nitems == 0) return ok();
    if (L->device < 0) return fail(NUNA_ERR_INVALID_ARG, "layout has not been uploaded (nuna_a2a_layout_upload)");
    if ((st = check_placement_ready(place))) return st;
    const void* desc = place == NUNA_PLACE_XCD ? L->dev_group : L->dev_linear;
    hipError_t e = nuna::launch_all_to_all(send, recv, P, desc, L->nitems, L->xcd_start, row_bytes,
                                           static_cast<int>(es), place, stream);
    return hip_status(e, "all-to-all launch");
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_all_to_all_routed(const void* const* send, void* const* recv, const int32_t* topk_idx, int P,
                                     int tokens_per_rank, int topk, int num_experts, size_t row_elems,
                                     size_t recv_capacity_rows, nuna_dtype_t dtype, nuna_placement_t place,
                                     int64_t* rows_per_rank, hipStream_t stream) try {
    begin_launches();
    nuna_status_t st = check_common(P, dtype, place);
    if (st) return st;
    const int T = tokens_per_rank;
    if (T < 0) return fail(NUNA_ERR_INVALID_ARG, "tokens_per_rank=%d < 0", T);
    if (num_experts < P || num_experts % P != 0)
        return fail(NUNA_ERR_INVALID_ARG, "num_experts=%d is not a positive multiple of P=%d", num_experts, P);
    if (topk < 1 || topk > num_experts)
        return fail(NUNA_ERR_INVALID_ARG, "topk=%d outside [1, num_experts=%d]", topk, num_experts);
    if ((st = check_ptr_array(send, P, "send"))) return st;
    if ((st = check_ptr_array(const_cast<const void* const*>(recv), P, "recv"))) return st;
    if (T > 0 && !topk_idx) return fail(NUNA_ERR_INVALID_ARG, "topk_idx is NULL");
    if (!rows_per_rank) return fail(NUNA_ERR_INVALID_ARG, "rows_per_rank is NULL");
    if ((reinterpret_cast<uintptr_t>(topk_idx) & 3u) || (reinterpret_cast<uintptr_t>(rows_per_rank) & 7u))
        return fail(NUNA_ERR_MISALIGNED, "topk_idx must be 4-byte and rows_per_rank 8-byte aligned");
    const size_t es = nuna::dtype_size(dtype);
    if (row_elems == 0) return fail(NUNA_ERR_INVALID_ARG, "row_elems is 0");
    if (row_elems > kMaxBytes / es) return fail(NUNA_ERR_INVALID_ARG, "row_elems %zu too large", row_elems);
    const size_t row_bytes = row_elems * es;
    if (row_bytes % 16 != 0)
        return fail(NUNA_ERR_UNSUPPORTED, "routed dispatch rows must be whole 16-byte vectors (%zu bytes)", row_bytes);
    const int64_t ntok = static_cast<int64_t>(P) * T;
    if (ntok >= (int64_t(1) << 26))
        return fail(NUNA_ERR_INVALID_ARG, "P*tokens_per_rank=%lld: the routed dispatch takes fewer than 2^26 tokens",
                    static_cast<long long>(ntok));
    const size_t need = nuna::routed_scratch_need(P, T, topk);
    if (need > nuna::kRoutedScratchBytes)
        return fail(NUNA_ERR_INVALID_ARG,
                    "routing tables need %zu bytes (4*P*P + 4*P + 4*P*T*min(topk, P)), more than the %zu-byte scratch",
                    need, nuna::kRoutedScratchBytes);
    if (static_cast<size_t>(T) > kMaxBytes / row_bytes || recv_capacity_rows > kMaxBytes / row_bytes)
        return fail(NUNA_ERR_INVALID_ARG, "buffer sizes too large");
    SpanSet ins, outs;
    for (int r = 0; r < P; ++r) {
        ins.add(send[r], row_bytes * T, r);
        outs.add(recv[r], row_bytes * recv_capacity_rows, r);
    }
    if (T > 0) ins.add(topk_idx, sizeof(int32_t) * static_cast<size_t>(ntok) * topk, -1);
    outs.add(rows_per_rank, sizeof(int64_t) * (static_cast<size_t>(P) + 1), -1);
    st = check_overlaps(ins, outs, [](const Span&, const Span&) { return false; });
    if (st) return st;
    if ((st = check_placement_ready(place))) return st;
    int dev = 0;
    const hipError_t ge = hipGetDevice(&dev);
    if (ge != hipSuccess) return hip_status(ge, "hipGetDevice");
    void* scr = dev >= 0 && dev < kMaxDevices ? g_scratch[dev].load(std::memory_order_acquire) : nullptr;
    if (!scr) return fail(NUNA_ERR_UNSUPPORTED, "the routed dispatch needs nuna_init() on device %d first", dev);
    return hip_status(nuna::launch_routed_dispatch(send, recv, topk_idx, P, T, topk, num_experts,
                                                   static_cast<int64_t>(row_bytes / 16),
                                                   static_cast<int64_t>(recv_capacity_rows), scr, rows_per_rank,
                                                   place == NUNA_PLACE_XCD ? nuna::kPlaceXcd : nuna::kPlaceLinear,
                                                   stream),
                      "routed dispatch launch");
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_all_to_all_combine(const void* const* y, void* const* out, const nuna_a2a_layout_t* L,
                                      const float* weights, size_t row_elems, size_t y_capacity_rows,
                                      nuna_dtype_t dtype, nuna_placement_t place, hipStream_t stream) try {
    begin_launches();
    if (!L) return fail(NUNA_ERR_INVALID_ARG, "layout is NULL");
    const int P = L->P;
    nuna_status_t st = check_common(P, dtype, place);
    if (st) return st;
    if ((st = check_ptr_array(y, P, "y"))) return st;
    if ((st = check_ptr_array(const_cast<const void* const*>(out), P, "out"))) return st;
    const size_t es = nuna::dtype_size(dtype);
    if (row_elems == 0) return fail(NUNA_ERR_INVALID_ARG, "row_elems is 0");
    if (row_elems > kMaxBytes / es) return fail(NUNA_ERR_INVALID_ARG, "row_elems %zu too large", row_elems);
    const size_t row_bytes = row_elems * es;
    for (int d = 0; d < P; ++d)
        if (static_cast<size_t>(L->rows[d]) > y_capacity_rows)
            return fail(NUNA_ERR_INVALID_ARG, "rank %d holds %lld result rows, capacity is %zu", d,
                        static_cast<long long>(L->rows[d]), y_capacity_rows);
    if (static_cast<size_t>(L->T) > kMaxBytes / row_bytes || y_capacity_rows > kMaxBytes / row_bytes)
        return fail(NUNA_ERR_INVALID_ARG, "buffer sizes too large");
    if (weights && (reinterpret_cast<uintptr_t>(weights) & 3u) != 0)
        return fail(NUNA_ERR_MISALIGNED, "weights is not 4-byte aligned");
    SpanSet ys, os;
    for (int r = 0; r < P; ++r) {
        ys.add(y[r], row_bytes * y_capacity_rows, r);
        os.add(out[r], row_bytes * L->T, r);
    }
    if (weights) ys.add(weights, sizeof(float) * static_cast<size_t>(P) * static_cast<size_t>(L->T) * P, -1);
    st = check_overlaps(ys, os, [](const Span&, const Span&) { return false; });
    if (st) return st;
    if (L->nitems == 0) return ok();
    if (L->device < 0) return fail(NUNA_ERR_INVALID_ARG, "layout has not been uploaded (nuna_a2a_layout_upload)");
    if ((st = check_placement_ready(place))) return st;
    hipError_t e = nuna::launch_combine(y, out, P, L->T, L->dev_comb_off, L->dev_comb_ent, L->dev_comb_rec, weights,
                                        row_bytes, static_cast<int>(dtype), place, stream);
    return hip_status(e, "all-to-all combine launch");
} catch (...) {
    return host_exception();
}

static_assert(NUNA_NAP_MAX_DOMAINS == nuna::kNapMaxDomains && NUNA_NAP_MAX_STACKS == nuna::kNapMaxStacks,
              "planner limits");

nuna_status_t nuna_nap_topology_mi355x(nuna_nap_topology_t* topo) {
    if (!topo) return fail(NUNA_ERR_INVALID_ARG, "topo is NULL");
    const nuna::NapTopology t = nuna::nap_topology_mi355x();
    std::memset(topo, 0, sizeof *topo);
    topo->num_domains = t.domains;
    topo->cus_per_domain = t.cus_per_domain;
    topo->num_stacks = t.stacks;
    topo->cu_budget = t.cu_budget;
    topo->stack_budget = t.stack_budget;
    std::memcpy(topo->stack_pref, t.stack_pref, sizeof t.stack_pref);
    return ok();
}

nuna_status_t nuna_nap_plan(const nuna_nap_topology_t* topo, int nar_max, int64_t num_tb,
                            const int64_t* chunk_offsets, const int64_t* chunk_ids, const int64_t* tb_bytes,
                            const int64_t* chunk_pages, int64_t* tb_group, int32_t* tb_domain, int32_t* tb_cu,
                            int32_t* entry_stack, int64_t* num_groups) try {
    if (!topo) return fail(NUNA_ERR_INVALID_ARG, "topo is NULL");
    if (topo->num_domains < 1 || topo->num_domains > NUNA_NAP_MAX_DOMAINS || topo->cus_per_domain < 1 ||
        topo->cus_per_domain > (1 << 16) || topo->num_stacks < 1 || topo->num_stacks > NUNA_NAP_MAX_STACKS)
        return fail(NUNA_ERR_INVALID_ARG, "invalid topology (domains %d, CUs per domain %d, stacks %d)",
                    topo->num_domains, topo->cus_per_domain, topo->num_stacks);
    for (int d = 0; d < topo->num_domains; ++d) {
        uint32_t seen = 0;
        for (int k = 0; k < topo->num_stacks; ++k) {
            const int s = topo->stack_pref[d][k];
            if (s < 0 || s >= topo->num_stacks || (seen >> s & 1u))
                return fail(NUNA_ERR_INVALID_ARG, "stack_pref[%d] is not a permutation of the %d stacks", d,
                            topo->num_stacks);
            seen |= 1u << s;
        }
    }
    if (nar_max < 1 || topo->num_domains % nar_max != 0)
        return fail(NUNA_ERR_INVALID_ARG, "nar_max=%d does not divide the %d domains", nar_max, topo->num_domains);
    if (num_tb < 0 || num_tb > (int64_t(1) << 40)) return fail(NUNA_ERR_INVALID_ARG, "num_tb=%lld", (long long)num_tb);
    if (num_tb > 0) {
        if (!chunk_offsets || !tb_bytes) return fail(NUNA_ERR_INVALID_ARG, "chunk_offsets or tb_bytes is NULL");
        if (chunk_offsets[0] != 0) return fail(NUNA_ERR_INVALID_ARG, "chunk_offsets[0] != 0");
        for (int64_t t = 0; t < num_tb; ++t) {
            if (chunk_offsets[t + 1] < chunk_offsets[t])
                return fail(NUNA_ERR_INVALID_ARG, "chunk_offsets decrease at %lld", (long long)t);
            if (tb_bytes[t] < 0) return fail(NUNA_ERR_INVALID_ARG, "tb_bytes[%lld] < 0", (long long)t);
        }
        if (chunk_offsets[num_tb] > 0 && !chunk_ids) return fail(NUNA_ERR_INVALID_ARG, "chunk_ids is NULL");
    }
    nuna::NapTopology t{};
    t.domains = topo->num_domains;
    t.cus_per_domain = topo->cus_per_domain;
    t.stacks = topo->num_stacks;
    t.cu_budget = topo->cu_budget;
    t.stack_budget = topo->stack_budget;
    std::memcpy(t.stack_pref, topo->stack_pref, sizeof t.stack_pref);
    const nuna::NapPlan p = nuna::nap_plan(t, nar_max, num_tb, chunk_offsets, chunk_ids, tb_bytes, chunk_pages);
    for (int64_t i = 0; i < num_tb; ++i) {
        if (tb_group) tb_group[i] = p.tb_group[static_cast<size_t>(i)];
        if (tb_domain) tb_domain[i] = p.tb_domain[static_cast<size_t>(i)];
        if (tb_cu) tb_cu[i] = p.tb_cu[static_cast<size_t>(i)];
    }
    if (entry_stack)
        for (size_t e = 0; e < p.entry_stack.size(); ++e) entry_stack[e] = p.entry_stack[e];
    if (num_groups) *num_groups = static_cast<int64_t>(p.groups.size());
    return ok();
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_placement_items(nuna_placement_t place, int64_t b, int64_t G, int64_t groups, int64_t group_size,
                                   int64_t* items, int64_t capacity, int64_t* count) try {
    if (!valid_place(place)) return fail(NUNA_ERR_INVALID_ARG, "invalid placement mode %d", static_cast<int>(place));
    if (!count || (capacity > 0 && !items) || capacity < 0) return fail(NUNA_ERR_INVALID_ARG, "bad output buffer");
    if (G < 1 || b < 0 || b >= G || groups < 0 || group_size < 1 || group_size > (1 << 20) ||
        groups > (int64_t(1) << 40) || G > (int64_t(1) << 31))
        return fail(NUNA_ERR_INVALID_ARG, "invalid geometry b=%lld G=%lld groups=%lld group_size=%lld",
                    static_cast<long long>(b), static_cast<long long>(G), static_cast<long long>(groups),
                    static_cast<long long>(group_size));
    const nuna::Place pl = nuna::make_place_uniform(place, groups, group_size);
    const nuna::ItemRange r = nuna::items_of(pl, b, G);
    int64_t n = 0;
    for (int64_t i = r.first; i < r.end; i += r.stride, ++n)
        if (n < capacity) items[n] = nuna::item_at(pl, b, G, i);
    *count = n;
    if (n > capacity) return fail(NUNA_ERR_INVALID_ARG, "capacity %lld < %lld items", static_cast<long long>(capacity),
                                  static_cast<long long>(n));
    return ok();
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_placement_direct(nuna_placement_t place, int64_t items, int64_t chunk_bytes, int64_t* item_of,
                                    int64_t capacity, int64_t* workgroups) try {
    if (!valid_place(place)) return fail(NUNA_ERR_INVALID_ARG, "invalid placement mode %d", static_cast<int>(place));
    if (!workgroups || (capacity > 0 && !item_of) || capacity < 0) return fail(NUNA_ERR_INVALID_ARG, "bad output buffer");
    if (items < 1 || items > (int64_t(1) << 40) || chunk_bytes < 16 || chunk_bytes % 16 != 0 ||
        (chunk_bytes & (chunk_bytes - 1)) != 0)
        return fail(NUNA_ERR_INVALID_ARG, "invalid geometry items=%lld chunk_bytes=%lld", (long long)items,
                    (long long)chunk_bytes);
    int gs = 0;
    if (place == NUNA_PLACE_XCD && nuna::tuning().page_groups != 0) gs = nuna::page_shift(chunk_bytes);
    const int64_t G = nuna::page_grid(items, gs);
    *workgroups = G;
    if (G > capacity) return fail(NUNA_ERR_INVALID_ARG, "capacity %lld < %lld workgroups", (long long)capacity,
                                  (long long)G);
    for (int64_t b = 0; b < G; ++b) {
        const int64_t w = nuna::page_item(b, gs);
        item_of[b] = w < items ? w : -1;
    }
    return ok();
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_placement_grid(nuna_placement_t place, int64_t groups, int64_t group_size, int64_t* workgroups) {
    if (!valid_place(place)) return fail(NUNA_ERR_INVALID_ARG, "invalid placement mode %d", static_cast<int>(place));
    if (!workgroups || groups < 0 || group_size < 1 || groups > (int64_t(1) << 40))
        return fail(NUNA_ERR_INVALID_ARG, "invalid geometry");
    *workgroups = nuna::place_grid(nuna::make_place_uniform(place, groups, group_size));
    return ok();
}

nuna_status_t nuna_probe_xcc(int G, int32_t* xcc, int32_t* hw_id, hipStream_t stream) {
    if (G < 1 || G > (1 << 24)) return fail(NUNA_ERR_INVALID_ARG, "G=%d outside [1, 2^24]", G);
    if (!xcc) return fail(NUNA_ERR_INVALID_ARG, "xcc is NULL");
    if ((reinterpret_cast<uintptr_t>(xcc) & 3u) || (reinterpret_cast<uintptr_t>(hw_id) & 3u))
        return fail(NUNA_ERR_MISALIGNED, "probe outputs must be 4-byte aligned");
    return hip_status(nuna::launch_probe_xcc(G, xcc, hw_id, stream), "probe launch");
}

nuna_status_t nuna_probe_load_latency(const void* buf, size_t nbytes, size_t stride, size_t line_offset, int xcd,
                                      uint32_t* cycles, hipStream_t stream) {
    if (!buf || !cycles) return fail(NUNA_ERR_INVALID_ARG, "NULL pointer");
    if ((reinterpret_cast<uintptr_t>(buf) & 3u) || (reinterpret_cast<uintptr_t>(cycles) & 3u))
        return fail(NUNA_ERR_MISALIGNED, "probe buffers must be 4-byte aligned");
    if (stride < 4 || stride % 4 || line_offset % 4 || line_offset + 4 > stride)
        return fail(NUNA_ERR_INVALID_ARG, "need stride >= 4, stride and line_offset multiples of 4, line_offset + 4 <= stride");
    if (xcd < 0 || xcd >= NUNA_NUM_XCD) return fail(NUNA_ERR_INVALID_ARG, "xcd %d outside [0, %d)", xcd, NUNA_NUM_XCD);
    if (nbytes > kMaxBytes) return fail(NUNA_ERR_INVALID_ARG, "nbytes too large");
    const int64_t nblocks = static_cast<int64_t>(nbytes / stride);
    if (nblocks < 1) return fail(NUNA_ERR_INVALID_ARG, "buffer holds no whole block");
    // Warm-up line: the 128-byte line half a block away from the probed one,
    // when the block is large enough for the two to be different lines.
    int64_t warm = -1;
    if (stride >= 256) warm = static_cast<int64_t>(((line_offset / 128 + stride / 256) * 128) % stride);
    return hip_status(nuna::launch_probe_latency(buf, nblocks, static_cast<int64_t>(stride),
                                                 static_cast<int64_t>(line_offset), warm, xcd, cycles, stream),
                      "latency probe launch");
}

nuna_status_t nuna_probe_load_latency_cus(const void* buf, size_t nbytes, size_t stride, int xcd, int32_t* work,
                                          uint32_t* cycles, int32_t* cu_of, hipStream_t stream) {
    if (!buf || !work || !cycles || !cu_of) return fail(NUNA_ERR_INVALID_ARG, "NULL pointer");
    if ((reinterpret_cast<uintptr_t>(buf) & 3u) || (reinterpret_cast<uintptr_t>(work) & 3u) ||
        (reinterpret_cast<uintptr_t>(cycles) & 3u) || (reinterpret_cast<uintptr_t>(cu_of) & 3u))
        return fail(NUNA_ERR_MISALIGNED, "probe buffers must be 4-byte aligned");
    const size_t lines = 2 * static_cast<size_t>(nuna::kProbeCuSlotsMax) * 128;
    if (stride < lines || stride % 128 != 0)
        return fail(NUNA_ERR_INVALID_ARG, "stride %zu: need a multiple of 128 of at least %zu bytes (two lines per slot)",
                    stride, lines);
    if (xcd < 0 || xcd >= NUNA_NUM_XCD) return fail(NUNA_ERR_INVALID_ARG, "xcd %d outside [0, %d)", xcd, NUNA_NUM_XCD);
    if (nbytes > kMaxBytes) return fail(NUNA_ERR_INVALID_ARG, "nbytes too large");
    const int64_t nblocks = static_cast<int64_t>(nbytes / stride);
    if (nblocks < 1) return fail(NUNA_ERR_INVALID_ARG, "buffer holds no whole block");
    return hip_status(nuna::launch_probe_latency_cus(buf, nblocks, static_cast<int64_t>(stride), xcd, work, cycles,
                                                     cu_of, stream),
                      "per-CU latency probe launch");
}

nuna_status_t nuna_ref_stream(nuna_ref_t kind, const void* const* src, void* const* dst, int n, size_t bytes,
                              hipStream_t stream) try {
    begin_launches();
    if (kind != NUNA_REF_READ && kind != NUNA_REF_WRITE && kind != NUNA_REF_COPY)
        return fail(NUNA_ERR_INVALID_ARG, "invalid reference stream kind %d", static_cast<int>(kind));
    if (n != 1 && n != 2 && n != 4 && n != 8 && n != 16)
        return fail(NUNA_ERR_INVALID_ARG, "n=%d: reference streams take 1, 2, 4, 8 or 16 buffers", n);
    if (bytes % 16 != 0) return fail(NUNA_ERR_INVALID_ARG, "bytes %zu is not a multiple of 16", bytes);
    if (bytes > kRefMaxBytes) return fail(NUNA_ERR_INVALID_ARG, "bytes %zu too large", bytes);
    nuna_status_t st;
    if (kind != NUNA_REF_WRITE && (st = check_ptr_array(src, n, "src"))) return st;
    if ((st = check_ptr_array(const_cast<const void* const*>(dst), kind == NUNA_REF_READ ? 1 : n, "dst"))) return st;
    if (bytes == 0) return ok();
    SpanSet is, os;
    if (kind != NUNA_REF_WRITE)
        for (int r = 0; r < n; ++r) is.add(src[r], bytes, r);
    if (kind == NUNA_REF_READ) {
        const size_t item = static_cast<size_t>(n >= 8 ? 1 : 8 / n) * 4096;  // read item: 8/n blocks of 4 KiB
        os.add(dst[0], (bytes + item - 1) / item * 16, 0);
    }
    else
        for (int r = 0; r < n; ++r) os.add(dst[r], bytes, r);
    if ((st = check_overlaps(is, os, [](const Span&, const Span&) { return false; }))) return st;
    return hip_status(nuna::launch_ref_stream(static_cast<int>(kind), src, dst, n, bytes, stream),
                      "reference stream launch");
} catch (...) {
    return host_exception();
}

nuna_status_t nuna_copy(void* dst, const void* src, size_t bytes, hipStream_t stream) {
    if (!dst || !src) return fail(NUNA_ERR_INVALID_ARG, "NULL pointer");
    if (!aligned16(dst) || !aligned16(src)) return fail(NUNA_ERR_MISALIGNED, "copy pointers must be 16-byte aligned");
    if (bytes > kMaxBytes) return fail(NUNA_ERR_INVALID_ARG, "bytes %zu too large", bytes);
    if (bytes == 0) return ok();
    const uintptr_t d = reinterpret_cast<uintptr_t>(dst), s = reinterpret_cast<uintptr_t>(src);
    if (d < s + bytes && s < d + bytes) return fail(NUNA_ERR_OVERLAP, "copy source and destination overlap");
    return hip_status(nuna::launch_copy(dst, src, bytes, stream), "copy launch");
}

}  // extern "C"
