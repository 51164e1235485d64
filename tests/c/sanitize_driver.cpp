// sanitize_driver.cpp -- drives libnuna's host code through its C ABI under
// AddressSanitizer and UndefinedBehaviorSanitizer (built with the HIP stand-in
// of hip_host_stub.cpp, no GPU).  Seeded random calls cover argument checks
// with overlapping, misaligned, null and oversized buffers, every tunable, the
// all-to-all layout builder with its upload, dispatch and combine tables, the
// placement planner, the placement mirrors and the dispatch-map check.  The
// data pointers are made up and never dereferenced; the tables the host builds
// are read end to end by the launch stubs.  Exit status 0 means every call
// returned a valid status, no stub check failed and the sanitizers reported
// nothing (they abort the process on their first report).
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "nuna.h"

extern "C" int stub_failures(void);

namespace {

uint64_t g_rng = 0x9E3779B97F4A7C15ull;

uint64_t rnd() {
    g_rng ^= g_rng << 13;
    g_rng ^= g_rng >> 7;
    g_rng ^= g_rng << 17;
    return g_rng;
}

int64_t rnd_in(int64_t lo, int64_t hi) { return lo + static_cast<int64_t>(rnd() % static_cast<uint64_t>(hi - lo + 1)); }

int g_bad = 0;

void expect(bool ok, const char* what, int st) {
    if (!ok) {
        std::fprintf(stderr, "driver: %s (status %d: %s)\n", what, st, nuna_last_error_string());
        ++g_bad;
    }
}

bool valid_status(int st) { return st >= NUNA_OK && st <= NUNA_ERR_NO_MEMORY; }

// Made-up device addresses: 16-byte aligned unless asked otherwise, spread so
// that most sets do not overlap; a few overlap on purpose.
void* fake(uint64_t base, int64_t off) { return reinterpret_cast<void*>(static_cast<uintptr_t>(base + off)); }

void collective_fuzz(int iters) {
    std::vector<const void*> in(70);
    std::vector<void*> out(70);
    for (int it = 0; it < iters; ++it) {
        const int P = static_cast<int>(rnd_in(-1, 66));
        const int op = static_cast<int>(rnd_in(0, 2));
        const int dtype = static_cast<int>(rnd_in(-1, 2));
        const int algo = static_cast<int>(rnd_in(-1, 5));
        const int place = static_cast<int>(rnd_in(-1, 2));
        size_t count;
        switch (rnd() % 6) {
            case 0: count = 0; break;
            case 1: count = static_cast<size_t>(rnd_in(1, 100)); break;
            case 2: count = static_cast<size_t>(rnd_in(1, 1 << 20)); break;
            case 3: count = size_t(1) << rnd_in(40, 62); break;
            default: count = static_cast<size_t>(rnd_in(1, 1 << 14)) * 64; break;
        }
        const uint64_t stride = uint64_t(1) << rnd_in(4, 40);
        const uint64_t base_in = 0x100000000000ull + (rnd() % 4096) * 16;
        const uint64_t base_out = rnd() % 4 == 0 ? base_in : 0x300000000000ull;
        const int n = P > 0 && P < 70 ? P : 1;
        for (int r = 0; r < n; ++r) {
            in[r] = fake(base_in, static_cast<int64_t>(stride) * r);
            out[r] = fake(base_out, static_cast<int64_t>(stride) * r);
        }
        const int mess = static_cast<int>(rnd() % 8);
        if (mess == 0) in[rnd() % n] = nullptr;
        if (mess == 1) out[rnd() % n] = fake(base_out, static_cast<int64_t>(rnd() % 16));
        if (mess == 2 && n > 1) out[1] = out[0];
        const void* const* ip = rnd() % 50 ? in.data() : nullptr;
        void* const* op_ = rnd() % 50 ? out.data() : nullptr;
        int st;
        if (op == 0)
            st = nuna_allreduce(ip, op_, P, count, static_cast<nuna_dtype_t>(dtype), static_cast<nuna_algo_t>(algo),
                                static_cast<nuna_placement_t>(place), nullptr);
        else if (op == 1)
            st = nuna_reduce_scatter(ip, op_, P, count, static_cast<nuna_dtype_t>(dtype),
                                     static_cast<nuna_placement_t>(place), nullptr);
        else
            st = nuna_all_gather(ip, op_, P, count, static_cast<nuna_dtype_t>(dtype),
                                 static_cast<nuna_placement_t>(place), nullptr);
        expect(valid_status(st), "collective status out of range", st);
        nuna_launch_info_t li;
        expect(nuna_last_launch(&li) == NUNA_OK, "last launch", 0);
        if (st == NUNA_OK && count > 0) expect(li.launches >= 1 && li.kernels[0] != '\0', "launch recorded", st);
        if (st != NUNA_OK) expect(li.launches == 0, "failed call launched", st);
    }
}

void tunable_fuzz() {
    const char* names[] = {"NUNA_MAX_GRID", "NUNA_WG_THREADS", "NUNA_VPT", "NUNA_LPR_MIN_RANKS",
                           "NUNA_LPR_MAX_VECTORS", "NUNA_COMBINE_VPT", "NUNA_COMBINE_CHUNKS", "NUNA_TILE_V",
                           "NUNA_COMBINE_LISTS", "NUNA_WRITE_THROUGH", "NUNA_PAGE_GROUPS", "NUNA_DIRECT_MAX_GRID",
                           "NUNA_TWO_SHOT_FORM", "NUNA_NOT_A_KNOB", nullptr};
    for (const char* name : names) {
        int64_t old = 0;
        const int g = nuna_get_tunable(name, &old);
        for (int k = 0; k < 50; ++k) {
            const int64_t v = rnd() % 3 == 0 ? rnd_in(-10, 300) : static_cast<int64_t>(rnd() >> rnd_in(1, 63));
            const int st = nuna_set_tunable(name, v);
            expect(st == NUNA_OK || st == NUNA_ERR_INVALID_ARG, "tunable status", st);
        }
        if (g == NUNA_OK) expect(nuna_set_tunable(name, old) == NUNA_OK, "tunable restore", 0);
    }
    expect(nuna_set_max_workgroups(-1) == NUNA_ERR_INVALID_ARG, "negative cap", 0);
}

void layout_fuzz(int iters) {
    for (int it = 0; it < iters; ++it) {
        const int P = static_cast<int>(rnd_in(1, 64));
        const int E = P * static_cast<int>(rnd_in(1, 8));
        const int T = static_cast<int>(rnd_in(0, 300));
        const int k = static_cast<int>(rnd_in(1, E < 9 ? E : 9));
        std::vector<int32_t> topk(static_cast<size_t>(P) * T * k);
        for (auto& e : topk) e = static_cast<int32_t>(rnd() % E);
        if (rnd() % 10 == 0 && !topk.empty()) topk[rnd() % topk.size()] = E + 3;  // invalid expert
        nuna_a2a_layout_t* L = nullptr;
        int st = nuna_a2a_layout_create(P, T, k, E, topk.empty() ? nullptr : topk.data(), &L);
        expect(valid_status(st), "layout create status", st);
        if (st != NUNA_OK) {
            expect(L == nullptr, "failed create returned a layout", st);
            continue;
        }
        std::vector<int64_t> rows(P);
        expect(nuna_a2a_layout_recv_rows(L, rows.data()) == NUNA_OK, "recv rows", 0);
        int64_t total = 0, cap = 0;
        for (int d = 0; d < P; ++d) {
            total += rows[d];
            cap = rows[d] > cap ? rows[d] : cap;
            std::vector<int32_t> src(rows[d] + 1), tok(rows[d] + 1);
            expect(nuna_a2a_layout_recv_map(L, d, src.data(), tok.data()) == NUNA_OK, "recv map", 0);
            for (int64_t j = 0; j < rows[d]; ++j)
                expect(src[j] >= 0 && src[j] < P && tok[j] >= 0 && tok[j] < T, "recv map entry", 0);
        }
        expect(total <= static_cast<int64_t>(P) * T * (k < P ? k : P), "routed rows bounded", 0);
        std::vector<const void*> send(P);
        std::vector<void*> recv(P);
        for (int r = 0; r < P; ++r) {
            send[r] = fake(0x100000000000ull, static_cast<int64_t>(r) << 32);
            recv[r] = fake(0x500000000000ull, static_cast<int64_t>(r) << 32);
        }
        const size_t row = static_cast<size_t>(rnd_in(1, 4096)) * (rnd() % 2 ? 8 : 1);
        const nuna_placement_t place = rnd() % 2 ? NUNA_PLACE_XCD : NUNA_PLACE_LINEAR;
        st = nuna_all_to_all(send.data(), recv.data(), L, row, static_cast<size_t>(cap), NUNA_BF16, place, nullptr);
        expect(total == 0 ? st == NUNA_OK : st == NUNA_ERR_INVALID_ARG, "dispatch before upload", st);
        expect(nuna_a2a_layout_upload(L) == NUNA_OK, "upload", 0);
        st = nuna_all_to_all(send.data(), recv.data(), L, row, static_cast<size_t>(cap), NUNA_BF16, place, nullptr);
        expect(st == NUNA_OK, "dispatch", st);
        if (cap > 0) {
            st = nuna_all_to_all(send.data(), recv.data(), L, row, static_cast<size_t>(cap - 1), NUNA_BF16, place,
                                 nullptr);
            expect(st == NUNA_ERR_INVALID_ARG, "dispatch beyond capacity", st);
        }
        const float* w = rnd() % 2 ? static_cast<const float*>(fake(0x700000000000ull, 0)) : nullptr;
        const nuna_dtype_t dt = rnd() % 2 ? NUNA_BF16 : NUNA_F32;
        std::vector<const void*> ys(recv.begin(), recv.end());
        std::vector<void*> outs(P);
        for (int r = 0; r < P; ++r) outs[r] = fake(0x100000000000ull, static_cast<int64_t>(r) << 32);
        st = nuna_all_to_all_combine(ys.data(), outs.data(), L, w, row, static_cast<size_t>(cap), dt, place, nullptr);
        expect(st == NUNA_OK, "combine", st);
        nuna_a2a_layout_destroy(L);
        // The allocation-free dispatch on the same routing (topk_idx is host memory here; the stand-in
        // launcher does not read it).
        std::vector<int64_t> rows_dev(P + 1);
        const size_t rrow = static_cast<size_t>(rnd_in(1, 512)) * 8;
        st = nuna_all_to_all_routed(send.data(), recv.data(), topk.empty() ? nullptr : topk.data(), P, T, k, E, rrow,
                                    static_cast<size_t>(cap), NUNA_BF16, place, rows_dev.data(), nullptr);
        expect(st == NUNA_OK || st == NUNA_ERR_INVALID_ARG, "routed dispatch", st);
    }
    nuna_a2a_layout_destroy(nullptr);
}

void planner_fuzz(int iters) {
    nuna_nap_topology_t topo;
    expect(nuna_nap_topology_mi355x(&topo) == NUNA_OK, "topology", 0);
    for (int it = 0; it < iters; ++it) {
        nuna_nap_topology_t t = topo;
        t.cu_budget = rnd_in(0, 4096);
        t.stack_budget = rnd_in(0, 1 << 16);
        const int64_t ntb = rnd_in(0, 200);
        std::vector<int64_t> off(ntb + 1, 0), ids, bytes(ntb), pages;
        const int64_t pool = rnd_in(1, 64);
        for (int64_t b = 0; b < ntb; ++b) {
            const int64_t nc = rnd_in(0, 6);
            for (int64_t c = 0; c < nc; ++c) ids.push_back(rnd_in(0, pool - 1));
            off[b + 1] = static_cast<int64_t>(ids.size());
            bytes[b] = rnd_in(0, 1024);
        }
        const bool with_pages = rnd() % 2;
        for (int64_t id : ids) pages.push_back(id / 4);  // a chunk keeps one page everywhere
        const int nar = static_cast<int>(1 << rnd_in(0, 3));
        std::vector<int64_t> grp(ntb + 1);
        std::vector<int32_t> dom(ntb + 1), cu(ntb + 1), stk(ids.size() + 1);
        int64_t ng = -1;
        const int st = nuna_nap_plan(&t, rnd() % 20 ? nar : 3, ntb, off.data(), ids.empty() ? nullptr : ids.data(),
                                     bytes.data(), with_pages && !ids.empty() ? pages.data() : nullptr, grp.data(),
                                     dom.data(), cu.data(), stk.data(), &ng);
        expect(valid_status(st), "planner status", st);
        if (st != NUNA_OK) continue;
        for (int64_t b = 0; b < ntb; ++b)
            expect(grp[b] >= 0 && grp[b] < ng && dom[b] >= 0 && dom[b] < nar && cu[b] >= 0 && cu[b] < 256,
                   "plan entry", st);
        for (size_t e = 0; e < ids.size(); ++e) expect(stk[e] >= 0 && stk[e] < 8, "plan stack", st);
    }
}

void placement_fuzz(int iters) {
    std::vector<int64_t> items(1 << 16);
    for (int it = 0; it < iters; ++it) {
        const nuna_placement_t place = rnd() % 2 ? NUNA_PLACE_XCD : NUNA_PLACE_LINEAR;
        const int64_t groups = rnd_in(0, 3000), gs = rnd_in(1, 9);
        int64_t G = 0, cnt = 0;
        expect(nuna_placement_grid(place, groups, gs, &G) == NUNA_OK, "grid", 0);
        if (G < 1) continue;
        const int64_t b = rnd_in(0, G - 1);
        const int st = nuna_placement_items(place, b, G, groups, gs, items.data(), static_cast<int64_t>(items.size()),
                                            &cnt);
        expect(st == NUNA_OK, "items", st);
        for (int64_t i = 0; i < cnt; ++i) expect(items[i] >= 0 && items[i] < groups * gs, "item range", 0);
        const int64_t n = rnd_in(1, 20000), cb = int64_t(16) << rnd_in(0, 9);
        int64_t wg = 0;
        const int pg = nuna_set_tunable("NUNA_PAGE_GROUPS", static_cast<int64_t>(rnd() % 2));
        expect(pg == NUNA_OK, "page groups tunable", pg);
        const int s2 = nuna_placement_direct(place, n, cb, items.data(), static_cast<int64_t>(items.size()), &wg);
        expect(s2 == NUNA_OK || (s2 == NUNA_ERR_INVALID_ARG && wg > static_cast<int64_t>(items.size())), "direct",
               s2);
        if (s2 == NUNA_OK)
            for (int64_t w = 0; w < wg; ++w) expect(items[w] >= -1 && items[w] < n, "direct item range", 0);
    }
    expect(nuna_set_tunable("NUNA_PAGE_GROUPS", 0) == NUNA_OK, "page groups restore", 0);
}

void map_check_fuzz(int iters) {
    std::vector<int32_t> x(4096);
    for (int it = 0; it < iters; ++it) {
        const int64_t G = rnd_in(0, 4096);
        for (int64_t b = 0; b < G; ++b) x[b] = static_cast<int32_t>(rnd() % 3 ? b % 8 : rnd() % 16);
        const int st = nuna_check_dispatch_map(x.data(), G, rnd() % 4 ? 256 : static_cast<int32_t>(rnd_in(0, 400)));
        expect(st == NUNA_OK || st == NUNA_ERR_UNSUPPORTED || st == NUNA_ERR_INVALID_ARG, "map check", st);
    }
}

}  // namespace

int main() {
    int st = nuna_init();
    expect(st == NUNA_OK, "init with the stand-in runtime", st);
    nuna_device_info_t info;
    st = nuna_get_device_info(&info);
    expect(st == NUNA_OK && info.map_verified == 1 && info.cu_count == 256 && info.xcd_count == 8, "device info", st);
    collective_fuzz(30000);
    tunable_fuzz();
    layout_fuzz(300);
    planner_fuzz(400);
    placement_fuzz(400);
    map_check_fuzz(300);
    int32_t probe[64];
    expect(nuna_probe_xcc(0, probe, nullptr, nullptr) == NUNA_ERR_INVALID_ARG, "probe G=0", 0);
    expect(nuna_copy(nullptr, probe, 16, nullptr) == NUNA_ERR_INVALID_ARG, "copy null", 0);
    {
        // NUNA_ALGO_AUTO: the two-shot for 8 ranks of bf16 from 16 MiB per rank, the one-shot below and for
        // other rank counts, dtypes and ragged shards (the launch stubs touch no buffer: made-up addresses).
        const void* in[8];
        void* out[8];
        const uintptr_t base = uintptr_t(1) << 44;
        for (int r = 0; r < 8; ++r) {
            in[r] = reinterpret_cast<const void*>(base + (uintptr_t(2 * r) << 28));
            out[r] = reinterpret_cast<void*>(base + (uintptr_t(2 * r + 1) << 28));
        }
        struct Case { int P; size_t count; nuna_dtype_t dt; const char* kernel; };
        const Case cases[] = {{8, size_t(8) << 20, NUNA_BF16, "stub_two_shot"},
                              {8, size_t(32) << 20, NUNA_BF16, "stub_two_shot"},
                              {8, (size_t(8) << 20) - 64, NUNA_BF16, "stub_allreduce"},
                              {8, (size_t(8) << 20) + 4, NUNA_BF16, "stub_allreduce"},
                              {8, size_t(4) << 20, NUNA_F32, "stub_allreduce"},
                              {4, size_t(8) << 20, NUNA_BF16, "stub_allreduce"}};
        for (const Case& c : cases) {
            const int st = nuna_allreduce(in, out, c.P, c.count, c.dt, NUNA_ALGO_AUTO, NUNA_PLACE_LINEAR, nullptr);
            nuna_launch_info_t li;
            nuna_last_launch(&li);
            expect(st == NUNA_OK && std::strcmp(li.kernels, c.kernel) == 0, "AUTO algorithm choice",
                   static_cast<int>(c.count >> 10));
        }
    }
    {
        // Reference streams: every kind at every buffer count through the launch stub, and refusals.
        static unsigned char pool[32 * 8192 + 16] __attribute__((aligned(16)));
        const void* src[16];
        void* dst[16];
        for (int r = 0; r < 16; ++r) {
            src[r] = pool + r * 8192;
            dst[r] = pool + (16 + r) * 8192;
        }
        for (int kind = 0; kind < 3; ++kind)
            for (int n : {1, 2, 4, 8, 16})
                expect(nuna_ref_stream(static_cast<nuna_ref_t>(kind), src, dst, n, 8192, nullptr) == NUNA_OK,
                       "reference stream", kind * 100 + n);
        expect(nuna_ref_stream(NUNA_REF_COPY, src, dst, 3, 8192, nullptr) == NUNA_ERR_INVALID_ARG, "ref n=3", 0);
        void* src_as_dst[16];
        for (int r = 0; r < 16; ++r) src_as_dst[r] = pool + r * 8192;
        expect(nuna_ref_stream(NUNA_REF_COPY, src, src_as_dst, 2, 8192, nullptr) == NUNA_ERR_OVERLAP, "ref overlap",
               0);
        expect(nuna_ref_stream(NUNA_REF_WRITE, nullptr, dst, 16, 8192 + 16, nullptr) == NUNA_ERR_OVERLAP,
               "ref write overlap", 0);
    }
    const int sf = stub_failures();
    std::printf("sanitize driver: %d failed expectations, %d failed launch checks\n", g_bad, sf);
    return g_bad == 0 && sf == 0 ? 0 : 1;
}
