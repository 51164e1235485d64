// nap_planner.cpp -- Algorithm 1 (NUNA-aware placement) on the host.
#include "nap_planner.h"

#include <algorithm>
#include <unordered_map>

namespace nuna {

NapTopology nap_topology_mi355x() {
    NapTopology t{};
    t.domains = 8;
    t.cus_per_domain = 32;
    t.stacks = 8;
    t.cu_budget = 700 * 128;     // outstanding requests per CU x 128-byte lines
    t.stack_budget = 1 << 20;    // about 1 TB/s per stack x 1 us
    for (int x = 0; x < 8; ++x) {
        const int die = x / 4;
        int k = 0;
        t.stack_pref[x][k++] = x;
        for (int s = 4 * die; s < 4 * die + 4; ++s)
            if (s != x) t.stack_pref[x][k++] = s;
        for (int s = 0; s < 8; ++s)
            if (s / 4 != die) t.stack_pref[x][k++] = s;
    }
    return t;
}

NapPlan nap_plan(const NapTopology& topo, int nar_max, int64_t num_tb, const int64_t* offsets, const int64_t* chunks,
                 const int64_t* tb_bytes, const int64_t* pages) {
    NapPlan p;
    p.tb_group.assign(static_cast<size_t>(num_tb), -1);
    p.tb_domain.assign(static_cast<size_t>(num_tb), -1);
    p.tb_cu.assign(static_cast<size_t>(num_tb), -1);
    const int64_t nent = num_tb > 0 ? offsets[num_tb] : 0;
    p.entry_stack.assign(static_cast<size_t>(nent), -1);

    // Logical allocation.
    std::unordered_map<int64_t, int64_t> chunk_group;
    chunk_group.reserve(static_cast<size_t>(nent));
    std::vector<std::pair<int64_t, int64_t>> shared;  // (group, count)
    for (int64_t tb = 0; tb < num_tb; ++tb) {
        shared.clear();
        for (int64_t e = offsets[tb]; e < offsets[tb + 1]; ++e) {
            auto it = chunk_group.find(chunks[e]);
            if (it == chunk_group.end()) continue;
            auto s = std::find_if(shared.begin(), shared.end(), [&](const auto& q) { return q.first == it->second; });
            if (s == shared.end())
                shared.emplace_back(it->second, 1);
            else
                ++s->second;
        }
        int64_t g;
        if (shared.empty()) {
            g = static_cast<int64_t>(p.groups.size());
            p.groups.emplace_back();
        } else {
            g = shared[0].first;
            int64_t best = shared[0].second;
            for (const auto& q : shared)
                if (q.second > best || (q.second == best && q.first < g)) {
                    g = q.first;
                    best = q.second;
                }
        }
        p.groups[static_cast<size_t>(g)].push_back(tb);
        p.tb_group[static_cast<size_t>(tb)] = g;
        for (int64_t e = offsets[tb]; e < offsets[tb + 1]; ++e) chunk_group.emplace(chunks[e], g);
    }
    const int64_t ngroups = static_cast<int64_t>(p.groups.size());
    p.group_order.resize(static_cast<size_t>(ngroups));
    for (int64_t g = 0; g < ngroups; ++g) p.group_order[static_cast<size_t>(g)] = g;
    std::stable_sort(p.group_order.begin(), p.group_order.end(), [&](int64_t a, int64_t b) {
        return p.groups[static_cast<size_t>(a)].size() > p.groups[static_cast<size_t>(b)].size();
    });

    // Physical placement.
    const int per = topo.domains / nar_max;
    const int span = per * topo.cus_per_domain;
    std::vector<int64_t> r_cu(static_cast<size_t>(topo.domains) * topo.cus_per_domain, topo.cu_budget);
    std::vector<int64_t> r_st(static_cast<size_t>(topo.stacks), topo.stack_budget);
    std::unordered_map<int64_t, int32_t> chunk_stack, page_stack;
    chunk_stack.reserve(static_cast<size_t>(nent));
    for (int64_t i = 0; i < ngroups; ++i) {
        const int nar = static_cast<int>(i % nar_max);
        const int lo = nar * span;
        for (int64_t tb : p.groups[static_cast<size_t>(p.group_order[static_cast<size_t>(i)])]) {
            const int64_t cs = tb_bytes[tb];
            int cu = -1;
            for (int c = lo; c < lo + span; ++c)
                if (r_cu[static_cast<size_t>(c)] >= cs) {
                    cu = c;
                    break;
                }
            if (cu < 0) {
                cu = lo;
                for (int c = lo; c < lo + span; ++c)
                    if (r_cu[static_cast<size_t>(c)] > r_cu[static_cast<size_t>(cu)]) cu = c;
            }
            const int32_t* pref = topo.stack_pref[cu / topo.cus_per_domain];
            int stack = -1;
            for (int k = 0; k < topo.stacks; ++k)
                if (r_st[static_cast<size_t>(pref[k])] >= cs) {
                    stack = pref[k];
                    break;
                }
            if (stack < 0) stack = pref[0];
            r_cu[static_cast<size_t>(cu)] -= cs;
            r_st[static_cast<size_t>(stack)] -= cs;
            p.tb_domain[static_cast<size_t>(tb)] = nar;
            p.tb_cu[static_cast<size_t>(tb)] = cu;
            for (int64_t e = offsets[tb]; e < offsets[tb + 1]; ++e) {
                if (chunk_stack.count(chunks[e])) continue;
                int32_t s = stack;
                if (pages) s = page_stack.emplace(pages[e], stack).first->second;
                chunk_stack.emplace(chunks[e], s);
            }
        }
    }
    for (int64_t e = 0; e < nent; ++e) p.entry_stack[static_cast<size_t>(e)] = chunk_stack[chunks[e]];
    return p;
}

}  // namespace nuna
