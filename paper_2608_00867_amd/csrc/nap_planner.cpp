// nap_planner.cpp -- NUNA-aware placement (Sec. 4.2.2) on the host, in four
// passes over a threadblock workload:
//
//   1. form_groups     logical allocation: threadblocks that share data chunks
//                      end up in one group (Sec. 4.2.1);
//   2. rank_groups     groups in decreasing size, creation order among equals;
//   3. place           groups dealt round-robin to the NAR domains, each
//                      threadblock given a CU of its domain and an HBM stack
//                      under the request budgets (BudgetPool);
//   4. home_chunks     every chunk (or page) homed on the stack of the first
//                      threadblock placed that touches it.
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

namespace {

// Pass 1.  A threadblock joins the group holding the most of its chunk entries
// (ties: the older group) or, sharing none, opens a new group; its chunks not
// yet in a group join the one it lands in.
void form_groups(int64_t num_tb, const int64_t* offsets, const int64_t* chunks, NapPlan& p) {
    std::unordered_map<int64_t, int64_t> owner;  // chunk -> group
    owner.reserve(num_tb > 0 ? static_cast<size_t>(offsets[num_tb]) : 0);
    std::unordered_map<int64_t, int64_t> votes;  // group -> shared entries of the current threadblock
    for (int64_t tb = 0; tb < num_tb; ++tb) {
        votes.clear();
        for (int64_t e = offsets[tb]; e < offsets[tb + 1]; ++e) {
            const auto it = owner.find(chunks[e]);
            if (it != owner.end()) ++votes[it->second];
        }
        int64_t g = static_cast<int64_t>(p.groups.size());
        int64_t most = 0;
        for (const auto& v : votes)
            if (v.second > most || (v.second == most && v.first < g)) {
                g = v.first;
                most = v.second;
            }
        if (g == static_cast<int64_t>(p.groups.size())) p.groups.emplace_back();
        p.groups[static_cast<size_t>(g)].push_back(tb);
        p.tb_group[static_cast<size_t>(tb)] = g;
        for (int64_t e = offsets[tb]; e < offsets[tb + 1]; ++e) owner.emplace(chunks[e], g);
    }
}

// Pass 2.
void rank_groups(NapPlan& p) {
    p.group_order.resize(p.groups.size());
    for (size_t g = 0; g < p.groups.size(); ++g) p.group_order[g] = static_cast<int64_t>(g);
    std::stable_sort(p.group_order.begin(), p.group_order.end(), [&](int64_t a, int64_t b) {
        return p.groups[static_cast<size_t>(a)].size() > p.groups[static_cast<size_t>(b)].size();
    });
}

// Remaining request budgets (R in Sec. 4.2.2) of a set of resources.
class BudgetPool {
  public:
    BudgetPool(size_t n, int64_t each) : left_(n, each) {}

    // The first resource of `cands` whose remaining budget covers `need`;
    // if none does, `fallback(cands)`.
    template <class Cands, class Fallback>
    int pick(const Cands& cands, int64_t need, Fallback fallback) const {
        for (int r : cands)
            if (left_[static_cast<size_t>(r)] >= need) return r;
        return fallback(cands);
    }
    int64_t left(int r) const { return left_[static_cast<size_t>(r)]; }
    void charge(int r, int64_t bytes) { left_[static_cast<size_t>(r)] -= bytes; }

  private:
    std::vector<int64_t> left_;
};

// The CUs of one NAR domain, in index order.
struct CuRange {
    int lo, hi;
    struct It {
        int v;
        int operator*() const { return v; }
        It& operator++() {
            ++v;
            return *this;
        }
        bool operator!=(const It& o) const { return v != o.v; }
    };
    It begin() const { return {lo}; }
    It end() const { return {hi}; }
};

// Pass 3.  Group order[i] goes to NAR domain i mod nar_max (Sec. 4.2.2: the
// next domain for every group); a threadblock takes the first CU of its
// domain with budget for it (none: the CU with the most budget left) and the
// first stack in its physical domain's preference order with budget (none:
// the preferred stack).
void place(const NapTopology& topo, int nar_max, const int64_t* tb_bytes, NapPlan& p) {
    const int span = topo.domains / nar_max * topo.cus_per_domain;
    BudgetPool cus(static_cast<size_t>(topo.domains) * topo.cus_per_domain, topo.cu_budget);
    BudgetPool stacks(static_cast<size_t>(topo.stacks), topo.stack_budget);
    p.tb_stack.assign(p.tb_group.size(), -1);
    for (size_t i = 0; i < p.group_order.size(); ++i) {
        const int nar = static_cast<int>(i % static_cast<size_t>(nar_max));
        const CuRange domain{nar * span, nar * span + span};
        for (int64_t tb : p.groups[static_cast<size_t>(p.group_order[i])]) {
            const int64_t need = tb_bytes[tb];
            const int cu = cus.pick(domain, need, [&](const CuRange& r) {
                int best = r.lo;
                for (int c : r)
                    if (cus.left(c) > cus.left(best)) best = c;
                return best;
            });
            const int32_t* pref = topo.stack_pref[cu / topo.cus_per_domain];
            const std::vector<int> order(pref, pref + topo.stacks);
            const int stack = stacks.pick(order, need, [](const std::vector<int>& o) { return o[0]; });
            cus.charge(cu, need);
            stacks.charge(stack, need);
            p.tb_domain[static_cast<size_t>(tb)] = nar;
            p.tb_cu[static_cast<size_t>(tb)] = cu;
            p.tb_stack[static_cast<size_t>(tb)] = stack;
        }
    }
}

// Pass 4.  In placement order, a chunk not yet homed takes the stack of the
// threadblock touching it; with pages, the page is homed by its first chunk
// and every later chunk of the page follows it.
void home_chunks(const int64_t* offsets, const int64_t* chunks, const int64_t* pages, NapPlan& p) {
    std::unordered_map<int64_t, int32_t> chunk_home, page_home;
    for (int64_t g : p.group_order)
        for (int64_t tb : p.groups[static_cast<size_t>(g)])
            for (int64_t e = offsets[tb]; e < offsets[tb + 1]; ++e) {
                if (chunk_home.count(chunks[e])) continue;
                int32_t s = p.tb_stack[static_cast<size_t>(tb)];
                if (pages) s = page_home.emplace(pages[e], s).first->second;
                chunk_home.emplace(chunks[e], s);
            }
    for (size_t e = 0; e < p.entry_stack.size(); ++e) p.entry_stack[e] = chunk_home[chunks[e]];
}

}  // namespace

NapPlan nap_plan(const NapTopology& topo, int nar_max, int64_t num_tb, const int64_t* offsets, const int64_t* chunks,
                 const int64_t* tb_bytes, const int64_t* pages) {
    NapPlan p;
    p.tb_group.assign(static_cast<size_t>(num_tb), -1);
    p.tb_domain.assign(static_cast<size_t>(num_tb), -1);
    p.tb_cu.assign(static_cast<size_t>(num_tb), -1);
    p.entry_stack.assign(num_tb > 0 ? static_cast<size_t>(offsets[num_tb]) : 0, -1);
    form_groups(num_tb, offsets, chunks, p);
    rank_groups(p);
    place(topo, nar_max, tb_bytes, p);
    home_chunks(offsets, chunks, pages, p);
    return p;
}

}  // namespace nuna
