// nap_planner.h -- host planner for NUNA-aware placement (Algorithm 1,
// Sec. 4.2.2 of the paper): threadblocks and the chunks they touch in,
// threadblock -> (logical group, NAR domain, CU) and chunk -> HBM stack out.
// The implementation runs four passes (form groups, rank them, place
// threadblocks under budgets, home chunks); the rules they apply:
//
// Logical allocation: threadblocks are taken in the given order; one whose
// chunks belong to no group starts a group, otherwise it joins the group it
// shares the most chunks with (ties: the group created first) and brings its
// unassigned chunks along.  Groups are then ordered by decreasing number of
// threadblocks (stable).
//
// Physical placement: the i-th group of that order goes to NAR domain
// i mod nar_max.  NAR domain n spans the physical domains
// [n*D/nar_max, (n+1)*D/nar_max) and their CUs in order.  Each threadblock of
// the group takes the first of those CUs whose remaining budget covers its
// bytes (none: the first CU with the most budget left), and a stack: the
// first in its physical domain's preference order whose remaining budget
// covers them (none: the most preferred).  Both budgets are charged.  A chunk
// lives on the stack chosen for the first threadblock placed that touches
// it; with pages given, a page's stack is fixed by its first chunk.
#pragma once

#include <stdint.h>

#include <vector>

namespace nuna {

constexpr int kNapMaxDomains = 16;
constexpr int kNapMaxStacks = 16;

struct NapTopology {
    int domains;
    int cus_per_domain;
    int stacks;
    int64_t cu_budget;
    int64_t stack_budget;
    int32_t stack_pref[kNapMaxDomains][kNapMaxStacks];
};

struct NapPlan {
    std::vector<int64_t> tb_group;   // group index in creation order
    std::vector<int32_t> tb_domain;  // NAR domain
    std::vector<int32_t> tb_cu;      // physical domain * cus_per_domain + CU within it
    std::vector<int32_t> tb_stack;     // stack charged for each threadblock
    std::vector<int32_t> entry_stack;  // stack of each (threadblock, chunk) entry's chunk
    std::vector<int64_t> group_order;  // group indices in placement order (decreasing size)
    std::vector<std::vector<int64_t>> groups;  // members of each group, in joining order
};

// MI355X: 8 XCDs of 32 CUs, 8 HBM stacks; XCDs 0-3 and stacks 0-3 on one I/O
// die, 4-7 on the other.  XCD x prefers stack x, then the other stacks of its
// die, then the far die's, each in index order.
NapTopology nap_topology_mi355x();

// Inputs are assumed valid (checked by the C ABI): nar_max divides
// topo.domains; offsets[0] == 0, offsets non-decreasing.
NapPlan nap_plan(const NapTopology& topo, int nar_max, int64_t num_tb, const int64_t* offsets, const int64_t* chunks,
                 const int64_t* tb_bytes, const int64_t* pages);

}  // namespace nuna
