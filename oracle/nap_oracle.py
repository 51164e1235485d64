"""NUNA-aware placement (Algorithm 1 of the paper) in plain Python -- TEST INFRASTRUCTURE ONLY.

Only ``tests/`` may import this module.  The library's planner (C++, host side)
is checked against it entry by entry; the two share no code.

Algorithm 1 (Sec. 4.2.2, "NUNA-Aware Placement") takes a collective's
threadblocks with the chunks each one touches and produces two maps:
threadblock -> CU and chunk -> HBM stack.  It runs in two phases:

* logical allocation (Sec. 4.2.2, "Logical Allocation"): threadblocks are
  taken in the order given.  A threadblock none of whose chunks belongs to a
  group starts a new group.  Otherwise it joins the existing group with which
  it shares the most chunks, and its chunks that belong to no group join that
  group too.  The groups are then sorted by decreasing size.
* physical placement (Sec. 4.2.2, "Physical Placement"): groups are dealt
  round-robin to the NAR domains.  Each threadblock of a group, in turn, goes
  to the first CU of the domain whose remaining budget fits the threadblock's
  chunk bytes, and its chunks to a stack, preferring the CU's nearest stack.
  Both budgets are then charged.  A page's stack is fixed by the first chunk
  placed in it (first come, first served).

Readings where the paper leaves a choice (each one also listed with the
library's planner):

* Group size is the number of threadblocks in the group; the sort is stable
  (equal sizes keep creation order).
* A tie between groups sharing equally many chunks goes to the group created
  first.
* The domain counter starts so that the first group lands in domain 0 (the
  paper's figure deals groups to domains 0, 1, 2, ...).
* NAR domain n of nar_max covers the CUs of the physical domains
  [n*D/nar_max, (n+1)*D/nar_max) in order (D physical domains, nar_max
  divides D); its CUs are tried in that order.
* When no CU of the domain fits, the threadblock goes to the domain's CU with
  the largest remaining budget (the first such CU); budgets may go negative.
* The stack is the first stack in the CU's preference order whose remaining
  budget fits; when none fits, the CU's nearest stack.
* A chunk touched by several threadblocks takes the stack chosen for the first
  of them (first come, first served, in placement order); with pages given,
  the same holds per page.
"""


def logical_allocation(tb_chunks):
    """tb_chunks: list (one per threadblock, in the given order) of lists of chunk ids.
    Returns (groups, chunk_group): groups is a list of lists of threadblock indices in creation
    order; chunk_group maps each chunk id to its group index."""
    groups = []
    chunk_group = {}
    for tb, chunks in enumerate(tb_chunks):
        shared = {}
        for c in chunks:
            if c in chunk_group:
                g = chunk_group[c]
                shared[g] = shared.get(g, 0) + 1
        if not shared:
            g = len(groups)
            groups.append([])
        else:
            best = None
            for g_i in sorted(shared):
                if best is None or shared[g_i] > shared[best]:
                    best = g_i
            g = best
        groups[g].append(tb)
        for c in chunks:
            if c not in chunk_group:
                chunk_group[c] = g
    return groups, chunk_group


def sorted_groups(groups):
    """Group indices in decreasing order of size, creation order among equal sizes."""
    return sorted(range(len(groups)), key=lambda g: (-len(groups[g]), g))


def mi355x_topology(cu_budget=700 * 128, stack_budget=1 << 20):
    """8 physical domains (XCDs) of 32 CUs, 8 HBM stacks.  XCDs 0-3 and their stacks 0-3 sit on
    one I/O die, 4-7 on the other.  XCD x prefers stack x, then the other stacks of its die in
    index order, then the far die's stacks in index order."""
    pref = []
    for x in range(8):
        die = x // 4
        near = [x] + [s for s in range(4 * die, 4 * die + 4) if s != x]
        far = [s for s in range(8) if s // 4 != die]
        pref.append(near + far)
    return {"domains": 8, "cus_per_domain": 32, "stacks": 8, "stack_pref": pref,
            "cu_budget": cu_budget, "stack_budget": stack_budget}


def plan(tb_chunks, tb_bytes, nar_max, topo, chunk_page=None):
    """Algorithm 1.  tb_bytes[tb]: bytes the threadblock's chunks take (the resource charge).
    chunk_page: optional dict chunk id -> page id (page-level first come, first served).
    Returns dict with tb_group (index into the creation-order group list), tb_domain (NAR domain),
    tb_cu (global CU index = physical domain * cus_per_domain + local CU), chunk_stack."""
    D, ncu, S = topo["domains"], topo["cus_per_domain"], topo["stacks"]
    if nar_max < 1 or D % nar_max:
        raise ValueError("nar_max must divide the number of physical domains")
    groups, _ = logical_allocation(tb_chunks)
    R_cu = [topo["cu_budget"]] * (D * ncu)
    R_st = [topo["stack_budget"]] * S
    per = D // nar_max
    tb_group = [None] * len(tb_chunks)
    tb_domain = [None] * len(tb_chunks)
    tb_cu = [None] * len(tb_chunks)
    chunk_stack = {}
    page_stack = {}
    for i, g in enumerate(sorted_groups(groups)):
        nar = i % nar_max
        cus = list(range(nar * per * ncu, (nar + 1) * per * ncu))
        for tb in groups[g]:
            cs = tb_bytes[tb]
            cu = None
            for c in cus:
                if R_cu[c] >= cs:
                    cu = c
                    break
            if cu is None:
                cu = cus[0]
                for c in cus:
                    if R_cu[c] > R_cu[cu]:
                        cu = c
            prefs = topo["stack_pref"][cu // ncu]
            stack = None
            for s in prefs:
                if R_st[s] >= cs:
                    stack = s
                    break
            if stack is None:
                stack = prefs[0]
            R_cu[cu] -= cs
            R_st[stack] -= cs
            tb_group[tb] = g
            tb_domain[tb] = nar
            tb_cu[tb] = cu
            for c in tb_chunks[tb]:
                if c in chunk_stack:
                    continue
                if chunk_page is not None:
                    pg = chunk_page[c]
                    if pg not in page_stack:
                        page_stack[pg] = stack
                    chunk_stack[c] = page_stack[pg]
                else:
                    chunk_stack[c] = stack
    return {"groups": groups, "tb_group": tb_group, "tb_domain": tb_domain, "tb_cu": tb_cu,
            "chunk_stack": chunk_stack}
