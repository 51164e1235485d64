"""Pins of the Algorithm 1 oracle (oracle/nap_oracle.py) to things other than itself: hand-derived
cases (tests/golden/nap_plan_cases.json, each derivation written out there), special cases that
reduce to a plain round-robin, and structural properties on random workloads."""
import json
import os
import random

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "nap_plan_cases.json")


def _golden():
    return json.load(open(GOLDEN))["cases"]


def pin_golden_cases(nap):
    for case in _golden():
        topo = nap.mi355x_topology(case["cu_budget"], case["stack_budget"])
        pages = {int(k): v for k, v in case["chunk_page"].items()} if "chunk_page" in case else None
        got = nap.plan(case["tb_chunks"], case["tb_bytes"], case["nar_max"], topo, pages)
        exp = case["expect"]
        assert got["tb_group"] == exp["tb_group"], (case["name"], got["tb_group"])
        assert got["tb_domain"] == exp["tb_domain"], (case["name"], got["tb_domain"])
        assert got["tb_cu"] == exp["tb_cu"], (case["name"], got["tb_cu"])
        assert {str(k): v for k, v in got["chunk_stack"].items()} == exp["chunk_stack"], (case["name"],
                                                                                          got["chunk_stack"])


def pin_disjoint_threadblocks_are_dealt_round_robin(nap):
    """No shared chunks: every threadblock is its own group, and groups of one keep their order, so
    threadblock i lands in NAR domain i mod nar_max on that domain's first CU (ample budgets)."""
    topo = nap.mi355x_topology(1 << 30, 1 << 30)
    for nar_max in (1, 2, 4, 8):
        n = 37
        got = nap.plan([[i] for i in range(n)], [64] * n, nar_max, topo)
        per = 8 // nar_max
        assert got["tb_domain"] == [i % nar_max for i in range(n)]
        assert got["tb_cu"] == [(i % nar_max) * per * 32 for i in range(n)]


def pin_uniform_groups_match_xcd_round_robin(nap):
    """Uniform logical groups (the split all-reduce: g members reading chunk c) -> group c in domain
    c mod 8, members in order: the closed form the kernels' XCD mode uses."""
    topo = nap.mi355x_topology(1 << 30, 1 << 30)
    chunks, gsize = 21, 4
    tbs = [[("in", c), ("out", c, m)] for c in range(chunks) for m in range(gsize)]
    got = nap.plan(tbs, [1] * len(tbs), 8, topo)
    for tb in range(len(tbs)):
        c = tb // gsize
        assert got["tb_group"][tb] == c and got["tb_domain"][tb] == c % 8, tb


def pin_one_shared_chunk_makes_one_group(nap):
    topo = nap.mi355x_topology(1 << 30, 1 << 30)
    got = nap.plan([[0, i + 1] for i in range(10)], [1] * 10, 8, topo)
    assert got["tb_group"] == [0] * 10 and got["tb_domain"] == [0] * 10


def pin_sorted_by_decreasing_size(nap):
    """Groups of sizes 1, 3, 2 (creation order) are dealt in the order 3, 2, 1."""
    topo = nap.mi355x_topology(1 << 30, 1 << 30)
    tbs = [[0], [1, 10], [1, 11], [1, 12], [2, 20], [2, 21]]
    got = nap.plan(tbs, [1] * len(tbs), 8, topo)
    assert got["tb_group"] == [0, 1, 1, 1, 2, 2]
    assert got["tb_domain"] == [2, 0, 0, 0, 1, 1]


def pin_random_structure(nap):
    """Random workloads: groups partition the threadblocks; a threadblock that joined a group shares a
    chunk with it; each group sits in one domain, dealt round-robin in non-increasing size order; every
    CU lies in its domain; budgets are exceeded only when nothing in the domain fit."""
    rng = random.Random(7)
    for trial in range(60):
        n = rng.randint(1, 60)
        tbs = [rng.sample(range(40), rng.randint(1, 4)) for _ in range(n)]
        cs = [rng.randint(1, 50) for _ in range(n)]
        nar_max = rng.choice([1, 2, 4, 8])
        topo = nap.mi355x_topology(rng.randint(20, 400), rng.randint(50, 2000))
        got = nap.plan(tbs, cs, nar_max, topo)
        groups = got["groups"]
        assert sorted(tb for g in groups for tb in g) == list(range(n))
        for g, members in enumerate(groups):
            seen = set(tbs[members[0]])
            for tb in members[1:]:
                assert seen & set(tbs[tb]), (trial, g, tb)
                seen |= set(tbs[tb])
            assert len({got["tb_domain"][tb] for tb in members}) == 1
        order = sorted(range(len(groups)), key=lambda g: (-len(groups[g]), g))
        sizes = [len(groups[g]) for g in order]
        assert sizes == sorted(sizes, reverse=True)
        for i, g in enumerate(order):
            assert got["tb_domain"][groups[g][0]] == i % nar_max
        per = 8 // nar_max
        R = [topo["cu_budget"]] * 256
        for g in order:
            for tb in groups[g]:
                d = got["tb_domain"][tb]
                cu = got["tb_cu"][tb]
                lo, hi = d * per * 32, (d + 1) * per * 32
                assert lo <= cu < hi
                if R[cu] < cs[tb]:
                    assert all(R[c] < cs[tb] for c in range(lo, hi)), (trial, tb)
                else:
                    assert all(R[c] < cs[tb] for c in range(lo, cu)), (trial, tb)
                R[cu] -= cs[tb]


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
