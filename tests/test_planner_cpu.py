"""CPU: the library's Algorithm 1 planner (nuna_nap_plan) against the Python oracle, entry by entry,
and against the closed-form XCD map the kernels compute for uniform logical groups."""
import json
import os
import random
import sys

import numpy as np
import pytest

from paper_2608_00867_amd import nuna

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from oracle import nap_oracle  # noqa: E402

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "nap_plan_cases.json")


def _compare(tbs, cs, nar_max, cu_budget, stack_budget, pages=None):
    ref = nap_oracle.plan(tbs, cs, nar_max, nap_oracle.mi355x_topology(cu_budget, stack_budget), pages)
    entry_pages = None if pages is None else [pages[c] for t in tbs for c in t]
    got = nuna.nap_plan(tbs, cs, nar_max, nuna.nap_topology_mi355x(cu_budget, stack_budget), entry_pages)
    assert got["num_groups"] == len(ref["groups"])
    assert got["tb_group"].tolist() == ref["tb_group"]
    assert got["tb_domain"].tolist() == ref["tb_domain"]
    assert got["tb_cu"].tolist() == ref["tb_cu"]
    assert got["entry_stack"].tolist() == [ref["chunk_stack"][c] for t in tbs for c in t]


def test_topology_matches_oracle():
    t = nuna.nap_topology_mi355x()
    ref = nap_oracle.mi355x_topology()
    assert (t.num_domains, t.cus_per_domain, t.num_stacks) == (ref["domains"], ref["cus_per_domain"], ref["stacks"])
    assert (t.cu_budget, t.stack_budget) == (ref["cu_budget"], ref["stack_budget"])
    for x in range(8):
        assert list(t.stack_pref[x])[:8] == ref["stack_pref"][x]


def test_golden_cases():
    for case in json.load(open(GOLDEN))["cases"]:
        pages = {int(k): v for k, v in case["chunk_page"].items()} if "chunk_page" in case else None
        _compare(case["tb_chunks"], case["tb_bytes"], case["nar_max"], case["cu_budget"], case["stack_budget"],
                 pages)


@pytest.mark.parametrize("seed", range(40))
def test_random_workloads_match_oracle(seed):
    rng = random.Random(1000 + seed)
    n = rng.randint(0, 300)
    nchunks = rng.randint(1, 400)
    tbs = [rng.sample(range(nchunks), rng.randint(0, min(6, nchunks))) for _ in range(n)]
    cs = [rng.randint(0, 5000) for _ in range(n)]
    pages = {c: c // rng.randint(1, 4) for c in range(nchunks)} if seed % 3 == 0 else None
    _compare(tbs, cs, rng.choice([1, 2, 4, 8]), rng.randint(1000, 200000), rng.randint(1000, 1 << 20), pages)


@pytest.mark.parametrize("groups,gsize,G", [(21, 4, 84), (64, 8, 512), (9, 2, 18), (300, 3, 900), (5, 8, 40)])
def test_planner_domain_equals_kernel_xcd(groups, gsize, G):
    """Uniform groups (the split all-reduce / all-gather: gsize items read one chunk): the planner's
    NAR domain of every item equals the XCD (workgroup mod 8) the kernels' XCD mode runs it on."""
    tbs = [[("c", g), ("m", g, m)] for g in range(groups) for m in range(gsize)]
    ids = {k: i for i, k in enumerate(sorted({c for t in tbs for c in t}))}
    plan = nuna.nap_plan([[ids[c] for c in t] for t in tbs], [1] * len(tbs), 8)
    Gk = nuna.placement_grid("xcd", groups, gsize)
    xcd_of = {}
    for b in range(Gk):
        for w in nuna.placement_items("xcd", b, Gk, groups, gsize):
            xcd_of[int(w)] = b % 8
    assert sorted(xcd_of) == list(range(groups * gsize))
    assert [xcd_of[w] for w in range(groups * gsize)] == plan["tb_domain"].tolist()


@pytest.mark.parametrize("case", ["nar_not_divisor", "nar_zero", "bad_offsets", "first_offset", "neg_bytes",
                                  "bad_pref", "null_topo", "null_ids"])
def test_plan_rejects(case):
    import ctypes
    t = nuna.nap_topology_mi355x()
    off = np.array([0, 2, 3], dtype=np.int64)
    ids = np.array([1, 2, 3], dtype=np.int64)
    cs = np.array([1, 1], dtype=np.int64)
    nar = 8
    topo = ctypes.byref(t)
    if case == "nar_not_divisor":
        nar = 3
    elif case == "nar_zero":
        nar = 0
    elif case == "bad_offsets":
        off = np.array([0, 3, 2], dtype=np.int64)
    elif case == "first_offset":
        off = np.array([1, 2, 3], dtype=np.int64)
    elif case == "neg_bytes":
        cs = np.array([1, -1], dtype=np.int64)
    elif case == "bad_pref":
        t.stack_pref[2][1] = t.stack_pref[2][0]
    elif case == "null_topo":
        topo = None
    p64 = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))  # noqa: E731
    st = nuna.lib().nuna_nap_plan(topo, nar, 2, p64(off), None if case == "null_ids" else p64(ids), p64(cs),
                                  None, None, None, None, None, None)
    assert st == nuna.ERR_INVALID_ARG, nuna.last_error()


def test_empty_workload():
    plan = nuna.nap_plan([], [], 8)
    assert plan["num_groups"] == 0 and plan["tb_group"].size == 0
