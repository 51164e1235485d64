"""CPU: the Algorithm 1 oracle against its pins, and planted mistakes in copies of it that the pins
must catch."""
import importlib.util
import os
import sys

import pytest

import planner_pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "nap_oracle.py")


def _load(source, name):
    spec = importlib.util.spec_from_loader(name, loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(source, SRC, "exec"), mod.__dict__)
    return mod


@pytest.fixture(scope="module")
def nap():
    sys.path.insert(0, ROOT)
    from oracle import nap_oracle
    return nap_oracle


@pytest.mark.parametrize("pin", planner_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(nap, pin):
    pin(nap)


# Planted mistakes, plus one reading: "domain_counter_first_advanced" is not a mistake against the
# printed listing of Algorithm 1, which increments the domain counter before its first use (so the first
# group would land in domain 1).  The oracle takes the reading that the first group lands in domain 0, as
# the algorithm's figure deals threadblock groups round-robin starting from NAR domain 0; the pins fix
# that reading, and the variant checks that they do.
MUTANTS = {
    "join_fewest_shared": ("if best is None or shared[g_i] > shared[best]:",
                           "if best is None or shared[g_i] < shared[best]:"),
    "tie_to_latest_group": ("for g_i in sorted(shared):", "for g_i in sorted(shared, reverse=True):"),
    "sort_increasing": ("key=lambda g: (-len(groups[g]), g)", "key=lambda g: (len(groups[g]), g)"),
    "domain_counter_first_advanced": ("nar = i % nar_max", "nar = (i + 1) % nar_max"),  # the other reading
    "last_fitting_cu": ("                if R_cu[c] >= cs:\n                    cu = c\n                    break",
                        "                if R_cu[c] >= cs:\n                    cu = c"),
    "stack_ignores_budget": ("if R_st[s] >= cs:", "if True:"),
    "cu_never_charged": ("R_cu[cu] -= cs", "R_cu[cu] -= 0"),
    "last_come_chunk_stack": ("                if c in chunk_stack:\n                    continue\n", ""),
    "page_ignored": ("                    chunk_stack[c] = page_stack[pg]", "                    chunk_stack[c] = stack"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    src = open(SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mod = _load(src.replace(old, new), f"nap_mutant_{name}")
    caught = []
    for pin in planner_pins.ALL_PINS:
        try:
            pin(mod)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"
