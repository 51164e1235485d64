"""CPU: the host-side argument checks against a brute-force reference on random pointer layouts.

Pointers are fake (never dereferenced): a call whose arguments are valid reaches the launch and, with
no GPU here, returns NUNA_ERR_HIP; an invalid one must be rejected with the status the reference
predicts before any HIP call."""
import random

import pytest

from paper_2608_00867_amd import nuna

BASE = 0x7F0000000000


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def _overlap(a, b):
    return a[0] < b[1] and b[0] < a[1]


def _expected(op, P, nbytes_in, nbytes_out, ins, outs, shard_bytes):
    """Reference status: OVERLAP if two outputs overlap, or an input overlaps an output other than by the
    documented in-place alias; otherwise the call is valid."""
    ospans = [(o, o + nbytes_out) for o in outs]
    ispans = [(i, i + nbytes_in) for i in ins]
    for a in range(P):
        for b in range(a + 1, P):
            if _overlap(ospans[a], ospans[b]):
                return nuna.ERR_OVERLAP
    for r in range(P):
        for d in range(P):
            if not _overlap(ispans[r], ospans[d]):
                continue
            if op == "allreduce" and r == d and ins[r] == outs[d]:
                continue
            if op == "reduce_scatter" and r == d and outs[d] == ins[r] + r * shard_bytes:
                continue
            if op == "all_gather" and r == d and ins[r] == outs[d] + r * shard_bytes:
                continue
            return nuna.ERR_OVERLAP
    return None


@pytest.mark.parametrize("seed", range(400))
def test_overlap_checks_match_reference(seed):
    if _gpu_visible():
        pytest.skip("GPU visible: valid calls would launch")
    rng = random.Random(seed)
    P = rng.choice([1, 2, 3, 4, 8, 16, 64])
    op = rng.choice(["allreduce", "reduce_scatter", "all_gather"])
    es = rng.choice([2, 4])
    dt = nuna.BF16 if es == 2 else nuna.F32
    m = rng.choice([8, 16, 24, 64, 1000]) * (16 // es)  # elements per shard, 16-byte multiple
    shard = m * es
    if op == "allreduce":
        nin = nout = P * shard
    elif op == "reduce_scatter":
        nin, nout = P * shard, shard
    else:
        nin, nout = shard, P * shard
    # Place buffers on a coarse grid of 16-byte slots so that overlaps and in-place aliases happen often.
    slot = 16
    span = (P + 2) * max(nin, nout) // slot
    outs = [BASE + slot * rng.randrange(0, span) for _ in range(P)]
    ins = [BASE + (1 << 36) + slot * rng.randrange(0, span) for _ in range(P)]
    if seed >= 300:     # outputs in address order, as callers usually pass them
        outs.sort()
    mode = rng.random()
    if mode < 0.3:      # in-place aliases, maybe broken for one rank
        for r in range(P):
            if op == "allreduce":
                ins[r] = outs[r]
            elif op == "reduce_scatter":
                outs[r] = ins[r] + r * shard
            else:
                ins[r] = outs[r] + r * shard
        if rng.random() < 0.5:
            r = rng.randrange(P)
            ins[r] += 16
    elif mode < 0.6:    # inputs in the output region
        for r in range(P):
            if rng.random() < 0.3:
                ins[r] = outs[rng.randrange(P)] + slot * rng.randrange(0, max(1, nout // slot))
    if op == "allreduce":
        count = P * m
        st = nuna.allreduce_raw(ins, outs, P, count, dt)
    elif op == "reduce_scatter":
        st = nuna.reduce_scatter_raw(ins, outs, P, m, dt)
    else:
        st = nuna.all_gather_raw(ins, outs, P, m, dt)
    exp = _expected(op, P, nin, nout, ins, outs, shard)
    if exp is None:
        assert st == nuna.ERR_HIP, (seed, op, P, st, nuna.last_error())
    else:
        assert st == exp, (seed, op, P, st, nuna.last_error())
