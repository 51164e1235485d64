"""Pins for the CPU oracle: checks against things other than the oracle itself.

Each ``pin_*`` function takes an ``oracle.Oracle`` instance and raises
AssertionError when the oracle disagrees with an independent source of truth:

* numpy's ``add.accumulate`` (a sequential left-to-right running sum by
  definition) for the fp32 ascending-rank accumulation;
* torch's CPU fp32->bf16 conversion and a from-the-definition fp64
  round-to-nearest-even for the bf16 narrowing;
* exact integer arithmetic (Python ints) for integer-valued inputs;
* closed forms: one-hot ranks, constant ranks, all -0.0;
* the recursive-summation error bound against exactly rounded sums (fsum);
* hand-derived cases in ``tests/golden/ar_hand_cases.txt``;
* invariants: all destinations identical, all-gather(reduce-scatter) equals
  all-reduce, permutation invariance of integer sums, byte-exact copies;
* a brute-force Python enumeration of the all-to-all routing rule on tiny
  inputs, and the closed-form mean number of destination ranks per token.

The same functions run against deliberately broken builds of the oracle
(tests/test_oracle_mutants.py) to show each planted mistake is caught.
"""
import math
import os

import numpy as np

from paper_2608_00867_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

U = 2.0 ** -24  # fp32 unit roundoff


# ---------------------------------------------------------------- helpers

def _bf16_to_f32_torch(bits):
    import torch
    return torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float32).numpy()


def _f32_to_bf16_torch(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(
        np.uint16)


def _seq_sum_f32(stack_f32):
    """Left-to-right fp32 running sum over axis 0 via numpy's accumulate."""
    return np.add.accumulate(stack_f32, axis=0, dtype=np.float32)[-1]


def _bf16_value(h):
    """Exact value of a bf16 pattern as a Python float (fp64 holds it exactly)."""
    return float(np.array([h << 16], dtype=np.uint32).view(np.float32)[0])


def rne_definition(u32):
    """Round an fp32 bit pattern to bf16 from the definition of RNE, in fp64.

    The two candidates are the bf16 values just below and just above (in
    magnitude) the input; the nearer wins, a tie goes to the even pattern.
    Overflow: the candidate past the largest finite bf16 is 2^128, which maps
    to infinity, as IEEE-754 prescribes.
    """
    u32 = int(u32)
    sign = u32 >> 31
    mag = u32 & 0x7FFFFFFF
    if mag > 0x7F800000:
        return None  # NaN: only NaN-ness is compared
    x = abs(float(np.array([mag], dtype=np.uint32).view(np.float32)[0]))
    lo = mag >> 16
    if (mag & 0xFFFF) == 0:
        res = lo
    else:
        hi = lo + 1
        vlo = _bf16_value(lo)
        vhi = 2.0 ** 128 if hi == 0x7F80 else _bf16_value(hi)
        dlo, dhi = x - vlo, vhi - x
        if dlo < dhi:
            res = lo
        elif dhi < dlo:
            res = hi
        else:
            res = lo if lo % 2 == 0 else hi
    return res | (sign << 15)


# ---------------------------------------------------------------- all-reduce pins

def pin_ar_f32_sequential(orc):
    """fp32 all-reduce equals numpy's sequential accumulate, bit for bit."""
    for P, n, seed in [(1, 33, 1), (2, 100, 2), (3, 257, 3), (5, 1000, 4), (8, 4097, 5), (64, 515, 6)]:
        x = wl.normal_f32(P, n, seed)
        # spread magnitudes so rounding order matters
        x = [a * np.float32(2.0 ** ((i * 7) % 23 - 11)) for i, a in enumerate(x)]
        out = orc.allreduce(x)
        ref = _seq_sum_f32(np.stack(x))
        for d in range(P):
            assert np.array_equal(out[d].view(np.uint32), ref.view(np.uint32)), (P, n, d)


def pin_ar_bf16_widen_accumulate_round(orc):
    """bf16 all-reduce == torch widen -> sequential fp32 accumulate -> torch RNE narrow."""
    for P, n, seed in [(2, 64, 11), (3, 129, 12), (8, 2048 + 5, 13), (64, 300, 14)]:
        x = wl.normal_bf16(P, n, seed)
        x = [wl.f32_to_bf16_bits(_bf16_to_f32_torch(a) * np.float32(2.0 ** ((i * 5) % 17 - 8)))
             for i, a in enumerate(x)]
        out = orc.allreduce(x)
        acc = _seq_sum_f32(np.stack([_bf16_to_f32_torch(a) for a in x]))
        ref = _f32_to_bf16_torch(acc)
        for d in range(P):
            assert np.array_equal(out[d], ref), (P, n, d)
        acc_o = orc.allreduce_acc(x)
        assert np.array_equal(acc_o.view(np.uint32), acc.view(np.uint32))


def pin_ar_integer_exact(orc):
    """Integer-valued inputs sum exactly: equals the Python integer sum."""
    cases = [(8, 2048, -8, 8, np.float32), (64, 4096, -4, 4, np.float32), (8, 1000, -8, 8, np.uint16),
             (64, 777, -4, 4, np.uint16), (3, 9, -8, 8, np.float32)]
    for i, (P, n, lo, hi, dt) in enumerate(cases):
        ints = [np.random.default_rng(100 + i).integers(lo, hi, size=n, endpoint=True) for _ in range(P)]
        exact = np.zeros(n, dtype=np.int64)
        for a in ints:
            exact += a
        if dt == np.float32:
            x = [a.astype(np.float32) for a in ints]
            out = orc.allreduce(x)
            got = [o.astype(np.int64) for o in out]
            for g, o in zip(got, out):
                assert np.array_equal(o, o.astype(np.int64).astype(np.float32))
        else:
            x = [wl.f32_to_bf16_bits(a.astype(np.float32)) for a in ints]
            out = orc.allreduce(x)
            got = [_bf16_to_f32_torch(o).astype(np.int64) for o in out]
        for d in range(P):
            assert np.array_equal(got[d], exact), (P, n, dt, d)


def pin_ar_one_hot(orc):
    """Only rank k non-zero: every output equals in[k] bit for bit (each rank counted once,
    pointer order respected)."""
    for dt in (np.float32, np.uint16):
        for P in (2, 5, 8, 64):
            n = 300
            for k in sorted({0, 1, P // 2, P - 1}):
                v = wl.normal_f32(1, n, 7 * P + k)[0]
                x = [np.zeros(n, dtype=np.float32) for _ in range(P)]
                x[k] = v
                if dt == np.uint16:
                    x = [wl.f32_to_bf16_bits(a) for a in x]
                out = orc.allreduce(x)
                view = np.uint32 if dt == np.float32 else np.uint16
                for d in range(P):
                    assert np.array_equal(out[d].view(view), x[k].view(view)), (dt, P, k, d)


def pin_ar_constant_ranks(orc):
    """in[r][i] = c_r for all i: every output element is sum(c_r) (small integers, exact)."""
    for P in (1, 2, 7, 8, 64):
        c = [((r * 5) % 11) - 5 for r in range(P)]
        x = [np.full(129, cr, dtype=np.float32) for cr in c]
        out = orc.allreduce(x)
        for d in range(P):
            assert np.all(out[d] == np.float32(sum(c))), (P, d)


def pin_ar_negative_zero(orc):
    """All ranks -0.0 -> -0.0 (the sum starts from rank 0's value); one +0.0 -> +0.0."""
    for dt, neg, pos in ((np.float32, 0x80000000, 0), (np.uint16, 0x8000, 0)):
        for P in (1, 2, 8):
            view = np.uint32 if dt == np.float32 else np.uint16
            x = [np.full(17, neg, dtype=view).view(dt) for _ in range(P)]
            out = orc.allreduce(x)
            assert all(int(o.view(view)[0]) == neg for o in out), (dt, P)
            if P > 1:
                x[P - 1] = np.full(17, pos, dtype=view).view(dt)
                out = orc.allreduce(x)
                assert all(int(o.view(view)[3]) == pos for o in out), (dt, P)


def pin_ar_error_bound(orc):
    """|acc - exact| <= gamma_{P-1} * sum|x| with exact from math.fsum; bf16 narrowing adds at most
    half a bf16 ulp (relative 2^-8)."""
    for P, n, seed, dt in [(8, 400, 21, np.float32), (64, 200, 22, np.float32), (8, 400, 23, np.uint16),
                           (64, 200, 24, np.uint16)]:
        if dt == np.float32:
            x = wl.normal_f32(P, n, seed)
            xf = [a.astype(np.float64) for a in x]
        else:
            x = wl.normal_bf16(P, n, seed)
            xf = [_bf16_to_f32_torch(a).astype(np.float64) for a in x]
        acc = orc.allreduce_acc(x).astype(np.float64)
        out = orc.allreduce(x)[0]
        gamma = (P - 1) * U / (1 - (P - 1) * U)
        for i in range(n):
            terms = [a[i] for a in xf]
            exact = math.fsum(terms)
            bound = gamma * math.fsum(abs(t) for t in terms)
            assert abs(acc[i] - exact) <= bound, (P, i, acc[i], exact, bound)
            y = float(out[i]) if dt == np.float32 else _bf16_value(int(out[i]))
            assert abs(y - acc[i]) <= (U if dt == np.float32 else 2.0 ** -8) * abs(acc[i]), (P, i)


def pin_ar_hand_cases(orc):
    """Cases worked out by hand from IEEE round-to-nearest-even (tests/golden/ar_hand_cases.txt)."""
    n_cases = 0
    with open(os.path.join(GOLDEN, "ar_hand_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            dts, ins, exp = [s.strip() for s in line.split("|")]
            view = np.uint32 if dts == "f32" else np.uint16
            dt = np.float32 if dts == "f32" else np.uint16
            x = [np.full(5, int(h, 16), dtype=view).view(dt) for h in ins.split()]
            out = orc.allreduce(x)
            for o in out:
                assert np.all(o.view(view) == int(exp, 16)), (line, hex(int(o.view(view)[0])))
            n_cases += 1
    assert n_cases >= 10


def pin_ar_permutation_invariant_integers(orc):
    """Integer sums do not depend on the rank order."""
    x = wl.int_uniform_f32(8, 513, -8, 8, 31)
    a = orc.allreduce(x)[0]
    perm = np.random.default_rng(32).permutation(8)
    b = orc.allreduce([x[p] for p in perm])[0]
    assert np.array_equal(a, b)


def pin_ar_outputs_identical_and_inplace(orc):
    """All P destinations identical; in-place (out[r] is in[r]) gives the same bits."""
    x = wl.normal_bf16(8, 1000, 41)
    out = orc.allreduce(x)
    for d in range(1, 8):
        assert np.array_equal(out[0], out[d])
    y = [a.copy() for a in x]
    orc.allreduce(y, outs=y)
    for d in range(8):
        assert np.array_equal(y[d], out[0])


# ---------------------------------------------------------------- rounding pins

def pin_bf16_round_definition(orc):
    """fp32->bf16 narrowing agrees with the from-definition RNE on boundary and random patterns."""
    pats = []
    for hi in (0x0000, 0x0001, 0x007F, 0x0080, 0x3F80, 0x3F81, 0x4B80, 0x7F7E, 0x7F7F, 0x7F80):
        for lo in (0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF):
            for s in (0, 1):
                pats.append((s << 31) | (hi << 16) | lo)
    pats += list(np.random.default_rng(51).integers(0, 1 << 32, size=4000, dtype=np.uint64))
    u = np.array(pats, dtype=np.uint64).astype(np.uint32)
    got = orc.f32_to_bf16(u.view(np.float32))
    for p, g in zip(u, got):
        ref = rne_definition(p)
        if ref is None:
            assert (int(g) & 0x7FFF) > 0x7F80, hex(int(p))
        else:
            assert int(g) == ref, (hex(int(p)), hex(int(g)), hex(ref))


def pin_bf16_round_vs_torch_sample(orc):
    """fp32->bf16 narrowing agrees with torch's conversion on 2^22 random patterns."""
    u = np.random.default_rng(52).integers(0, 1 << 32, size=1 << 22, dtype=np.uint64).astype(np.uint32)
    _compare_with_torch(orc, u)


def _compare_with_torch(orc, u):
    f = u.view(np.float32)
    got = orc.f32_to_bf16(f)
    ref = _f32_to_bf16_torch(f)
    nan = np.isnan(f)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.all((got[nan] & 0x7FFF) > 0x7F80)


def bf16_round_exhaustive(orc, chunk_bits=24):
    """All 2^32 fp32 patterns, in chunks, with buffers reused across chunks."""
    import torch
    step = 1 << chunk_bits
    u = np.empty(step, dtype=np.uint32)
    got = np.empty(step, dtype=np.uint16)
    ref_t = torch.empty(step, dtype=torch.bfloat16)
    ramp = np.arange(step, dtype=np.uint32)
    f = u.view(np.float32)
    f_t = torch.from_numpy(f)
    ref = ref_t.view(torch.int16).numpy().view(np.uint16)
    for start in range(0, 1 << 32, step):
        np.add(ramp, np.uint32(start), out=u)
        orc.lib.oracle_f32_to_bf16_array(u.ctypes.data, got.ctypes.data, step)
        ref_t.copy_(f_t)
        nan = np.isnan(f)
        if nan.any():
            assert np.array_equal(got[~nan], ref[~nan]), hex(start)
            assert np.all((got[nan] & 0x7FFF) > 0x7F80), hex(start)
        else:
            assert np.array_equal(got, ref), hex(start)


# ---------------------------------------------------------------- RS / AG pins

def pin_rs_index_coded(orc):
    """Reduce-scatter of index-coded integers: rank r gets sum_q in[q][r*m+j] at j (closed form)."""
    for P, m in ((1, 5), (2, 3), (3, 7), (8, 64), (5, 1)):
        n = P * m
        # in[q][i] = q + 16*i  (exact in fp32 for these sizes)
        x = [(q + 16.0 * np.arange(n)).astype(np.float32) for q in range(P)]
        out = orc.reduce_scatter(x)
        for r in range(P):
            i = r * m + np.arange(m)
            expect = (P * (P - 1) // 2 + 16.0 * P * i).astype(np.float32)
            assert np.array_equal(out[r], expect), (P, m, r)


def pin_ag_index_coded_and_bits(orc):
    """All-gather places in[r][j] at out[d][r*m+j] for every d, copying bytes (NaN payloads kept)."""
    for dt in (np.uint16, np.float32):
        for P, m in ((1, 4), (2, 9), (3, 5), (8, 33)):
            x = wl.random_bits(P, m, dt, 61 + P)
            view = np.uint16 if dt == np.uint16 else np.uint32
            # signalling and quiet NaNs with payloads, infinities, -0, denormals
            special = ([0x7F81, 0xFFBF, 0x7FC1, 0x7F80, 0x8000, 0x0001] if dt == np.uint16 else
                       [0x7F800001, 0xFFBFFFFF, 0x7FC00123, 0x7F800000, 0x80000000, 0x00000001])
            for r in range(P):
                k = min(m, len(special))
                x[r].view(view)[:k] = np.array(special[:k], dtype=view)
            out = orc.all_gather(x)
            for d in range(P):
                for r in range(P):
                    assert np.array_equal(out[d][r * m:(r + 1) * m].view(view), x[r].view(view)), (dt, P, d, r)


def pin_two_shot_equals_one_shot(orc):
    """all-gather(reduce-scatter(x)) == all-reduce(x) bit for bit."""
    for dt, P, m, seed in ((np.uint16, 8, 129, 71), (np.float32, 8, 64, 72), (np.uint16, 3, 11, 73),
                           (np.uint16, 64, 5, 74)):
        n = P * m
        x = wl.normal_bf16(P, n, seed) if dt == np.uint16 else wl.normal_f32(P, n, seed)
        ar = orc.allreduce(x)
        ag = orc.all_gather(orc.reduce_scatter(x))
        view = np.uint16 if dt == np.uint16 else np.uint32
        for d in range(P):
            assert np.array_equal(ag[d].view(view), ar[d].view(view)), (dt, P, d)


# ---------------------------------------------------------------- all-to-all pins

def _a2a_brute(topk, E):
    """Routing rule written out with Python sets: token (s,t) goes once to every rank owning one
    of its experts; rank d receives rows ordered by (s, t)."""
    P, T, _ = topk.shape
    per = E // P
    lists = {d: [] for d in range(P)}
    for s in range(P):
        for t in range(T):
            owners = {int(e) // per for e in topk[s, t]}
            for d in owners:
                lists[d].append((s, t))
    for d in lists:
        lists[d].sort()
    return lists


def pin_a2a_brute_force(orc):
    """Counts, maps and row copies equal a brute-force enumeration on small inputs."""
    for P, T, k, E, seed in ((1, 3, 1, 1, 81), (2, 5, 2, 4, 82), (3, 7, 2, 6, 83), (4, 16, 3, 16, 84),
                             (8, 20, 8, 256, 85), (8, 1, 8, 64, 86), (2, 0, 1, 2, 87)):
        topk = wl.moe_routing(P, T, k, E, seed)
        ref = _a2a_brute(topk, E)
        rows = orc.a2a_counts(topk, E)
        for d in range(P):
            assert rows[d] == len(ref[d]), (P, T, d)
            sr, st = orc.a2a_map(topk, E, d)
            assert list(zip(sr.tolist(), st.tolist())) == ref[d], (P, T, d)
        send = wl.random_bits(P, max(T, 1) * 6, np.uint16, seed)
        send = [a[:T * 6].reshape(T, 6) for a in send]
        recv = orc.all_to_all(send, topk, E)
        for d in range(P):
            assert recv[d].shape == (len(ref[d]), 6)
            for j, (s, t) in enumerate(ref[d]):
                assert np.array_equal(recv[d][j], send[s][t]), (P, T, d, j)


def pin_a2a_distinct_rank_mean(orc):
    """At the MoE shape (P=8, 512 tokens, top-8 of 256, 32 experts per rank) the mean number of
    destination ranks per token matches 8 * (1 - C(224,8)/C(256,8)) = 5.295 (closed form)."""
    P, T, k, E = 8, 512, 8, 256
    topk = wl.moe_routing(P, T, k, E, wl.seed_for(4))
    assert topk.min() >= 0 and topk.max() < E
    assert all(len(set(topk[s, t].tolist())) == k for s in range(P) for t in range(T))
    rows = orc.a2a_counts(topk, E)
    expect = P * (1 - math.comb(E - E // P, k) / math.comb(E, k))
    mean = rows.sum() / (P * T)
    assert abs(mean - expect) < 0.05, (mean, expect)


def pin_a2a_conservation(orc):
    """sum_d rows[d] == sum over tokens of the number of distinct owner ranks."""
    topk = wl.moe_routing(8, 300, 8, 256, 91)
    rows = orc.a2a_counts(topk, 256)
    total = sum(len({int(e) // 32 for e in topk[s, t]}) for s in range(8) for t in range(300))
    assert rows.sum() == total


# ---------------------------------------------------------------- combine pins

def pin_combine_k1_inverts_dispatch(orc):
    """With one expert per token, combine(dispatch(x)) returns x bit for bit (one term per token)."""
    for dt in (np.uint16, np.float32):
        P, T, E, H = 4, 9, 8, 24
        topk = wl.moe_routing(P, T, 1, E, 301)
        x = [a.reshape(T, H) for a in (wl.normal_bf16(P, T * H, 302) if dt == np.uint16 else wl.normal_f32(P, T * H, 302))]
        back = orc.combine(orc.all_to_all(x, topk, E), topk, E)
        view = np.uint16 if dt == np.uint16 else np.uint32
        for s in range(P):
            assert np.array_equal(back[s].view(view), x[s].view(view)), (dt, s)


def pin_combine_identity_experts_count_destinations(orc):
    """Identity experts on integer rows: each token comes back multiplied by its number of distinct
    destination ranks (exact: small integers)."""
    P, T, k, E, H = 8, 40, 8, 256, 16
    topk = wl.moe_routing(P, T, k, E, 311)
    ints = [np.random.default_rng(312 + s).integers(-8, 8, size=(T, H), endpoint=True) for s in range(P)]
    x = [wl.f32_to_bf16_bits(a.astype(np.float32)).reshape(T, H) for a in ints]
    back = orc.combine(orc.all_to_all(x, topk, E), topk, E)
    per = E // P
    for s in range(P):
        c = np.array([len({int(e) // per for e in topk[s, t]}) for t in range(T)])
        got = _bf16_to_f32_torch(back[s].ravel()).reshape(T, H)
        assert np.array_equal(got, (ints[s] * c[:, None]).astype(np.float32)), s


def pin_combine_sequential_sum(orc):
    """Combine equals, per token, numpy's sequential accumulate over its results in ascending
    destination order (rows located by a brute-force routing enumeration), then torch's rounding.
    The fp32 case draws results of mixed magnitude so that a different summation order changes
    the rounded sum."""
    P, T, k, E, H = 4, 12, 3, 16, 8
    topk = wl.moe_routing(P, T, k, E, 321)
    lists = _a2a_brute(topk, E)
    for dt in ("bf16", "f32"):
        if dt == "bf16":
            y = [wl.normal_bf16(1, len(lists[d]) * H, 330 + d)[0].reshape(len(lists[d]), H) for d in range(P)]
        else:
            y = []
            for d in range(P):
                g = np.random.default_rng(340 + d)
                v = g.standard_normal((len(lists[d]), H)) * np.exp2(g.integers(-12, 12, size=(len(lists[d]), H)))
                y.append(v.astype(np.float32))
        out = orc.combine(y, topk, E)
        for s in range(P):
            for t in range(T):
                dests = [d for d in range(P) if (s, t) in lists[d]]
                rows = [y[d][lists[d].index((s, t))] for d in dests]
                if dt == "bf16":
                    terms = np.stack([_bf16_to_f32_torch(r) for r in rows])
                    ref = _f32_to_bf16_torch(np.add.accumulate(terms, axis=0, dtype=np.float32)[-1])
                    assert np.array_equal(out[s][t], ref), (dt, s, t)
                else:
                    ref = np.add.accumulate(np.stack(rows), axis=0, dtype=np.float32)[-1]
                    assert np.array_equal(out[s][t].view(np.uint32), ref.view(np.uint32)), (dt, s, t)


def pin_combine_conserves_integer_totals(orc):
    """Integer results: the grand total over all output rows equals the total over all result rows."""
    P, T, k, E, H = 8, 30, 8, 256, 4
    topk = wl.moe_routing(P, T, k, E, 341)
    rows = orc.a2a_counts(topk, E)
    ys = [np.random.default_rng(342 + d).integers(-4, 4, size=(int(rows[d]), H), endpoint=True) for d in range(P)]
    y = [wl.f32_to_bf16_bits(a.astype(np.float32)).reshape(-1, H) for a in ys]
    out = orc.combine(y, topk, E)
    tot_out = sum(int(_bf16_to_f32_torch(o.ravel()).astype(np.int64).sum()) for o in out)
    assert tot_out == sum(int(a.sum()) for a in ys)


def pin_combine_unit_weights_change_nothing(orc):
    """Weights of 1.0 leave every term as it is: the weighted combine equals the unweighted one."""
    P, T, k, E, H = 8, 20, 8, 64, 24
    topk = wl.moe_routing(P, T, k, E, 351)
    rows = orc.a2a_counts(topk, E)
    for dt in (np.uint16, np.float32):
        y = wl.result_rows(rows, H, dt, 352)
        a = orc.combine(y, topk, E)
        b = orc.combine(y, topk, E, np.ones((P, T, P), dtype=np.float32))
        for s in range(P):
            assert np.array_equal(a[s].view(np.uint8), b[s].view(np.uint8)), (dt, s)


def pin_combine_power_of_two_weights_scale_exactly(orc):
    """One expert per token and weights 2^j: each token row comes back multiplied by 2^j exactly
    (N(0,1) values: no overflow or underflow)."""
    P, T, E, H = 4, 16, 8, 32
    topk = wl.moe_routing(P, T, 1, E, 361)
    x = wl.result_rows(orc.a2a_counts(topk, E), H, np.uint16, 362)
    g = np.random.default_rng(363)
    w = np.exp2(g.integers(-4, 4, size=(P, T, P), endpoint=True)).astype(np.float32)
    out = orc.combine(x, topk, E, w)
    per = E // P
    for s in range(P):
        for t in range(T):
            d = int(topk[s, t, 0]) // per
            j = [(ss, tt) for ss in range(P) for tt in range(T) if int(topk[ss, tt, 0]) // per == d].index((s, t))
            ref = _f32_to_bf16_torch(_bf16_to_f32_torch(x[d][j]) * w[s, t, d])
            assert np.array_equal(out[s][t], ref), (s, t)


def pin_combine_gate_weighted_sum(orc):
    """One expert per rank (E == P): the combine is the MoE layer's top-k weighted sum.  Per token:
    fp32 products gate * result, added one by one in ascending expert order (numpy float32 arithmetic,
    rows located by brute-force enumeration)."""
    P, T, k, H = 8, 12, 3, 16
    E = P
    topk = wl.moe_routing(P, T, k, E, 371)
    lists = _a2a_brute(topk, E)
    g = np.random.default_rng(372)
    gates = g.random((P, T, k)).astype(np.float32)
    w = np.zeros((P, T, P), dtype=np.float32)
    for s in range(P):
        for t in range(T):
            for q in range(k):
                w[s, t, int(topk[s, t, q])] = gates[s, t, q]
    y = []
    for d in range(P):
        v = g.standard_normal((len(lists[d]), H)) * np.exp2(g.integers(-12, 12, size=(len(lists[d]), H)))
        y.append(v.astype(np.float32))
    out = orc.combine(y, topk, E, w)
    for s in range(P):
        for t in range(T):
            order = sorted(range(k), key=lambda q: int(topk[s, t, q]))
            terms = [np.float32(gates[s, t, q]) * y[int(topk[s, t, q])][lists[int(topk[s, t, q])].index((s, t))]
                     for q in order]
            ref = np.add.accumulate(np.stack(terms).astype(np.float32), axis=0, dtype=np.float32)[-1]
            assert np.array_equal(out[s][t].view(np.uint32), ref.view(np.uint32)), (s, t)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
