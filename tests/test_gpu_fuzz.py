"""GPU: seeded random collective calls through the C ABI against the oracle.

Each case draws the rank count, size, dtype, algorithm, placement, in-place form and a launch-shape
variant (through the run-time tunables), so that combinations no hand-written case names get run.
Bit-exact except for NaN payloads of arithmetic NaNs (random bit patterns include NaNs)."""
import numpy as np
import pytest

import oracle
from gpu_util import assert_bitwise_nan_aware, to_dev, to_host
from paper_2608_00867_amd import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

VARIANTS = [{}, dict(NUNA_MAX_GRID=7), dict(NUNA_WG_THREADS=64), dict(NUNA_WG_THREADS=128, NUNA_VPT=2),
            dict(NUNA_VPT=4), dict(NUNA_VPT=8), dict(NUNA_TILE_V=32), dict(NUNA_TILE_V=64, NUNA_LPR_MIN_RANKS=2),
            dict(NUNA_LPR_MIN_RANKS=1, NUNA_LPR_MAX_VECTORS=1 << 20)]
MOE_VARIANTS = [{}, dict(NUNA_COMBINE_LISTS=1), dict(NUNA_MAX_GRID=7), dict(NUNA_WG_THREADS=64, NUNA_COMBINE_VPT=1),
                dict(NUNA_COMBINE_CHUNKS=3, NUNA_COMBINE_VPT=4)]


@pytest.fixture(scope="module")
def nuna():
    from paper_2608_00867_amd import nuna as n
    n.init()
    return n


def _case(seed):
    g = np.random.default_rng(seed)
    P = int(g.choice([1, 2, 3, 4, 5, 7, 8, 12, 16, 24, 32, 48, 64]))
    n = int(np.exp(g.uniform(0, np.log(400000 // P + 2))))
    dtype = np.uint16 if g.random() < 0.6 else np.float32
    op = g.choice(["allreduce", "reduce_scatter", "all_gather"])
    algo = str(g.choice(["auto", "one_shot", "two_shot", "one_shot_split", "two_shot_two_kernels"]))
    place = str(g.choice(["linear", "xcd"]))
    inplace = bool(g.random() < 0.3)
    bits = bool(g.random() < 0.3)
    variant = VARIANTS[int(g.integers(len(VARIANTS)))]
    return P, n, dtype, op, algo, place, inplace, bits, variant


def _inputs(P, n, dtype, bits, seed):
    if bits:
        return wl.random_bits(P, n, dtype, seed)
    return wl.normal_bf16(P, n, seed) if dtype == np.uint16 else wl.normal_f32(P, n, seed)


@pytest.mark.parametrize("seed", range(400))
def test_fuzz(nuna, seed):
    P, n, dtype, op, algo, place, inplace, bits, variant = _case(9000 + seed)
    what = f"seed={seed} P={P} n={n} {dtype.__name__} {op} {algo} {place} inplace={inplace} {variant}"
    print(what, flush=True)
    with nuna.tunables(**variant):
        if op == "allreduce":
            x = _inputs(P, n, dtype, bits, seed)
            ref = oracle.allreduce(x)
            ins = [to_dev(a) for a in x]
            if inplace and algo == "one_shot_split":
                algo = "one_shot"
            outs = ins if inplace else [torch.empty_like(t) for t in ins]
            nuna.allreduce(ins, outs, algo=algo, placement=place)
        elif op == "reduce_scatter":
            es = 2 if dtype == np.uint16 else 4
            m = max(1, n // P)
            if inplace:
                m = (m + 16 // es - 1) // (16 // es) * (16 // es)  # in-place shards must stay 16-byte aligned
            x = _inputs(P, P * m, dtype, bits, seed)
            ref = oracle.reduce_scatter(x)
            ins = [to_dev(a) for a in x]
            outs = [ins[r][r * m:(r + 1) * m] for r in range(P)] if inplace else \
                [torch.empty(m, dtype=ins[0].dtype, device="cuda") for _ in range(P)]
            nuna.reduce_scatter(ins, outs, placement=place)
        else:
            es = 2 if dtype == np.uint16 else 4
            m = max(1, n // P)
            if inplace:
                m = (m + 16 // es - 1) // (16 // es) * (16 // es)
            x = _inputs(P, m, dtype, bits, seed)
            ref = oracle.all_gather(x)
            src = [to_dev(a) for a in x]
            outs = [torch.empty(P * m, dtype=src[0].dtype, device="cuda") for _ in range(P)]
            if inplace:
                for r in range(P):
                    outs[r][r * m:(r + 1) * m].copy_(src[r])
                ins = [outs[r][r * m:(r + 1) * m] for r in range(P)]
            else:
                ins = src
            nuna.all_gather(ins, outs, placement=place)
        torch.cuda.synchronize()
    for d in range(P):
        assert_bitwise_nan_aware(to_host(outs[d]), ref[d], f"{what} rank {d}")


@pytest.mark.parametrize("seed", range(120))
def test_fuzz_moe(nuna, seed):
    """Seeded random MoE dispatch + combine (unweighted or weighted) in a random placement."""
    g = np.random.default_rng(20000 + seed)
    P = int(g.choice([1, 2, 3, 4, 6, 8, 16, 64]))
    E = P * int(g.choice([1, 2, 4, 32]))
    k = int(g.integers(1, min(E, 9) + 1))
    T = int(g.integers(0, 70))
    H = int(g.choice([8, 10, 64, 100, 512, 7168]))
    dtype = np.uint16 if g.random() < 0.6 else np.float32
    place = str(g.choice(["linear", "xcd"]))
    weighted = bool(g.random() < 0.4)
    variant = MOE_VARIANTS[int(g.integers(len(MOE_VARIANTS)))]
    what = f"seed={seed} P={P} E={E} k={k} T={T} H={H} {dtype.__name__} {place} weighted={weighted} {variant}"
    print(what, flush=True)
    with nuna.tunables(**variant):
        _moe_case(nuna, g, what, P, E, k, T, H, dtype, place, weighted, seed)


def _moe_case(nuna, g, what, P, E, k, T, H, dtype, place, weighted, seed):
    topk = wl.moe_routing(P, T, k, E, 20000 + seed)
    lay = nuna.A2ALayout(topk, E).upload()
    rows = lay.recv_rows()
    cap = max(int(rows.max()) if rows.size else 0, 1)
    send_np = [a.reshape(T, H) for a in wl.random_bits(P, T * H, dtype, 30000 + seed)]
    send = [to_dev(a) if T else torch.empty((0, H), dtype=torch.bfloat16 if dtype == np.uint16 else torch.float32,
                                            device="cuda") for a in send_np]
    recv = [torch.zeros((cap, H), dtype=send[0].dtype, device="cuda") for _ in range(P)]
    if T:
        nuna.all_to_all(send, recv, lay, placement=place)
        torch.cuda.synchronize()
        ref = oracle.all_to_all(send_np, topk, E)
        for d in range(P):
            got = to_host(recv[d][:int(rows[d])])
            assert np.array_equal(got.view(np.uint8), ref[d].view(np.uint8)), f"{what} dispatch rank {d}"
    y_np = wl.result_rows(rows, H, dtype, 40000 + seed)
    y = [torch.zeros((cap, H), dtype=send[0].dtype, device="cuda") for _ in range(P)]
    for d in range(P):
        if int(rows[d]):
            y[d][:int(rows[d])] = to_dev(y_np[d])
    w_np = g.random((P, T, P)).astype(np.float32) if weighted else None
    out = [torch.empty((T, H), dtype=send[0].dtype, device="cuda") for _ in range(P)]
    if T:
        nuna.all_to_all_combine(y, out, lay, placement=place, weights=to_dev(w_np) if weighted else None)
        torch.cuda.synchronize()
        ref = oracle.combine(y_np, topk, E, w_np)
        for s in range(P):
            assert_bitwise_nan_aware(to_host(out[s]), ref[s], f"{what} combine rank {s}")
    lay.close()
