"""GPU: collectives on buffers of more than 2^31 elements per rank (64-bit indexing throughout).

Inputs are generated on the device from an index formula, v(r, i) = ((i * A + r * B) mod 17) - 8,
integers in [-8, 8] that bf16 holds exactly; every sum of 8 of them is exact in fp32, so the
expected value of any sampled output is the same formula summed on the host.  Sampled outputs
include both ends, the neighbourhood of element 2^31 and the ragged tail.  About 64 GiB of device
memory at most.
"""
import numpy as np
import pytest

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

torch = pytest.importorskip("torch")

A, B, MOD = 2654435761, 97, 17
P = 8


def _fill(t, r, base=0, chunk=1 << 27):
    """t[i] = v(r, base + i), written in chunks."""
    n = t.numel()
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        idx = torch.arange(base + s, base + e, dtype=torch.int64, device="cuda")
        t[s:e] = ((idx * A + r * B) % MOD - 8).to(torch.bfloat16)
        del idx


def _v(r, i):
    return ((np.asarray(i, dtype=np.int64) * A + r * B) % MOD) - 8


def _samples(n, rng):
    pts = [0, 1, 2, 7, 8, n - 1, n - 2, n - 9, n // 2, (1 << 31) - 1, 1 << 31, (1 << 31) + 1]
    pts += list(range(max(0, (1 << 31) - 40), min(n, (1 << 31) + 40)))
    pts += rng.integers(0, n, size=2000).tolist()
    return np.unique(np.array([p for p in pts if 0 <= p < n], dtype=np.int64))


def _get(t, idx):
    return t[torch.from_numpy(idx).cuda()].float().cpu().numpy()


@pytest.fixture(scope="module")
def nuna():
    from paper_2608_00867_amd import nuna as n
    n.init()
    return n


@pytest.mark.parametrize("algo", ["one_shot", "two_shot", "two_shot_two_kernels"])
def test_allreduce_beyond_2_31_elements(nuna, algo):
    n = (1 << 31) + 27 if algo == "one_shot" else (1 << 31) + 8 * 24  # two-shot needs count % P == 0
    ins = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    for r, t in enumerate(ins):
        _fill(t, r)
    outs = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    nuna.allreduce(ins, outs, algo=algo, placement="xcd")
    torch.cuda.synchronize()
    idx = _samples(n, np.random.default_rng(5))
    exp = sum(_v(r, idx) for r in range(P)).astype(np.float32)
    for d in (0, 3, 7):
        got = _get(outs[d], idx)
        bad = np.flatnonzero(got != exp)
        assert bad.size == 0, f"{algo} rank {d}: {bad.size} mismatches, first at element {idx[bad[0]]}"
    del ins, outs
    torch.cuda.empty_cache()


def test_reduce_scatter_and_all_gather_beyond_2_31_elements(nuna):
    m = (1 << 28) + 5  # P * m > 2^31 elements per input (reduce-scatter) and per output (all-gather)
    ins = [torch.empty(P * m, dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    for r, t in enumerate(ins):
        _fill(t, r)
    shards = [torch.empty(m, dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    nuna.reduce_scatter(ins, shards, placement="xcd")
    torch.cuda.synchronize()
    del ins
    torch.cuda.empty_cache()
    rng = np.random.default_rng(6)
    j = np.unique(np.concatenate([[0, 1, m - 1, m - 2], rng.integers(0, m, size=500)]))
    for q in (0, 4, 7):
        exp = sum(_v(r, q * m + j) for r in range(P)).astype(np.float32)
        assert np.array_equal(_get(shards[q], j), exp), f"reduce-scatter shard {q}"
    gathered = [torch.empty(P * m, dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    nuna.all_gather(shards, gathered, placement="xcd")
    torch.cuda.synchronize()
    idx = _samples(P * m, rng)
    exp = np.zeros(idx.size, dtype=np.float32)
    for r in range(P):
        exp += _v(r, idx)
    for d in (0, 5):
        assert np.array_equal(_get(gathered[d], idx), exp), f"all-gather rank {d}"
    del shards, gathered
    torch.cuda.empty_cache()
