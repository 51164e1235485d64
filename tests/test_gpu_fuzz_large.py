"""GPU: seeded random calls at large sizes through the C ABI against the oracle, bit for bit, with guard
bands around every output: the all-reduce, the reduce-scatter, the all-gather, the MoE dispatch (layout-driven
and allocation-free) and the combine.

The cases of test_gpu_fuzz.py stay below 400,000 elements in all.  These reach 24 MiB per rank (per-rank
bytes log-uniform from one element, half of them snapped near a power of two or to whole 16-byte vectors:
two-shot shards for the all-reduce, shards for the others), where the size rules switch to the 8-vector
one-shot, write-through and paced stores, and the fused or two-kernel two-shot.  Rank counts, dtypes,
algorithms, placements and in-place forms are drawn at random.  Half of the cases also set one family of
tunables: vectors per thread and workgroup size, store pauses, store cache policy, two-shot form, shard
order, page groups, or a workgroup cap.  The MoE cases draw rank counts, experts per rank, top-k, tokens per
rank, row widths, dtypes, gate weights and placements, and half of the combines set one combine tunable.
Tunables change launch shapes only, never results, so every case must give the oracle's bits.  The draw is
fixed by its seed; each case's id names it.
"""
import numpy as np
import pytest

import oracle
from gpu_util import assert_bitwise, gate_weights, run_a2a, run_combine, to_dev, to_host
from paper_2608_00867_amd import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

RANKS = [1, 2, 3, 4, 5, 7, 8, 8, 8, 9, 16, 17, 24, 32, 64]
AR_ALGOS = ["one_shot", "one_shot_split", "two_shot", "two_shot_two_kernels", "auto"]
PLACES = ["linear", "xcd"]
GUARD = 64


def _tunable(rng):
    """No tunable (half the cases) or one family of launch-shape tunables; 'cap' is a workgroup cap."""
    k = int(rng.integers(0, 14))
    if k < 7:
        return {}
    if k == 7:
        return {"NUNA_VPT": int(rng.choice([1, 2, 4, 8])), "NUNA_WG_THREADS": int(rng.choice([64, 128, 256]))}
    if k == 8:
        return {"NUNA_STORE_GAP": int(rng.choice([0, 1, 3]))}
    if k == 9:
        return {"NUNA_WRITE_THROUGH": int(rng.choice([1, 2]))}
    if k == 10:
        return {"NUNA_TWO_SHOT_FORM": int(rng.choice([1, 2]))}
    if k == 11:
        return {"NUNA_SHARD_XCD": int(rng.choice([1, 2]))}
    if k == 12:
        return {"NUNA_PAGE_GROUPS": 1}
    return {"cap": int(rng.choice([1, 7, 64, 1000]))}


def _size(rng, es, copies, multiple, max_total):
    """Elements per buffer: log-uniform bytes from one element up to max_total / copies bytes (at most
    24 MiB), `copies` being how many such buffers one side of the call holds; a quarter snapped to a power
    of two plus or minus a few elements, a quarter to a multiple of `multiple`."""
    hi = min(24 << 20, max_total // copies) // es
    n = max(1, int(np.exp(rng.uniform(0.0, np.log(hi)))))
    snap = rng.random()
    if snap < 0.25:
        n = max(1, (1 << int(np.log2(n))) + int(rng.integers(-3, 4)))
    elif snap < 0.5:
        n = max(multiple, n // multiple * multiple)
    return min(n, hi)


def _cases(kind, count, seed):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        P = int(rng.choice(RANKS))
        dtype = str(rng.choice(["f32", "bf16"]))
        es = 4 if dtype == "f32" else 2
        if kind == "ar":  # elements per rank; snapped to whole two-shot shards of 16-byte vectors
            n = _size(rng, es, P, 8 * P, 192 << 20)
            algo = str(rng.choice(AR_ALGOS))
        else:  # shard elements per rank; an RS input or AG output holds P of them, P buffers in all
            n = _size(rng, es, P * P, 8, 192 << 20)
            algo = None
        place = str(rng.choice(PLACES))
        in_place = bool(rng.random() < 0.25)
        tun = _tunable(rng)
        desc = [f"{kind}{i:02d}", f"P{P}", f"n{n}", dtype, place] + ([algo] if algo else []) + \
            (["inplace"] if in_place else []) + [f"{k.replace('NUNA_', '')}={v}" for k, v in tun.items()]
        out.append(pytest.param(dict(P=P, n=n, dtype=dtype, algo=algo, place=place, in_place=in_place, tun=tun,
                                     seed=seed * 1000 + i), id="-".join(desc)))
    return out


def _moe_cases(kind, count, seed):
    """Routing shapes: E = P * (experts per rank) up to 512 experts, top-k from 1 to 8 (or every expert),
    1-512 tokens per rank, rows of 1-8192 elements, at most 96 MiB of rows received in all."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        P = int(rng.choice([1, 2, 3, 4, 5, 8, 8, 8, 16, 64]))
        per = int(rng.choice([1, 2, 4, 8, 32]))
        E = P * max(1, min(per, 512 // P))
        k = E if (E <= 64 and rng.random() < 0.1) else int(rng.integers(1, min(E, 8) + 1))
        dtype = str(rng.choice(["f32", "bf16"]))
        es = 4 if dtype == "f32" else 2
        H = int(np.exp(rng.uniform(0.0, np.log(8192))))
        if kind == "routed":  # the routed dispatch moves whole 16-byte vectors
            H = max(16 // es, H // (16 // es) * (16 // es))
        T = int(np.exp(rng.uniform(0.0, np.log(512))))
        T = max(1, min(T, (96 << 20) // (P * H * es * min(k, P))))
        place = str(rng.choice(PLACES))
        weighted = kind == "combine" and bool(rng.random() < 0.5)
        tun = {}
        if kind == "combine":
            j = int(rng.integers(0, 8))
            tun = ({"NUNA_COMBINE_VPT": int(rng.choice([1, 2, 4]))} if j == 4 else
                   {"NUNA_COMBINE_LISTS": 1} if j == 5 else
                   {"NUNA_COMBINE_CHUNKS": int(rng.integers(1, 9))} if j == 6 else
                   {"cap": int(rng.choice([1, 13, 200]))} if j == 7 else {})
        elif rng.random() < 0.25:
            tun = {"cap": int(rng.choice([1, 13, 200]))}
        misalign = kind == "routed" and bool(rng.random() < 0.25)
        desc = [f"{kind}{i:02d}", f"P{P}", f"E{E}", f"k{k}", f"T{T}", f"H{H}", dtype, place] + \
            (["weighted"] if weighted else []) + (["misaligned"] if misalign else []) + \
            [f"{a.replace('NUNA_', '')}={v}" for a, v in tun.items()]
        out.append(pytest.param(dict(P=P, E=E, k=k, T=T, H=H, dtype=dtype, place=place, weighted=weighted,
                                     misalign=misalign, tun=tun, seed=seed * 1000 + i), id="-".join(desc)))
    return out


def _inputs(c, n):
    if c["dtype"] == "bf16":
        return wl.normal_bf16(c["P"], n, c["seed"])
    return wl.normal_f32(c["P"], n, c["seed"])


def _guarded(n, dtype):
    whole = torch.empty(n + 2 * GUARD, dtype=dtype, device="cuda")
    whole.view(torch.int16 if dtype == torch.bfloat16 else torch.int32).fill_(0x5A5A)
    return whole[GUARD:GUARD + n], whole


def _guards_intact(whole, n, what):
    w = whole.view(torch.int16 if whole.dtype == torch.bfloat16 else torch.int32).cpu().numpy()
    assert np.all(w[:GUARD] == 0x5A5A) and np.all(w[GUARD + n:] == 0x5A5A), f"{what}: write outside the output"


class _Tuned:
    """Set one case's tunables (or workgroup cap) and restore the defaults afterwards."""

    def __init__(self, nuna, tun):
        self.nuna, self.tun = nuna, dict(tun)

    def __enter__(self):
        cap = self.tun.pop("cap", 0)
        self.ctx = self.nuna.tunables(**self.tun)
        self.ctx.__enter__()
        self.nuna.set_max_workgroups(cap)

    def __exit__(self, *exc):
        self.nuna.set_max_workgroups(0)
        self.ctx.__exit__(*exc)
        return False


@pytest.fixture(scope="module")
def nuna():
    from paper_2608_00867_amd import nuna as n
    n.init()
    return n


@pytest.fixture(autouse=True)
def _free():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("c", _cases("ar", 128, 7301))
def test_allreduce_random(nuna, c):
    P, n = c["P"], c["n"]
    x = _inputs(c, n)
    ref = oracle.allreduce(x)
    ins = [to_dev(a) for a in x]
    with _Tuned(nuna, c["tun"]):
        if c["in_place"]:
            nuna.allreduce(ins, ins, algo=c["algo"], placement=c["place"])
            torch.cuda.synchronize()
            outs, wholes = ins, None
        else:
            pairs = [_guarded(n, ins[0].dtype) for _ in range(P)]
            outs, wholes = [p[0] for p in pairs], [p[1] for p in pairs]
            nuna.allreduce(ins, outs, algo=c["algo"], placement=c["place"])
            torch.cuda.synchronize()
    for d in range(P):
        if wholes is not None:
            _guards_intact(wholes[d], n, f"rank {d}")
        assert_bitwise(to_host(outs[d]), ref[d], f"rank {d}")


@pytest.mark.parametrize("c", _cases("rs", 64, 7302))
def test_reduce_scatter_random(nuna, c):
    P, m = c["P"], c["n"]
    x = _inputs(c, P * m)
    ref = oracle.reduce_scatter(x)
    ins = [to_dev(a) for a in x]
    aligned = (m * ins[0].element_size()) % 16 == 0 or P == 1
    with _Tuned(nuna, c["tun"]):
        if c["in_place"] and aligned:
            outs, wholes = [ins[r][r * m:(r + 1) * m] for r in range(P)], None
        else:
            pairs = [_guarded(m, ins[0].dtype) for _ in range(P)]
            outs, wholes = [p[0] for p in pairs], [p[1] for p in pairs]
        nuna.reduce_scatter(ins, outs, placement=c["place"])
        torch.cuda.synchronize()
    for r in range(P):
        if wholes is not None:
            _guards_intact(wholes[r], m, f"rank {r}")
        assert_bitwise(to_host(outs[r]), ref[r], f"rank {r}")


@pytest.mark.parametrize("c", _cases("ag", 64, 7303))
def test_all_gather_random(nuna, c):
    P, m = c["P"], c["n"]
    x = wl.random_bits(P, m, np.uint16 if c["dtype"] == "bf16" else np.float32, c["seed"])
    ref = oracle.all_gather(x)
    ins = [to_dev(a) for a in x]
    aligned = (m * ins[0].element_size()) % 16 == 0 or P == 1
    with _Tuned(nuna, c["tun"]):
        if c["in_place"] and aligned:
            outs = [torch.zeros(P * m, dtype=ins[0].dtype, device="cuda") for _ in range(P)]
            for r in range(P):
                outs[r][r * m:(r + 1) * m].copy_(ins[r])
            srcs, wholes = [outs[r][r * m:(r + 1) * m] for r in range(P)], None
        else:
            pairs = [_guarded(P * m, ins[0].dtype) for _ in range(P)]
            outs, wholes, srcs = [p[0] for p in pairs], [p[1] for p in pairs], ins
        nuna.all_gather(srcs, outs, placement=c["place"])
        torch.cuda.synchronize()
    for d in range(P):
        if wholes is not None:
            _guards_intact(wholes[d], P * m, f"rank {d}")
        assert_bitwise(to_host(outs[d]), ref[d], f"rank {d}")


@pytest.mark.parametrize("c", _moe_cases("dispatch", 32, 7304))
def test_dispatch_random(nuna, c):
    P, T, H = c["P"], c["T"], c["H"]
    dt = np.uint16 if c["dtype"] == "bf16" else np.float32
    topk = wl.moe_routing(P, T, c["k"], c["E"], c["seed"])
    send = [a.reshape(T, H) for a in wl.random_bits(P, T * H, dt, c["seed"] + 1)]
    ref = oracle.all_to_all(send, topk, c["E"])
    with _Tuned(nuna, c["tun"]):
        got = run_a2a(nuna, send, topk, c["E"], c["place"])
    for d in range(P):
        assert_bitwise(got[d], ref[d], f"rank {d}")


@pytest.mark.parametrize("c", _moe_cases("combine", 32, 7305))
def test_combine_random(nuna, c):
    P, T, H, E = c["P"], c["T"], c["H"], c["E"]
    dt = np.uint16 if c["dtype"] == "bf16" else np.float32
    topk = wl.moe_routing(P, T, c["k"], E, c["seed"])
    y = wl.result_rows(oracle.a2a_counts(topk, E), H, dt, c["seed"] + 1)
    w = gate_weights(topk, E, c["seed"] + 2) if c["weighted"] else None
    ref = oracle.combine(y, topk, E, w)
    with _Tuned(nuna, c["tun"]):
        got = run_combine(nuna, y, topk, E, c["place"], weights=w)
    for s in range(P):
        assert_bitwise(got[s], ref[s], f"rank {s}")


@pytest.mark.parametrize("c", _moe_cases("routed", 48, 7306))
def test_routed_dispatch_random(nuna, c):
    """The allocation-free dispatch (one kernel up to 256 tokens over all ranks, else routing then copy):
    receive rows and row counts against the oracle, sentinel rows past each rank's count untouched; a
    quarter of the top-k tables sit 4 bytes past a 16-byte boundary."""
    P, T, H, E = c["P"], c["T"], c["H"], c["E"]
    dt = np.uint16 if c["dtype"] == "bf16" else np.float32
    topk = wl.moe_routing(P, T, c["k"], E, c["seed"])
    send_np = [a.reshape(T, H) for a in wl.random_bits(P, T * H, dt, c["seed"] + 1)]
    ref = oracle.all_to_all(send_np, topk, E)
    rows = [r.shape[0] for r in ref]
    cap = max(rows) + 2
    send = [to_dev(a) for a in send_np]
    tdt = send[0].dtype
    sentinel = 0x7FA5 if tdt == torch.bfloat16 else 0x7FA5A5A5
    ity = torch.int16 if tdt == torch.bfloat16 else torch.int32
    recv = [torch.full((cap, H), sentinel, dtype=ity, device="cuda").view(tdt) for _ in range(P)]
    flat = torch.from_numpy(np.ascontiguousarray(topk, dtype=np.int32).reshape(-1))
    if c["misalign"]:
        buf = torch.zeros(flat.numel() + 1, dtype=torch.int32, device="cuda")
        buf[1:].copy_(flat)
        topk_dev = buf[1:].view(topk.shape)
    else:
        topk_dev = flat.cuda().view(topk.shape)
    rows_dev = torch.full((P + 1,), -1, dtype=torch.int64, device="cuda")
    with _Tuned(nuna, c["tun"]):
        nuna.all_to_all_routed(send, recv, topk_dev, E, rows_dev, placement=c["place"])
        torch.cuda.synchronize()
    assert rows_dev.cpu().tolist() == rows + [0]
    for d in range(P):
        got = to_host(recv[d])
        assert_bitwise(got[:rows[d]], ref[d], f"rank {d}")
        past = got[rows[d]:].view(np.int16 if tdt == torch.bfloat16 else np.int32)
        assert np.all(past == np.array(sentinel, dtype=past.dtype)), f"rank {d}: rows past the count written"
