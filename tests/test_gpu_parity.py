"""GPU parity: the HIP path through the C ABI against the CPU oracle, element by element.

Bar: bit-exact everywhere.  Reductions add ranks in ascending order with fp32
accumulation and one rounding on both sides, copies move bytes.  The only
relaxation is for NaN results of arithmetic (inf - inf), whose payload IEEE-754
leaves to the implementation: there only NaN-ness is compared.

Cases: the five workloads at full size (decode / prefill all-reduce, fp32
integer all-reduce, P=64 all-reduce, MoE all-to-all dispatch) and the MoE
combine that reverses the dispatch, both placement
modes, every algorithm, plus ragged and tiny sizes, in-place forms, special
values, guard bands around every output, persistent-loop launches and HIP
graph replay.
"""
import numpy as np
import pytest

import oracle
from gpu_util import assert_bitwise, assert_bitwise_nan_aware, gate_weights, run_a2a, run_combine, to_dev, \
    to_host
from paper_2608_00867_amd import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

PLACES = ["linear", "xcd"]
AR_ALGOS = ["one_shot", "one_shot_split", "two_shot", "two_shot_two_kernels", "auto"]


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


def _guarded(shape_elems, dtype, pad=256):
    """A CUDA buffer with `pad` sentinel elements on both sides; returns (view, whole)."""
    whole = torch.empty(shape_elems + 2 * pad, dtype=dtype, device="cuda")
    whole.view(torch.int16 if dtype == torch.bfloat16 else torch.int32).fill_(0x5A5A)
    return whole[pad:pad + shape_elems], whole


def _check_guards(whole, n, pad=256):
    w = whole.view(torch.int16 if whole.dtype == torch.bfloat16 else torch.int32).cpu().numpy()
    assert np.all(w[:pad] == 0x5A5A) and np.all(w[pad + n:] == 0x5A5A), "write outside the output buffer"


def run_allreduce(nuna, x, algo, place, guard=True):
    ins = [to_dev(a) for a in x]
    dt = ins[0].dtype
    n = x[0].size
    if guard:
        pairs = [_guarded(n, dt) for _ in x]
        outs = [p[0] for p in pairs]
    else:
        outs = [torch.empty_like(t) for t in ins]
    nuna.allreduce(ins, outs, algo=algo, placement=place)
    torch.cuda.synchronize()
    if guard:
        for _, whole in pairs:
            _check_guards(whole, n)
    return [to_host(o) for o in outs]


# ---------------------------------------------------------------- placement proof

@pytest.mark.parametrize("G", [8, 64, 1000, 4096])
def test_probe_workgroup_b_runs_on_xcd_b_mod_8(nuna, G):
    xcc, hw = nuna.probe_xcc(G)
    torch.cuda.synchronize()
    x = xcc.cpu().numpy()
    assert np.array_equal(x, np.arange(G) % 8), np.unique(x - np.arange(G) % 8)


def test_init_verified_the_dispatch_map(nuna):
    """nuna_init probed the device: 256 compute units in 8 XCDs, workgroup b on XCD b mod 8."""
    info = nuna.device_info()
    assert info["map_verified"] == 1 and info["cu_count"] == 256 and info["xcd_count"] == 8, info
    xcc, _ = nuna.probe_xcc(4096)
    torch.cuda.synchronize()
    assert nuna.check_dispatch_map_raw(xcc.cpu().numpy(), info["cu_count"]) == nuna.OK, nuna.last_error()


@pytest.mark.parametrize("items,chunk", [(16, 1024), (100, 1024), (4096, 1024), (1000, 256), (8192, 256)])
def test_page_groups_run_on_one_xcd(nuna, items, chunk):
    """Placement proof of the page-grouped map: a launch of the direct map's grid records the XCC each
    workgroup ran on; every page's chunks ran on one XCD, XCD (page mod 8)."""
    with nuna.tunables(NUNA_PAGE_GROUPS=1):
        m = nuna.placement_direct("xcd", items, chunk)
    xcc, _ = nuna.probe_xcc(int(m.size))
    torch.cuda.synchronize()
    x = xcc.cpu().numpy()
    gp = 4096 // chunk
    for b, w in enumerate(m):
        if w >= 0:
            assert x[b] == (w // gp) % 8, (b, w, x[b])


# ---------------------------------------------------------------- workload 1: fp32 integers, P=8, n=2048

@pytest.mark.parametrize("place", PLACES)
@pytest.mark.parametrize("algo", AR_ALGOS)
def test_ar_f32_int_p8(nuna, algo, place):
    x = wl.ar_f32_int()
    ref = oracle.allreduce(x)
    got = run_allreduce(nuna, x, algo, place)
    exact = np.sum(np.stack(x).astype(np.int64), axis=0)
    for d in range(8):
        assert_bitwise(got[d], ref[d], f"rank {d}")
        assert np.array_equal(got[d].astype(np.int64), exact)


# ---------------------------------------------------------------- workload 2: decode all-reduce bf16, P=8

@pytest.mark.parametrize("place", PLACES)
@pytest.mark.parametrize("algo", AR_ALGOS)
@pytest.mark.parametrize("T", wl.DECODE_TOKENS)
def test_ar_bf16_decode(nuna, T, algo, place):
    x = wl.ar_bf16_decode(T)
    ref = oracle.allreduce(x)
    got = run_allreduce(nuna, x, algo, place)
    for d in range(8):
        assert_bitwise(got[d], ref[d], f"T={T} rank {d}")


# ---------------------------------------------------------------- workload 3: prefill two-shot bf16, P=8

@pytest.mark.parametrize("place", PLACES)
@pytest.mark.parametrize("algo", ["two_shot", "two_shot_two_kernels", "one_shot"])
@pytest.mark.parametrize("T", wl.PREFILL_TOKENS)
def test_ar_bf16_prefill(nuna, T, algo, place):
    x = wl.ar_bf16_prefill(T)
    ref = oracle.allreduce(x)
    got = run_allreduce(nuna, x, algo, place, guard=(T <= 1024))
    for d in range(8):
        assert_bitwise(got[d], ref[d], f"T={T} rank {d}")


# ---------------------------------------------------------------- workload 5: P=64 bf16

@pytest.mark.parametrize("place", PLACES)
@pytest.mark.parametrize("algo", ["one_shot", "one_shot_split", "two_shot", "two_shot_two_kernels"])
@pytest.mark.parametrize("kib", wl.P64_KIB)
def test_ar_bf16_p64(nuna, kib, algo, place):
    x = wl.ar_bf16_p64(kib)
    ref = oracle.allreduce(x)
    got = run_allreduce(nuna, x, algo, place)
    for d in (0, 1, 31, 63):
        assert_bitwise(got[d], ref[d], f"{kib} KiB rank {d}")
    for d in range(64):
        assert_bitwise(got[d], got[0], f"{kib} KiB rank {d} vs rank 0")


# ---------------------------------------------------------------- ragged and tiny sizes

RAGGED_N = [1, 3, 7, 8, 9, 255, 4095, 4096, 4097, 2048 * 3 + 5, 70001]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("P", [1, 2, 3, 5, 8, 16, 24, 64])
def test_ar_ragged(nuna, P, dtype):
    for n in RAGGED_N:
        if P == 64 and n > 4097:
            continue
        seed = 1000 * P + n
        x = wl.normal_f32(P, n, seed) if dtype == "f32" else wl.normal_bf16(P, n, seed)
        ref = oracle.allreduce(x)
        for algo in AR_ALGOS:
            for place in PLACES:
                got = run_allreduce(nuna, x, algo, place)
                for d in range(P):
                    assert_bitwise(got[d], ref[d], f"P={P} n={n} {dtype} {algo} {place} rank {d}")


@pytest.mark.parametrize("P", [2, 4, 8, 16])
def test_ar_large_ragged(nuna, P):
    """Messages of 4-16 MiB per rank use several vectors per thread; ragged sizes end in a partial
    chunk and a scalar tail.  Also under a workgroup cap (persistent loop)."""
    for n, seed in ((2 ** 21 + 8 * 3 + 5, 1), (2 ** 23 + 8 * 1000 + 3, 2)):
        if P == 16 and n > 2 ** 22:
            continue
        x = wl.normal_bf16(P, n, 900 + P + seed)
        ref = oracle.allreduce(x)
        try:
            for cap in (0, 100):
                nuna.set_max_workgroups(cap)
                for algo in ("one_shot", "two_shot"):
                    for place in PLACES:
                        got = run_allreduce(nuna, x, algo, place, guard=True)
                        for d in range(P):
                            assert_bitwise(got[d], ref[d], f"P={P} n={n} cap={cap} {algo} {place} rank {d}")
        finally:
            nuna.set_max_workgroups(0)


@pytest.mark.parametrize("algo", AR_ALGOS)
def test_ar_in_place(nuna, algo):
    for P, n, dtype in [(8, 8192 * 4, "bf16"), (8, 4097, "f32"), (64, 8192, "bf16"), (3, 999, "bf16")]:
        x = wl.normal_bf16(P, n, 7 + P) if dtype == "bf16" else wl.normal_f32(P, n, 7 + P)
        ref = oracle.allreduce(x)
        for place in PLACES:
            bufs = [to_dev(a) for a in x]
            nuna.allreduce(bufs, bufs, algo=algo, placement=place)
            torch.cuda.synchronize()
            for d in range(P):
                assert_bitwise(to_host(bufs[d]), ref[d], f"in-place P={P} n={n} {algo} {place} rank {d}")


def test_ar_special_values(nuna):
    """-0.0 sums, denormals, overflow to inf, inf-inf NaN, NaN inputs."""
    P, n = 8, 4096
    rng = np.random.default_rng(5)
    for dt in (np.float32, np.uint16):
        view = np.uint32 if dt == np.float32 else np.uint16
        if dt == np.float32:
            specials = np.array([0x80000000, 0x00000001, 0x807FFFFF, 0x7F7FFFFF, 0xFF7FFFFF, 0x7F800000, 0xFF800000,
                                 0x7FC00000, 0x00800000, 0x3F800000], dtype=np.uint32)
        else:
            specials = np.array([0x8000, 0x0001, 0x807F, 0x7F7F, 0xFF7F, 0x7F80, 0xFF80, 0x7FC0, 0x0080, 0x3F80],
                                dtype=np.uint16)
        x = [specials[rng.integers(0, specials.size, size=n)].view(dt) for _ in range(P)]
        x[0][:64] = np.full(64, specials[0], dtype=view).view(dt)  # some all -0 columns
        for r in range(P):
            x[r][:64] = np.full(64, specials[0], dtype=view).view(dt)
        ref = oracle.allreduce(x)
        for algo in ("one_shot", "one_shot_split", "two_shot"):
            for place in PLACES:
                got = run_allreduce(nuna, x, algo, place)
                for d in range(P):
                    assert_bitwise_nan_aware(got[d], ref[d], f"specials {dt.__name__} {algo} {place} rank {d}")
                assert np.all(got[0].view(view)[:64] == specials[0])


def test_ar_persistent_loop(nuna):
    """Fewer workgroups than work items: every workgroup loops over its items."""
    x = wl.normal_bf16(8, 8192 * 64 + 24, 77)
    ref = oracle.allreduce(x)
    try:
        for cap in (1, 7, 8, 13, 64):
            nuna.set_max_workgroups(cap)
            for algo in AR_ALGOS:
                for place in PLACES:
                    got = run_allreduce(nuna, x, algo, place)
                    for d in range(8):
                        assert_bitwise(got[d], ref[d], f"cap={cap} {algo} {place} rank {d}")
    finally:
        nuna.set_max_workgroups(0)


# ---------------------------------------------------------------- reduce-scatter / all-gather standalone

@pytest.mark.parametrize("place", PLACES)
@pytest.mark.parametrize("P,m,dtype", [(8, 65536, "bf16"), (8, 1000, "bf16"), (8, 3, "f32"), (2, 4096, "f32"),
                                       (5, 777, "bf16"), (64, 2048, "bf16"), (1, 100, "f32"), (8, 4096 * 64, "bf16"),
                                       (8, 2 ** 17 + 1024 + 8, "bf16"), (4, 2 ** 18 + 8, "bf16")])
def test_reduce_scatter(nuna, P, m, dtype, place):
    x = wl.normal_bf16(P, P * m, 3 * m + P) if dtype == "bf16" else wl.normal_f32(P, P * m, 3 * m + P)
    ref = oracle.reduce_scatter(x)
    ins = [to_dev(a) for a in x]
    pairs = [_guarded(m, ins[0].dtype) for _ in range(P)]
    outs = [p[0] for p in pairs]
    nuna.reduce_scatter(ins, outs, placement=place)
    torch.cuda.synchronize()
    for r in range(P):
        _check_guards(pairs[r][1], m)
        assert_bitwise(to_host(outs[r]), ref[r], f"RS P={P} m={m} rank {r}")
    # in-place form: out[r] is shard r of in[r] (the ABI needs 16-byte aligned shards)
    bufs = [to_dev(a) for a in x]
    shard_views = [bufs[r][r * m:(r + 1) * m] for r in range(P)]
    if (m * bufs[0].element_size()) % 16 and P > 1:
        with pytest.raises(nuna.NunaError) as e:
            nuna.reduce_scatter(bufs, shard_views, placement=place)
        assert e.value.status == nuna.ERR_MISALIGNED
        return
    nuna.reduce_scatter(bufs, shard_views, placement=place)
    torch.cuda.synchronize()
    for r in range(P):
        assert_bitwise(to_host(shard_views[r]), ref[r], f"RS in-place P={P} m={m} rank {r}")


@pytest.mark.parametrize("place", PLACES)
@pytest.mark.parametrize("P,m,dtype", [(8, 65536, "bf16"), (8, 1000, "bf16"), (8, 3, "f32"), (3, 4096, "f32"),
                                       (2, 4096, "bf16"), (4, 2 ** 18 + 8, "bf16"), (2, 70001 * 4, "f32"),
                                       (64, 512, "bf16"), (1, 64, "bf16"), (8, 4096 * 64, "bf16"),
                                       (8, 2 ** 17 + 1024 + 8, "bf16"),
                                       # 8-rank shards on both sides of the launch-shape boundaries at 2, 4
                                       # and 16 MiB, ragged and not
                                       (8, 2 ** 20, "bf16"), (8, 2 ** 20 + 8, "bf16"), (8, 3 * 2 ** 19 + 8, "bf16"),
                                       (8, 2 ** 21 + 8, "bf16"), (8, 2 ** 22 - 8, "bf16"), (8, 2 ** 20 + 4, "f32"),
                                       (8, 2 ** 22, "bf16"), (8, 2 ** 22 + 8, "bf16"), (8, 2 ** 23 + 24, "bf16")])
def test_all_gather(nuna, P, m, dtype, place):
    x = wl.random_bits(P, m, np.uint16 if dtype == "bf16" else np.float32, 5 * m + P)
    ref = oracle.all_gather(x)
    ins = [to_dev(a) for a in x]
    pairs = [_guarded(P * m, ins[0].dtype) for _ in range(P)]
    outs = [p[0] for p in pairs]
    nuna.all_gather(ins, outs, placement=place)
    torch.cuda.synchronize()
    for d in range(P):
        _check_guards(pairs[d][1], P * m)
        assert_bitwise(to_host(outs[d]), ref[d], f"AG P={P} m={m} rank {d}")
    # in-place form: in[r] is shard r of out[r] (the ABI needs 16-byte aligned shards)
    if (m * ins[0].element_size()) % 16 and P > 1:
        return
    bufs = [torch.zeros(P * m, dtype=ins[0].dtype, device="cuda") for _ in range(P)]
    for r in range(P):
        bufs[r][r * m:(r + 1) * m].copy_(ins[r])
    nuna.all_gather([bufs[r][r * m:(r + 1) * m] for r in range(P)], bufs, placement=place)
    torch.cuda.synchronize()
    for d in range(P):
        assert_bitwise(to_host(bufs[d]), ref[d], f"AG in-place P={P} m={m} rank {d}")


# ---------------------------------------------------------------- workload 4: MoE all-to-all dispatch



@pytest.mark.parametrize("place", PLACES)
def test_a2a_moe_full(nuna, place):
    send, topk = wl.a2a_moe()
    ref = oracle.all_to_all(send, topk, wl.MOE_EXPERTS)
    got = run_a2a(nuna, send, topk, wl.MOE_EXPERTS, place)
    for d in range(8):
        assert_bitwise(got[d], ref[d], f"a2a rank {d}")


@pytest.mark.parametrize("place", PLACES)
@pytest.mark.parametrize("P,T,k,E,H,dtype", [(8, 16, 8, 256, 7168, np.uint16), (2, 5, 1, 2, 8, np.uint16),
                                             (3, 7, 2, 6, 13, np.uint16), (4, 33, 3, 16, 5, np.float32),
                                             (64, 4, 8, 256, 64, np.uint16), (8, 1, 8, 64, 7168, np.uint16),
                                             (1, 9, 1, 4, 256, np.float32)])
def test_a2a_small(nuna, P, T, k, E, H, dtype, place):
    topk = wl.moe_routing(P, T, k, E, 17 * P + T)
    send = [a.reshape(T, H) for a in wl.random_bits(P, T * H, dtype, 19 * P + T)]
    ref = oracle.all_to_all(send, topk, E)
    got = run_a2a(nuna, send, topk, E, place)
    for d in range(P):
        assert_bitwise(got[d], ref[d], f"a2a P={P} T={T} H={H} rank {d}")


@pytest.mark.parametrize("n", [(1 << 20) + 5, (1 << 22) + 3, (1 << 24) + 8])
def test_ar_f32_large_every_algo(nuna, n):
    """fp32 messages of 4, 16 and 64 MiB per rank at the default launch shapes (their chunk sizes use
    4, 2 and 1 vectors per thread); every algorithm and placement."""
    x = wl.normal_f32(8, n, 53 + n % 97)
    ref = oracle.allreduce(x)
    for place in PLACES:
        for algo in AR_ALGOS:
            got = run_allreduce(nuna, x, algo, place, guard=False)
            for d in range(8):
                assert_bitwise(got[d], ref[d], f"f32 n={n} {algo} {place} rank {d}")


# ---------------------------------------------------------------- launch-shape variants (tunables)

def _ar_vs_oracle(nuna, x, what):
    ref = oracle.allreduce(x)
    got = run_allreduce(nuna, x, "one_shot", "xcd")
    for d in range(len(x)):
        assert_bitwise(got[d], ref[d], f"{what} rank {d}")


@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
@pytest.mark.parametrize("V", [16, 32, 64])
def test_tile_allreduce_variants(nuna, V, dtype):
    """Rank-major tile all-reduce at every width, any rank count and ragged sizes."""
    with nuna.tunables(NUNA_TILE_V=V, NUNA_LPR_MAX_VECTORS=0, NUNA_LPR_MIN_RANKS=1):
        for P in (2, 3, 8, 16, 24, 64):
            for n in (7, 9, 1000, 4097, 70001):
                x = wl.random_bits(P, n, dtype, 97 * P + n) if n < 100 else \
                    (wl.normal_bf16(P, n, 89 * P + n) if dtype == np.uint16 else wl.normal_f32(P, n, 89 * P + n))
                if n < 100:
                    ref = oracle.allreduce(x)
                    got = run_allreduce(nuna, x, "one_shot", "linear")
                    for d in range(P):
                        assert_bitwise_nan_aware(got[d], ref[d], f"tile V={V} P={P} n={n} rank {d}")
                else:
                    _ar_vs_oracle(nuna, x, f"tile V={V} P={P} n={n}")


@pytest.mark.parametrize("cfg", [dict(NUNA_VPT=v, NUNA_WG_THREADS=t) for v in (1, 2, 4, 8) for t in (64, 128, 256)] +
                         [dict(NUNA_LPR_MIN_RANKS=1, NUNA_LPR_MAX_VECTORS=1 << 30)],  # lane per rank, P >= 1
                         ids=lambda c: ",".join(f"{k[5:]}={v}" for k, v in c.items()))
def test_launch_shape_variants(nuna, cfg):
    """Every forced launch shape gives the oracle's bits (P = 1 to 64; ragged and multi-chunk sizes)."""
    with nuna.tunables(**cfg):
        for P, n in ((1, 5003), (2, 70001), (3, 7001), (4, 70001), (8, 4097), (8, 262144 + 24), (16, 70001),
                     (64, 9000)):
            _ar_vs_oracle(nuna, wl.normal_bf16(P, n, 31 * P + n), f"{cfg} P={P} n={n}")


@pytest.mark.parametrize("gap", [0, 1, 5])
def test_store_gap_parity(nuna, gap):
    """Pauses between the per-destination stores change timing only: the one-shot (with and without
    destination split), the fused and two-kernel two-shot and the all-gather give the oracle's bits with
    the pause count forced, at 2-16 ranks, ragged and multi-chunk sizes, in place and under a grid cap."""
    with nuna.tunables(NUNA_STORE_GAP=gap):
        for P, n in ((2, 70001), (4, 4097), (8, 1), (8, 4097), (8, 262144 + 24), (16, 70001)):
            x = wl.normal_bf16(P, n, 37 * P + n + gap)
            ref = oracle.allreduce(x)
            for algo in ("one_shot", "one_shot_split", "two_shot", "two_shot_two_kernels"):
                for place in PLACES:
                    got = run_allreduce(nuna, x, algo, place)
                    for d in range(P):
                        assert_bitwise(got[d], ref[d], f"gap={gap} {algo} {place} P={P} n={n} rank {d}")
        x = wl.normal_bf16(8, 8 * 70001, 41 + gap)
        ref = oracle.allreduce(x)
        with nuna.tunables(NUNA_TWO_SHOT_FORM=1):
            got = run_allreduce(nuna, x, "two_shot", "xcd")
        for d in range(8):
            assert_bitwise(got[d], ref[d], f"gap={gap} fused two-shot rank {d}")
        nuna.set_max_workgroups(13)
        try:
            got = run_allreduce(nuna, x, "one_shot", "linear")
        finally:
            nuna.set_max_workgroups(0)
        for d in range(8):
            assert_bitwise(got[d], ref[d], f"gap={gap} capped one-shot rank {d}")
        bufs = [to_dev(a) for a in x]
        nuna.allreduce(bufs, bufs, algo="one_shot", placement="xcd")
        torch.cuda.synchronize()
        for d in range(8):
            assert_bitwise(to_host(bufs[d]), ref[d], f"gap={gap} in-place rank {d}")
        for P, m in ((8, 4096), (8, 70001 * 8), (16, 1024)):
            xs = wl.random_bits(P, m, np.uint16, 3 * m + P + gap)
            ref = oracle.all_gather(xs)
            ins = [to_dev(a) for a in xs]
            for place in PLACES:
                outs = [torch.empty(P * m, dtype=ins[0].dtype, device="cuda") for _ in range(P)]
                nuna.all_gather(ins, outs, placement=place)
                torch.cuda.synchronize()
                for d in range(P):
                    assert_bitwise(to_host(outs[d]), ref[d], f"gap={gap} AG {place} P={P} m={m} rank {d}")


@pytest.mark.parametrize("cfg", [dict(NUNA_WRITE_THROUGH=w, NUNA_VPT=v, NUNA_WG_THREADS=t)
                                 for w in (1, 2) for v, t in ((0, 0), (1, 64), (2, 128), (4, 256), (8, 256))],
                         ids=lambda c: ",".join(f"{k[5:]}={v}" for k, v in c.items()))
def test_write_through_stores(nuna, cfg):
    """The 8-rank one-shot and the two-shot's all-gather phase with write-through stores forced on (and
    off), at every launch shape: ragged chunks, one chunk, many chunks, the general kernel (grid caps),
    in place, and shards with and without whole vectors."""
    with nuna.tunables(**cfg):
        for n, dt in ((1, np.uint16), (9, np.float32), (4097, np.uint16), (70001, np.float32),
                      (2 ** 20 + 24, np.uint16), (2 ** 21 + 4, np.float32)):
            x = wl.normal_bf16(8, n, 13 * n + 5) if dt == np.uint16 else wl.normal_f32(8, n, 13 * n + 5)
            _ar_vs_oracle(nuna, x, f"{cfg} n={n}")
        x = wl.normal_bf16(8, 2 ** 19 + 40, 7)
        ref = oracle.allreduce(x)
        for cap in (7, 64):
            nuna.set_max_workgroups(cap)
            try:
                for place in PLACES:
                    got = run_allreduce(nuna, x, "one_shot", place)
                    for d in range(8):
                        assert_bitwise(got[d], ref[d], f"{cfg} cap={cap} {place} rank {d}")
            finally:
                nuna.set_max_workgroups(0)
        bufs = [to_dev(a) for a in x]
        nuna.allreduce(bufs, bufs, algo="one_shot", placement="xcd")
        torch.cuda.synchronize()
        for d in range(8):
            assert_bitwise(to_host(bufs[d]), ref[d], f"{cfg} in place rank {d}")
        # the two-shot's all-gather phase (its shards read through the caches)
        for n in (8 * 1024, 8 * 70001, 8 * 2 ** 18, 8 * (2 ** 19 + 8)):
            x = wl.normal_bf16(8, n, 11 * n + 3)
            ref = oracle.allreduce(x)
            for place in PLACES:
                got = run_allreduce(nuna, x, "two_shot", place)
                for d in range(8):
                    assert_bitwise(got[d], ref[d], f"{cfg} two-shot {place} n={n} rank {d}")


@pytest.mark.parametrize("cfg", [dict(NUNA_VPT=v, NUNA_WG_THREADS=t) for v in (0, 1, 2, 4, 8) for t in (64, 256)] +
                         [dict(NUNA_DIRECT_MAX_GRID=5), dict(NUNA_WRITE_THROUGH=2, NUNA_VPT=8, NUNA_WG_THREADS=256),
                          dict(NUNA_SHARD_XCD=2), dict(NUNA_SHARD_XCD=2, NUNA_DIRECT_MAX_GRID=5),
                          dict(NUNA_SHARD_XCD=2, NUNA_MAX_GRID=13), dict(NUNA_SHARD_XCD=1)],
                         ids=lambda c: ",".join(f"{k[5:]}={v}" for k, v in c.items()))
def test_two_shot_fused(nuna, cfg):
    """The fused two-shot (both phases per chunk in one kernel) at every launch shape, against the oracle
    and the two-kernel two-shot: 2, 4, 8 and 16 ranks, both dtypes, shards of 1 vector to several
    chunks with a partial last chunk, the persistent kernel (small direct-grid limit, grid caps), in
    place, with guard bands around every output."""
    with nuna.tunables(NUNA_TWO_SHOT_FORM=1, **cfg):
        for P in (2, 4, 8, 16):
            for dt in (np.uint16, np.float32):
                per_vec = 8 if dt == np.uint16 else 4
                for mv in (1, 7, 64, 65, 1000, 4097):
                    n = P * mv * per_vec
                    seed = 7919 * P + mv + (0 if dt == np.uint16 else 1)
                    x = wl.normal_bf16(P, n, seed) if dt == np.uint16 else wl.normal_f32(P, n, seed)
                    ref = oracle.allreduce(x)
                    for place in PLACES:
                        got = run_allreduce(nuna, x, "two_shot", place)
                        two = run_allreduce(nuna, x, "two_shot_two_kernels", place)
                        for d in range(P):
                            assert_bitwise(got[d], ref[d], f"{cfg} fused P={P} mv={mv} {place} rank {d}")
                            assert_bitwise(two[d], ref[d], f"{cfg} two kernels P={P} mv={mv} {place} rank {d}")
        x = wl.normal_bf16(8, 8 * 8 * 3000, 99)
        ref = oracle.allreduce(x)
        for cap in (1, 13, 100):
            nuna.set_max_workgroups(cap)
            try:
                got = run_allreduce(nuna, x, "two_shot", "xcd")
            finally:
                nuna.set_max_workgroups(0)
            for d in range(8):
                assert_bitwise(got[d], ref[d], f"{cfg} fused cap={cap} rank {d}")
        bufs = [to_dev(a) for a in x]
        nuna.allreduce(bufs, bufs, algo="two_shot", placement="xcd")
        torch.cuda.synchronize()
        for d in range(8):
            assert_bitwise(to_host(bufs[d]), ref[d], f"{cfg} fused in place rank {d}")


def _kernels(nuna, x, algo, place):
    ins = [to_dev(a) for a in x]
    outs = [torch.empty_like(t) for t in ins]
    nuna.allreduce(ins, outs, algo=algo, placement=place)
    rec = nuna.last_launch()
    torch.cuda.synchronize()
    return rec


def test_launch_record_names_what_ran(nuna):
    """nuna_last_launch: the two-shot's form by size and its tunable, the page-grouped map in XCD mode,
    the destination-split groups, the per-XCD lists of the dispatch."""
    x16 = wl.normal_bf16(8, 1024 * 8192, 3)  # 16 MiB per rank
    assert _kernels(nuna, x16, "two_shot", "xcd")["kernels"] == "k_reduce_scatter_direct+k_all_gather_direct"
    with nuna.tunables(NUNA_TWO_SHOT_FORM=1):
        assert _kernels(nuna, x16, "two_shot", "xcd")["kernels"] == "k_two_shot_direct"
    # AUTO: the two-shot for 8 ranks of bf16 from 16 MiB per rank, the one-shot below
    assert _kernels(nuna, x16, "auto", "xcd")["kernels"] == "k_reduce_scatter_direct+k_all_gather_direct"
    x4 = wl.ar_bf16_prefill(256)
    assert _kernels(nuna, x4, "auto", "xcd")["kernels"] == "k_allreduce_direct"
    r = _kernels(nuna, x4, "two_shot", "xcd")
    assert r["kernels"] == "k_two_shot_direct" and r["launches"] == 1 and r["map"] == "linear"
    with nuna.tunables(NUNA_TWO_SHOT_FORM=2):
        assert _kernels(nuna, x4, "two_shot", "xcd")["launches"] == 2
    d1 = wl.ar_bf16_decode(1)
    with nuna.tunables(NUNA_PAGE_GROUPS=1):
        r = _kernels(nuna, d1, "one_shot", "xcd")
        assert r["map"] == "xcd_pages" and r["group_size"] == 4 and r["grid"] % 32 == 0, r
        assert _kernels(nuna, d1, "one_shot", "linear")["map"] == "linear"
    assert _kernels(nuna, d1, "one_shot", "xcd")["map"] == "linear"
    r = _kernels(nuna, wl.ar_bf16_decode(64), "one_shot_split", "xcd")
    assert r["map"] == "xcd_groups" and r["group_size"] == 8, r
    x16 = wl.normal_bf16(16, 1 << 16, 9)
    assert _kernels(nuna, x16, "two_shot", "xcd")["map"] == "xcd_shards"
    assert _kernels(nuna, x16, "two_shot", "linear")["map"] == "linear"
    assert _kernels(nuna, x4, "two_shot", "xcd")["map"] == "linear"
    with nuna.tunables(NUNA_SHARD_XCD=2):
        assert _kernels(nuna, x4, "two_shot", "linear")["map"] == "xcd_shards"


@pytest.mark.parametrize("pg", [0, 1])
def test_page_groups_parity(nuna, pg):
    """XCD mode with the chunks of each 4 KiB page on one XCD (and without): the decode and 64-rank
    workloads, the fp32 integer workload, ragged sizes whose page-grouped grids end in padding
    workgroups, forced chunk sizes of 1-2 KiB (one-shot) and 256 B-1 KiB (tile), guard bands."""
    cases = [(wl.ar_f32_int(), "f32 int")] + [(wl.ar_bf16_decode(T), f"decode T={T}") for T in wl.DECODE_TOKENS]
    cases += [(wl.ar_bf16_p64(k), f"P=64 {k} KiB") for k in wl.P64_KIB]
    cases += [(wl.normal_bf16(P, n, 5 * P + n), f"P={P} n={n}") for P, n in ((8, 8 * 1000 + 3), (2, 4097), (16, 70001),
                                                                              (64, 3000), (24, 9001))]
    with nuna.tunables(NUNA_PAGE_GROUPS=pg):
        for x, what in cases:
            ref = oracle.allreduce(x)
            for algo in ("one_shot", "two_shot"):
                got = run_allreduce(nuna, x, algo, "xcd")
                for d in range(len(x)):
                    assert_bitwise(got[d], ref[d], f"page groups {pg} {algo} {what} rank {d}")
        for cfg in (dict(NUNA_WG_THREADS=64, NUNA_VPT=2), dict(NUNA_WG_THREADS=128, NUNA_VPT=1),
                    dict(NUNA_TILE_V=32), dict(NUNA_TILE_V=64)):
            with nuna.tunables(**cfg):
                for x, what in cases[1:3] + cases[5:7] + cases[-3:]:
                    ref = oracle.allreduce(x)
                    got = run_allreduce(nuna, x, "one_shot", "xcd")
                    for d in range(len(x)):
                        assert_bitwise(got[d], ref[d], f"page groups {pg} {cfg} {what} rank {d}")


def test_vpt8_every_collective(nuna):
    """Eight vectors per thread exist for the all-reduce with 2, 4 or 8 ranks only; forced for every
    collective, the others fall back to 4 and every result keeps the oracle's bits."""
    with nuna.tunables(NUNA_VPT=8):
        for P, n, dt in ((2, 70001, np.uint16), (4, 4097, np.float32), (8, 2 ** 17 * 8 + 40, np.uint16),
                         (8, 100003, np.float32), (3, 7001, np.uint16), (16, 70001, np.uint16)):
            x = wl.normal_bf16(P, n, 17 * P + n) if dt == np.uint16 else wl.normal_f32(P, n, 17 * P + n)
            ref = oracle.allreduce(x)
            for algo in AR_ALGOS:
                got = run_allreduce(nuna, x, algo, "xcd")
                for d in range(P):
                    assert_bitwise(got[d], ref[d], f"VPT=8 {algo} P={P} n={n} rank {d}")
            bufs = [to_dev(a) for a in x]
            nuna.allreduce(bufs, bufs, algo="one_shot", placement="linear")
            torch.cuda.synchronize()
            for d in range(P):
                assert_bitwise(to_host(bufs[d]), ref[d], f"VPT=8 in place P={P} n={n} rank {d}")
            m = n // P
            xs = [a[:P * m].copy() for a in x]
            rs = nuna.reduce_scatter([to_dev(a) for a in xs], placement="xcd")
            torch.cuda.synchronize()
            for r, want in enumerate(oracle.reduce_scatter(xs)):
                assert_bitwise(to_host(rs[r]), want, f"VPT=8 RS P={P} rank {r}")
            ag_in = [a[:m].copy() for a in x]
            ag = nuna.all_gather([to_dev(a) for a in ag_in], placement="xcd")
            torch.cuda.synchronize()
            for d, want in enumerate(oracle.all_gather(ag_in)):
                assert_bitwise(to_host(ag[d]), want, f"VPT=8 AG P={P} rank {d}")


def test_ar_eight_vector_rule_ragged(nuna):
    """8 ranks at about 15 MiB per rank: the default shape is 8 vectors per thread (its last round
    of workgroups is over 90 % full); the size ends in a partial chunk and a scalar tail."""
    n = 15 * (1 << 19) + 8 * 3 + 5
    x = wl.normal_bf16(8, n, 4242)
    ref = oracle.allreduce(x)
    for place in PLACES:
        got = run_allreduce(nuna, x, "one_shot", place)
        for d in range(8):
            assert_bitwise(got[d], ref[d], f"15 MiB ragged {place} rank {d}")


# ---------------------------------------------------------------- MoE combine (result collection)



@pytest.mark.parametrize("place", PLACES)
def test_combine_moe_full(nuna, place):
    _, topk = wl.a2a_moe()
    rows = oracle.a2a_counts(topk, wl.MOE_EXPERTS)
    y = wl.result_rows(rows, wl.HIDDEN_MOE, np.uint16, wl.seed_for(4, 7))
    ref = oracle.combine(y, topk, wl.MOE_EXPERTS)
    got = run_combine(nuna, y, topk, wl.MOE_EXPERTS, place)
    for s in range(8):
        assert_bitwise(got[s], ref[s], f"combine rank {s}")


@pytest.mark.parametrize("place", PLACES)
@pytest.mark.parametrize("P,T,k,E,H,dtype", [(2, 5, 2, 4, 24, np.float32), (3, 9, 2, 6, 10, np.uint16),
                                             (4, 33, 3, 16, 5, np.float32), (16, 32, 4, 64, 64, np.float32),
                                             (64, 16, 8, 256, 128, np.uint16), (64, 4, 64, 64, 256, np.float32),
                                             (8, 1, 8, 256, 7168, np.uint16), (8, 3, 8, 256, 7176, np.uint16),
                                             (1, 9, 1, 4, 256, np.float32), (8, 40, 8, 256, 1000, np.float32)])
def test_combine_small(nuna, P, T, k, E, H, dtype, place):
    topk = wl.moe_routing(P, T, k, E, 23 * P + T)
    y = wl.result_rows(oracle.a2a_counts(topk, E), H, dtype, 29 * P + T)
    ref = oracle.combine(y, topk, E)
    got = run_combine(nuna, y, topk, E, place)
    for s in range(P):
        assert_bitwise(got[s], ref[s], f"combine P={P} T={T} k={k} H={H} rank {s}")




@pytest.mark.parametrize("place", PLACES)
@pytest.mark.parametrize("P,T,k,E,H,dtype", [(8, 64, 4, 8, 7168, np.uint16), (8, 64, 4, 8, 7168, np.float32),
                                             (8, 40, 8, 256, 1000, np.float32), (3, 9, 2, 6, 10, np.uint16),
                                             (64, 4, 64, 64, 256, np.float32), (64, 16, 8, 256, 128, np.uint16)])
def test_combine_weighted(nuna, P, T, k, E, H, dtype, place):
    """Top-k weighted combine: each rank's result row scaled by its weight before the ascending sum."""
    topk = wl.moe_routing(P, T, k, E, 59 * P + T)
    y = wl.result_rows(oracle.a2a_counts(topk, E), H, dtype, 61 * P + T)
    w = gate_weights(topk, E, 67 * P + T)
    ref = oracle.combine(y, topk, E, w)
    got = run_combine(nuna, y, topk, E, place, weights=w)
    for s in range(P):
        assert_bitwise(got[s], ref[s], f"weighted combine P={P} T={T} k={k} E={E} H={H} rank {s}")


def test_combine_special_values(nuna):
    """inf, -inf, NaN payloads, signed zeros and denormals among the results."""
    P, T, k, E, H = 8, 24, 8, 64, 256
    topk = wl.moe_routing(P, T, k, E, 31)
    rows = oracle.a2a_counts(topk, E)
    for dtype in (np.uint16, np.float32):
        y = [wl.random_bits(1, int(r) * H, dtype, 37 + d)[0].reshape(int(r), H) for d, r in enumerate(rows)]
        ref = oracle.combine(y, topk, E)
        got = run_combine(nuna, y, topk, E, "xcd")
        for s in range(P):
            assert_bitwise_nan_aware(got[s], ref[s], f"combine specials {dtype.__name__} rank {s}")


def test_combine_inverts_dispatch(nuna):
    """With one expert per token, dispatch followed by combine returns every token row unchanged."""
    P, T, E, H = 8, 64, 64, wl.HIDDEN_MOE
    topk = wl.moe_routing(P, T, 1, E, 41)
    send = wl.moe_rows(P, T, H, 43)
    lay = nuna.A2ALayout(topk, E).upload()
    cap = int(lay.recv_rows().max())
    sd = [to_dev(a) for a in send]
    recv = [torch.empty((cap, H), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    back = [torch.empty((T, H), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    nuna.all_to_all(sd, recv, lay, placement="xcd")
    nuna.all_to_all_combine(recv, back, lay, placement="xcd")
    torch.cuda.synchronize()
    for s in range(P):
        assert_bitwise(to_host(back[s]), send[s], f"round trip rank {s}")
    lay.close()


@pytest.mark.parametrize("cap", [1, 5, 13])
def test_combine_persistent_loop(nuna, cap):
    """Fewer workgroups than work items: every workgroup loops over its items."""
    P, T, k, E, H = 8, 20, 8, 256, 1024
    topk = wl.moe_routing(P, T, k, E, 47)
    y = wl.result_rows(oracle.a2a_counts(topk, E), H, np.uint16, 53)
    ref = oracle.combine(y, topk, E)
    nuna.set_max_workgroups(cap)
    try:
        for place in PLACES:
            got = run_combine(nuna, y, topk, E, place)
            for s in range(P):
                assert_bitwise(got[s], ref[s], f"combine cap={cap} {place} rank {s}")
    finally:
        nuna.set_max_workgroups(0)


@pytest.mark.parametrize("P,T,k,E,H,dtype,weighted,cfg", [
    (8, 520, 2, 16, 4608, np.uint16, False, {}),  # 4160 tokens: 1 chunk by size, 576 vectors, raised to 2
    (8, 16, 8, 256, 7168, np.uint16, True, {}),
    (4, 8, 3, 16, 65536, np.uint16, False, {}),  # 8192-vector rows, 32 chunks by size
    (8, 24, 8, 64, 4096, np.float32, True, {"NUNA_COMBINE_CHUNKS": 1}),  # forced 1 chunk of 1024 vectors, raised
    (8, 40, 8, 256, 1000, np.float32, False, {"NUNA_WG_THREADS": 64, "NUNA_COMBINE_VPT": 1}),  # raised 2 -> 4
    (2, 7, 2, 4, 2056, np.uint16, True, {"NUNA_COMBINE_VPT": 4, "NUNA_COMBINE_CHUNKS": 5}),
    (1, 9, 1, 4, 256, np.float32, False, {}),
])
def test_combine_records_match_lists(nuna, P, T, k, E, H, dtype, weighted, cfg):
    """Per-token records (up to 8 ranks) and the offset lists both give the oracle's bits, also where the
    record kernel raises the chunk count so that a column chunk fits one pass of the workgroup."""
    topk = wl.moe_routing(P, T, k, E, 71 * P + T)
    y = wl.result_rows(oracle.a2a_counts(topk, E), H, dtype, 73 * P + T)
    w = gate_weights(topk, E, 79 * P + T) if weighted else None
    ref = oracle.combine(y, topk, E, w)
    for lists in (0, 1):
        with nuna.tunables(NUNA_COMBINE_LISTS=lists, **cfg):
            for place in PLACES:
                got = run_combine(nuna, y, topk, E, place, weights=w)
                for s in range(P):
                    assert_bitwise(got[s], ref[s], f"combine lists={lists} {cfg} {place} P={P} T={T} H={H} rank {s}")


# ---------------------------------------------------------------- graph capture and replay

def test_graph_replay_matches_eager(nuna):
    """Calls captured into a HIP graph and replayed several times, with eager work between replays."""
    x = wl.ar_bf16_decode(4)
    ref = oracle.allreduce(x)
    ins = [to_dev(a) for a in x]
    outs = [torch.empty_like(t) for t in ins]
    x2 = wl.ar_bf16_decode(16)
    ref2 = oracle.allreduce(x2)
    ins2 = [to_dev(a) for a in x2]
    outs2 = [torch.empty_like(t) for t in ins2]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        nuna.allreduce(ins, outs, algo="one_shot_split", placement="xcd")  # warm-up outside capture
        nuna.allreduce(ins2, outs2, algo="two_shot", placement="linear")
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        nuna.allreduce(ins, outs, algo="one_shot_split", placement="xcd")
        nuna.allreduce(ins2, outs2, algo="two_shot", placement="linear")
        nuna.allreduce(ins, outs, algo="one_shot", placement="linear")
    for rep in range(4):
        for o in outs + outs2:
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for d in range(8):
            assert_bitwise(to_host(outs[d]), ref[d], f"replay {rep} rank {d}")
            assert_bitwise(to_host(outs2[d]), ref2[d], f"replay {rep} rank {d} (two-shot)")


def test_all_gather_beside_gemm(nuna):
    """Collectives on one stream while a library GEMM runs on another: results stay bit-exact."""
    P, m = 8, 65536
    x = wl.normal_bf16(P, m, 71)
    ref = oracle.all_gather(x)
    ins = [to_dev(a) for a in x]
    outs = {p: [torch.empty(P * m, dtype=torch.bfloat16, device="cuda") for _ in range(P)] for p in PLACES}
    a = torch.randn(2560, 8192, dtype=torch.bfloat16, device="cuda")
    b = torch.randn(8192, 2560, dtype=torch.bfloat16, device="cuda")
    s_gemm, s_coll = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s_gemm):
        for _ in range(8):
            c = torch.matmul(a, b)
    with torch.cuda.stream(s_coll):
        for _ in range(50):
            for p in PLACES:
                nuna.all_gather(ins, outs[p], placement=p)
    torch.cuda.synchronize()
    assert torch.isfinite(c.float()).all()
    for p in PLACES:
        for d in range(P):
            assert_bitwise(to_host(outs[p][d]), ref[d], f"AG beside GEMM {p} rank {d}")


def test_split_allreduce_beside_gemm(nuna):
    """The destination-split all-reduce (the map the placement changes) beside a GEMM on another stream."""
    x = wl.ar_bf16_decode(64, seed=72)
    ref = oracle.allreduce(x)
    ins = [to_dev(a) for a in x]
    outs = {p: [torch.empty_like(t) for t in ins] for p in PLACES}
    a = torch.randn(2560, 8192, dtype=torch.bfloat16, device="cuda")
    b = torch.randn(8192, 2560, dtype=torch.bfloat16, device="cuda")
    s_gemm, s_coll = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s_gemm):
        for _ in range(8):
            c = torch.matmul(a, b)
    with torch.cuda.stream(s_coll):
        for _ in range(20):
            for p in PLACES:
                nuna.allreduce(ins, outs[p], algo="one_shot_split", placement=p)
    torch.cuda.synchronize()
    assert torch.isfinite(c.float()).all()
    for p in PLACES:
        for d in range(8):
            assert_bitwise(to_host(outs[p][d]), ref[d], f"split AR beside GEMM {p} rank {d}")



def test_dispatch_beside_gemm(nuna):
    """The MoE dispatch (the copies of a token row are one group under XCD placement) beside a GEMM on
    another stream, 128 tokens x 7168 per rank: every received row bit-exact, no write past a rank's rows."""
    T = 128
    send_np, topk = wl.a2a_moe(T=T)
    E = wl.MOE_EXPERTS
    ref = oracle.all_to_all(send_np, topk, E)
    rows = [r.shape[0] for r in ref]
    cap, H = max(rows) + 2, wl.HIDDEN_MOE
    send = [to_dev(a) for a in send_np]
    lay = nuna.A2ALayout(topk, E).upload()
    recv = {p: [torch.zeros((cap, H), dtype=torch.bfloat16, device="cuda") for _ in range(8)] for p in PLACES}
    a = torch.randn(2560, 8192, dtype=torch.bfloat16, device="cuda")
    b = torch.randn(8192, 2560, dtype=torch.bfloat16, device="cuda")
    s_gemm, s_coll = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s_gemm):
        for _ in range(8):
            c = torch.matmul(a, b)
    with torch.cuda.stream(s_coll):
        for _ in range(20):
            for p in PLACES:
                nuna.all_to_all(send, recv[p], lay, placement=p)
    torch.cuda.synchronize()
    lay.close()
    assert torch.isfinite(c.float()).all()
    for p in PLACES:
        for d in range(8):
            got = to_host(recv[p][d])
            assert_bitwise(got[:rows[d]], ref[d], f"dispatch beside GEMM {p} rank {d}")
            assert not got[rows[d]:].any(), f"dispatch beside GEMM {p} rank {d}: write past its rows"

def test_prepared_allreduce_repeats_the_call(nuna):
    """A prepared call gives the oracle's bits every time it runs, on the current stream or a given one."""
    x = wl.ar_bf16_decode(16)
    ref = oracle.allreduce(x)
    ins = [to_dev(a) for a in x]
    outs = [torch.empty_like(t) for t in ins]
    call = nuna.prepare_allreduce(ins, outs, algo="one_shot", placement="xcd")
    s = torch.cuda.Stream()
    for k in range(3):
        for o in outs:
            o.zero_()
        torch.cuda.synchronize()
        if k == 0:
            call()
        elif k == 1:
            call(s)
        else:
            call(s.cuda_stream)
        torch.cuda.synchronize()
        for d in range(8):
            assert_bitwise(to_host(outs[d]), ref[d], f"prepared call {k} rank {d}")


def test_graph_replay_moe_and_collectives(nuna):
    """Dispatch, weighted combine, reduce-scatter and all-gather captured in one HIP graph and replayed
    several times with eager work in between; every replay matches the oracle."""
    P, T, k, E, H = 8, 32, 8, 256, 1024
    topk = wl.moe_routing(P, T, k, E, 77)
    send_np = wl.moe_rows(P, T, H, 78)
    lay = nuna.A2ALayout(topk, E).upload()
    cap = int(lay.recv_rows().max())
    send = [to_dev(a) for a in send_np]
    recv = [torch.empty((cap, H), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    back = [torch.empty((T, H), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    w_np = np.random.default_rng(79).random((P, T, P)).astype(np.float32)
    w = to_dev(w_np)
    x = wl.normal_bf16(P, P * 4096, 80)
    ins = [to_dev(a) for a in x]
    shards = [torch.empty(4096, dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    gathered = [torch.empty(P * 4096, dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    ref_recv = oracle.all_to_all(send_np, topk, E)
    ref_back = oracle.combine(ref_recv, topk, E, w_np)
    ref_rs = oracle.reduce_scatter(x)
    ref_ag = oracle.all_gather(ref_rs)

    def work():
        nuna.all_to_all(send, recv, lay, placement="xcd")
        nuna.all_to_all_combine(recv, back, lay, placement="xcd", weights=w)
        nuna.reduce_scatter(ins, shards, placement="xcd")
        nuna.all_gather(shards, gathered, placement="xcd")

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        work()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    rows = lay.recv_rows()
    for rep in range(3):
        for t in recv + back + shards + gathered:
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for d in range(P):
            assert_bitwise(to_host(recv[d][:int(rows[d])]), ref_recv[d], f"replay {rep} dispatch rank {d}")
            assert_bitwise(to_host(back[d]), ref_back[d], f"replay {rep} combine rank {d}")
            assert_bitwise(to_host(shards[d]), ref_rs[d], f"replay {rep} reduce-scatter rank {d}")
            assert_bitwise(to_host(gathered[d]), ref_ag[d], f"replay {rep} all-gather rank {d}")
    lay.close()


def test_copy_kernel(nuna):
    for nbytes in (16, 4096, 1000003, 64 << 20):
        src = torch.randint(-2 ** 31, 2 ** 31 - 1, ((nbytes + 3) // 4,), dtype=torch.int32, device="cuda")
        srcb = src.view(torch.uint8)[:nbytes]
        dst = torch.zeros(nbytes + 64, dtype=torch.uint8, device="cuda")
        nuna.lib().nuna_copy(dst.data_ptr(), srcb.data_ptr(), nbytes, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        assert torch.equal(dst[:nbytes], srcb)
        assert int(dst[nbytes:].abs().sum()) == 0


@pytest.mark.parametrize("n", [1, 2, 4, 8, 16])
def test_ref_streams(nuna, n):
    """Reference read / write / copy streams over n buffers: the read's per-item XOR checksums, the write
    pattern and the copies, at one partial item, one item, and many items with a partial last one, with
    guard bands after every written range."""
    for nbytes in (16, 4096, 4096 * 5 + 48, (1 << 20) + 4096):
        words = nbytes // 4
        nv = nbytes // 16
        blocks = 1 if n >= 8 else 8 // n                # 4 KiB blocks per read item
        items = (nbytes + blocks * 4096 - 1) // (blocks * 4096)
        assert nuna.ref_read_checksum_bytes(n, nbytes) == items * 16
        srcs = [torch.randint(-2 ** 31, 2 ** 31 - 1, (words,), dtype=torch.int32, device="cuda") for _ in range(n)]
        host = np.stack([s.cpu().numpy().view(np.uint32).reshape(nv, 4) for s in srcs])
        # read: one checksum per item, the XOR of the item's vectors of all buffers
        sink = torch.zeros(items * 4 + 16, dtype=torch.int32, device="cuda")
        nuna.ref_stream("read", srcs, [sink[:items * 4]])
        rec = nuna.last_launch()
        assert rec["kernels"] == "k_ref_read" and rec["grid"] == items and rec["vectors_per_thread"] == blocks
        torch.cuda.synchronize()
        padded = np.zeros((n, items * blocks * 256, 4), dtype=np.uint32)
        padded[:, :nv] = host
        per_item = padded.reshape(n, items, blocks * 256, 4)
        want = np.bitwise_xor.reduce(np.bitwise_xor.reduce(per_item, axis=2), axis=0)
        got = sink.cpu().numpy().view(np.uint32)
        assert np.array_equal(got[:items * 4].reshape(items, 4), want), f"read n={n} bytes={nbytes}"
        assert not got[items * 4:].any(), f"read n={n} bytes={nbytes}: write past the checksums"
        # write: vector v of buffer r = {v mod 2^32, v div 2^32, r, 0x52454631}
        outs = [torch.full((words + 16,), -1, dtype=torch.int32, device="cuda") for _ in range(n)]
        nuna.ref_stream("write", None, [o[:words] for o in outs])
        torch.cuda.synchronize()
        v = np.arange(nv, dtype=np.uint64)
        for r in range(n):
            g = outs[r].cpu().numpy().view(np.uint32)
            w = np.stack([(v & 0xFFFFFFFF).astype(np.uint32), (v >> 32).astype(np.uint32),
                          np.full(nv, r, dtype=np.uint32), np.full(nv, 0x52454631, dtype=np.uint32)], axis=1)
            assert np.array_equal(g[:words].reshape(nv, 4), w), f"write n={n} bytes={nbytes} buffer {r}"
            assert np.all(g[words:] == 0xFFFFFFFF), f"write n={n} bytes={nbytes} buffer {r}: past the end"
        # copy
        outs = [torch.full((words + 16,), -1, dtype=torch.int32, device="cuda") for _ in range(n)]
        nuna.ref_stream("copy", srcs, [o[:words] for o in outs])
        torch.cuda.synchronize()
        for r in range(n):
            g = outs[r].cpu().numpy().view(np.uint32)
            assert np.array_equal(g[:words].reshape(nv, 4), host[r]), f"copy n={n} bytes={nbytes} buffer {r}"
            assert np.all(g[words:] == 0xFFFFFFFF), f"copy n={n} bytes={nbytes} buffer {r}: past the end"


def test_concurrent_host_threads(nuna):
    """Four host threads, each on its own stream, issue all-reduces, reduce-scatters, all-gathers,
    dispatches and combines at the same time (one layout shared by all); every result keeps the
    oracle's bits."""
    import threading
    P, T, k, E, H = 8, 64, 4, 32, 256
    topk = wl.moe_routing(P, T, k, E, 55)
    lay = nuna.A2ALayout(topk, E).upload()
    rows = lay.recv_rows()
    send = wl.normal_bf16(P, T * H, 56)
    send = [a.reshape(T, H) for a in send]
    want_recv = oracle.all_to_all(send, topk, E)
    want_comb = oracle.combine(want_recv, topk, E)
    errors = []
    barrier = threading.Barrier(4)

    def worker(w):
        try:
            s = torch.cuda.Stream()
            x = wl.normal_bf16(P, 4096 * (w + 1) + 8 * w, 60 + w)
            m = x[0].size // P
            ref_ar = oracle.allreduce(x)
            ref_rs = oracle.reduce_scatter([a[:P * m].copy() for a in x])
            ref_ag = oracle.all_gather([a[:m].copy() for a in x])
            with torch.cuda.stream(s):
                ins = [to_dev(a) for a in x]
                rs_in = [t[:P * m] for t in ins]
                ag_in = [t[:m] for t in ins]
                snd = [to_dev(a) for a in send]
                cap = int(rows.max())
                rcv = [torch.empty((cap, H), dtype=torch.bfloat16, device="cuda") for d in range(P)]
                out = [torch.empty((T, H), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
                s.synchronize()
                barrier.wait()
                for it in range(10):
                    place = PLACES[(w + it) % 2]
                    ar = [torch.empty_like(t) for t in ins]
                    nuna.allreduce(ins, ar, algo=AR_ALGOS[it % len(AR_ALGOS)], placement=place)
                    rs = nuna.reduce_scatter(rs_in, placement=place)
                    ag = nuna.all_gather(ag_in, placement=place)
                    nuna.all_to_all(snd, rcv, lay, placement=place)
                    nuna.all_to_all_combine(rcv, out, lay, placement=place)
                s.synchronize()
            for d in range(P):
                assert_bitwise(to_host(ar[d]), ref_ar[d], f"thread {w} AR rank {d}")
                assert_bitwise(to_host(rs[d]), ref_rs[d], f"thread {w} RS rank {d}")
                assert_bitwise(to_host(ag[d]), ref_ag[d], f"thread {w} AG rank {d}")
                assert_bitwise(to_host(rcv[d][:int(rows[d])]).reshape(-1), want_recv[d].reshape(-1),
                               f"thread {w} A2A rank {d}")
                assert_bitwise(to_host(out[d]).reshape(-1), want_comb[d].reshape(-1), f"thread {w} combine rank {d}")
        except Exception as e:  # reported by the main thread
            errors.append(f"thread {w}: {e!r}")

    threads = [threading.Thread(target=worker, args=(w,)) for w in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    lay.close()
    assert not errors, errors
