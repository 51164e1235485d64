"""C-ABI tests that need no GPU: exports, argument validation, host planning.

Argument checks in libnuna run before any HIP call, so invalid calls are
rejected here exactly as on a GPU machine.  Tests that pass made-up device
pointers skip themselves when a GPU is visible, so no kernel is ever launched
on addresses that do not exist.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2608_00867_amd import nuna
from paper_2608_00867_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nuna.h")


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


no_gpu_only = pytest.mark.skipif(_gpu_visible(), reason="uses made-up device pointers; CPU-only")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nuna_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_expected_entry_points():
    decl = _declared_functions()
    for name in ("nuna_allreduce", "nuna_reduce_scatter", "nuna_all_gather", "nuna_all_to_all",
                 "nuna_a2a_layout_create", "nuna_init", "nuna_last_error_string"):
        assert name in decl


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(nuna.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_binding_covers_every_declared_symbol():
    assert sorted(nuna.SIGNATURES) == _declared_functions()


# ---------------------------------------------------------------- validation with made-up pointers

BASE = 0x7F0000000000  # never dereferenced: every case below fails validation, or there is no device


def _bufs(P, stride=1 << 20, base=BASE):
    return [base + r * stride for r in range(P)]


@no_gpu_only
@pytest.mark.parametrize("case,expect", [
    ("null_in", nuna.ERR_INVALID_ARG),
    ("null_out", nuna.ERR_INVALID_ARG),
    ("null_elem", nuna.ERR_INVALID_ARG),
    ("P0", nuna.ERR_INVALID_ARG),
    ("P65", nuna.ERR_INVALID_ARG),
    ("bad_dtype", nuna.ERR_UNSUPPORTED),
    ("bad_place", nuna.ERR_INVALID_ARG),
    ("bad_algo", nuna.ERR_INVALID_ARG),
    ("misaligned_in", nuna.ERR_MISALIGNED),
    ("misaligned_out", nuna.ERR_MISALIGNED),
    ("huge_count", nuna.ERR_INVALID_ARG),
    ("outs_overlap", nuna.ERR_OVERLAP),
    ("in_is_other_ranks_out", nuna.ERR_OVERLAP),
    ("in_partially_overlaps_out", nuna.ERR_OVERLAP),
])
def test_allreduce_rejects(case, expect):
    P, n = 8, 4096
    ins, outs = _bufs(P), _bufs(P, base=BASE + (1 << 32))
    dtype, place, algo = nuna.BF16, nuna.XCD, nuna.ALGO_AUTO
    if case == "null_in":
        ins = None
    elif case == "null_out":
        outs = None
    elif case == "null_elem":
        ins[3] = None
    elif case == "P0":
        P = 0
    elif case == "P65":
        P = 65
        ins, outs = _bufs(P), _bufs(P, base=BASE + (1 << 32))
    elif case == "bad_dtype":
        dtype = 7
    elif case == "bad_place":
        place = 2
    elif case == "bad_algo":
        algo = 9
    elif case == "misaligned_in":
        ins[2] += 8
    elif case == "misaligned_out":
        outs[5] += 2
    elif case == "huge_count":
        n = 1 << 62
    elif case == "outs_overlap":
        outs[1] = outs[0] + 16
    elif case == "in_is_other_ranks_out":
        ins[2] = outs[3]
    elif case == "in_partially_overlaps_out":
        ins[4] = outs[4] + 16
    st = nuna.allreduce_raw(ins, outs, P, n, dtype, algo, place)
    assert st == expect, (st, nuna.last_error())
    assert nuna.last_error()


@no_gpu_only
def test_zero_count_is_a_noop_without_hip():
    assert nuna.allreduce_raw(_bufs(8), _bufs(8, base=BASE + (1 << 32)), 8, 0, nuna.BF16) == nuna.OK
    assert nuna.reduce_scatter_raw(_bufs(8), _bufs(8, base=BASE + (1 << 32)), 8, 0, nuna.BF16) == nuna.OK
    assert nuna.all_gather_raw(_bufs(8), _bufs(8, base=BASE + (1 << 32)), 8, 0, nuna.BF16) == nuna.OK


@no_gpu_only
def test_valid_call_without_device_reports_hip_error():
    """Validation passes, then the launch fails loudly: there is no host fallback."""
    st = nuna.allreduce_raw(_bufs(8), _bufs(8, base=BASE + (1 << 32)), 8, 4096, nuna.BF16)
    assert st == nuna.ERR_HIP, nuna.last_error()
    assert "HIP" in nuna.last_error()


@no_gpu_only
def test_in_place_forms_pass_validation():
    P, m = 8, 4096
    es = 2
    outs = _bufs(P, stride=1 << 24)
    # all-reduce in place
    assert nuna.allreduce_raw(outs, outs, P, P * m, nuna.BF16) == nuna.ERR_HIP
    # dest-split in place silently becomes one-shot; validation still passes
    assert nuna.allreduce_raw(outs, outs, P, P * m, nuna.BF16, nuna.ALGO_ONE_SHOT_SPLIT) == nuna.ERR_HIP
    # reduce-scatter: out[r] = in[r] + r*m elements
    rs_out = [outs[r] + r * m * es for r in range(P)]
    assert nuna.reduce_scatter_raw(outs, rs_out, P, m, nuna.BF16) == nuna.ERR_HIP
    # all-gather: in[r] = out[r] + r*m elements
    ag_in = [outs[r] + r * m * es for r in range(P)]
    assert nuna.all_gather_raw(ag_in, outs, P, m, nuna.BF16) == nuna.ERR_HIP
    # wrong in-place offsets are overlaps
    bad = [outs[r] + ((r + 1) % P) * m * es for r in range(P)]
    assert nuna.reduce_scatter_raw(outs, bad, P, m, nuna.BF16) == nuna.ERR_OVERLAP
    assert nuna.all_gather_raw(bad, outs, P, m, nuna.BF16) == nuna.ERR_OVERLAP


@no_gpu_only
def test_copy_and_probe_validation():
    L = nuna.lib()
    assert L.nuna_copy(BASE, BASE + 8, 64, None) == nuna.ERR_MISALIGNED
    assert L.nuna_copy(BASE, BASE + 16, 64, None) == nuna.ERR_OVERLAP
    assert L.nuna_copy(None, BASE, 64, None) == nuna.ERR_INVALID_ARG
    assert L.nuna_copy(BASE, BASE + 4096, 0, None) == nuna.OK
    assert L.nuna_probe_xcc(0, BASE, None, None) == nuna.ERR_INVALID_ARG
    assert L.nuna_probe_xcc(8, None, None, None) == nuna.ERR_INVALID_ARG


def test_flat_buffer_wrappers_refuse_views_and_host_tensors():
    """copy(), ref_stream() and the latency probes take a data pointer and numel() * element_size() bytes,
    so they accept only contiguous CUDA tensors: a host tensor or an expanded view (whose byte span exceeds
    its storage) is refused before any library call, as are an unknown kind and empty buffer lists."""
    import torch
    a, b = torch.zeros(64), torch.zeros(64)
    with pytest.raises(ValueError, match="contiguous CUDA"):
        nuna.copy(b, a)
    with pytest.raises(ValueError, match="contiguous CUDA"):
        nuna.copy(b, torch.zeros(1).expand(64))
    with pytest.raises(ValueError, match="contiguous CUDA"):
        nuna.ref_stream("copy", [a], [b])
    with pytest.raises(ValueError, match="contiguous CUDA"):
        nuna.ref_stream("write", None, [torch.zeros(8, 8).t()])
    with pytest.raises(ValueError, match="kind"):
        nuna.ref_stream("move", [a], [b])
    with pytest.raises(ValueError, match="at least one destination"):
        nuna.ref_stream("read", [a], [])
    with pytest.raises(ValueError, match="at least one destination"):
        nuna.ref_stream("write", None, [])
    with pytest.raises(ValueError, match="contiguous CUDA"):
        nuna.probe_load_latency(torch.zeros(1 << 12), 8192, 256, 0)
    with pytest.raises(ValueError, match="contiguous CUDA"):
        nuna.probe_load_latency_cus(torch.zeros(1 << 12), 0)


@no_gpu_only
def test_ref_stream_validation():
    """nuna_ref_stream refuses bad kinds, buffer counts, sizes, NULL, misaligned and overlapping buffers
    before any launch; zero bytes is a no-op."""
    MiB = 1 << 20
    src = [BASE + r * 4 * MiB for r in range(8)]
    dst = [BASE + (8 + r) * 4 * MiB for r in range(8)]
    raw = nuna.ref_stream_raw
    L = nuna.lib()
    assert L.nuna_ref_stream(3, nuna._ptr_array(src), nuna._ptr_array(dst), 1, 4096, None) == nuna.ERR_INVALID_ARG
    assert L.nuna_ref_stream(-1, nuna._ptr_array(src), nuna._ptr_array(dst), 1, 4096, None) == nuna.ERR_INVALID_ARG
    for n in (0, 3, 5, 32):
        assert raw("copy", src[:1] * max(n, 1), dst[:1] * max(n, 1), n, 4096) == nuna.ERR_INVALID_ARG
    assert raw("copy", src, dst, 8, 4095 * 4) == nuna.ERR_INVALID_ARG      # not a multiple of 16
    assert raw("copy", src, dst, 8, (1 << 34) + 16) == nuna.ERR_INVALID_ARG
    assert raw("read", None, dst, 8, 4096) == nuna.ERR_INVALID_ARG
    assert raw("copy", src, None, 8, 4096) == nuna.ERR_INVALID_ARG
    assert raw("copy", src[:7] + [None], dst, 8, 4096) == nuna.ERR_INVALID_ARG
    assert raw("write", None, dst[:3] + [None] + dst[4:], 8, 4096) == nuna.ERR_INVALID_ARG
    assert raw("copy", src[:7] + [src[7] + 8], dst, 8, 4096) == nuna.ERR_MISALIGNED
    assert raw("read", src, [dst[0] + 4], 8, 4096) == nuna.ERR_MISALIGNED
    # overlaps: a copy destination on a source, two write destinations, the read checksums on a source
    assert raw("copy", src, dst[:7] + [src[3] + 4096], 8, 8192) == nuna.ERR_OVERLAP
    assert raw("write", None, dst[:7] + [dst[6] + 4096], 8, 8192) == nuna.ERR_OVERLAP
    assert raw("read", src, [src[5] + 4 * MiB - 16], 8, 4 * MiB) == nuna.ERR_OVERLAP
    # a read's checksum range is ceil(bytes / item) * 16 bytes, item = max(1, 8 / n) * 4 KiB: 4 MiB + 16
    # bytes of 8 sources need 1025 checksums, so a range starting 1024 vectors below a source reaches
    # into it; with one source (32 KiB items) 129 checksums reach 16 bytes into it
    assert raw("read", src, [src[1] - 1024 * 16], 8, 4 * MiB + 16) == nuna.ERR_OVERLAP
    assert raw("read", src[1:2], [src[1] - 128 * 16], 1, 4 * MiB + 16) == nuna.ERR_OVERLAP
    assert nuna.ref_read_checksum_bytes(1, 4 * MiB + 16) == 129 * 16
    assert nuna.ref_read_checksum_bytes(8, 4 * MiB + 16) == 1025 * 16
    for kind in ("read", "write", "copy"):
        assert raw(kind, None if kind == "write" else src, dst, 8, 0) == nuna.OK
    assert nuna.last_launch()["launches"] == 0


def test_init_without_device_fails_cleanly():
    if _gpu_visible():
        pytest.skip("GPU visible")
    assert nuna.lib().nuna_init() == nuna.ERR_HIP


# ---------------------------------------------------------------- all-to-all planner (host, bit-exact)

@pytest.mark.parametrize("P,T,k,E,seed", [(1, 4, 1, 1, 1), (2, 5, 2, 4, 2), (3, 9, 2, 6, 3), (8, 64, 8, 256, 4),
                                          (8, 512, 8, 256, wl.seed_for(4)), (64, 16, 8, 256, 6), (4, 0, 2, 8, 7)])
def test_a2a_planner_matches_oracle(P, T, k, E, seed):
    topk = wl.moe_routing(P, T, k, E, seed)
    lay = nuna.A2ALayout(topk, E)
    rows = lay.recv_rows()
    assert np.array_equal(rows, oracle.a2a_counts(topk, E))
    for d in range(P):
        sr, st = lay.recv_map(d)
        osr, ost = oracle.a2a_map(topk, E, d)
        assert np.array_equal(sr, osr) and np.array_equal(st, ost), d
    lay.close()


@pytest.mark.parametrize("case", ["bad_expert", "negative_expert", "E_not_multiple", "topk0", "P0", "T_neg"])
def test_a2a_layout_rejects(case):
    P, T, k, E = 4, 3, 2, 8
    topk = np.zeros((P, T, k), dtype=np.int32)
    if case == "bad_expert":
        topk[1, 2, 1] = E
    elif case == "negative_expert":
        topk[0, 0, 0] = -1
    elif case == "E_not_multiple":
        E = 10
    elif case == "topk0":
        k = 0
    elif case == "P0":
        P = 0
    elif case == "T_neg":
        T = -1
    h = ctypes.c_void_p()
    st = nuna.lib().nuna_a2a_layout_create(P, T, k, E, topk.ctypes.data, ctypes.byref(h))
    assert st == nuna.ERR_INVALID_ARG, nuna.last_error()
    assert not h.value


def test_a2a_requires_upload_and_capacity():
    if _gpu_visible():
        pytest.skip("GPU visible")
    topk = wl.moe_routing(4, 8, 2, 8, 11)
    lay = nuna.A2ALayout(topk, 8)
    rows = lay.recv_rows()
    send = _bufs(4)
    recv = _bufs(4, base=BASE + (1 << 32))
    assert nuna.all_to_all_raw(send, recv, lay.handle, 64, int(rows.max()), nuna.BF16) == nuna.ERR_INVALID_ARG
    assert "upload" in nuna.last_error()
    assert nuna.all_to_all_raw(send, recv, lay.handle, 64, int(rows.max()) - 1, nuna.BF16) == nuna.ERR_INVALID_ARG
    assert "capacity" in nuna.last_error()
    recv[1] = send[2] + 16
    assert nuna.all_to_all_raw(send, recv, lay.handle, 64, int(rows.max()), nuna.BF16) == nuna.ERR_OVERLAP
    lay.close()


def test_combine_requires_upload_capacity_and_disjoint_buffers():
    if _gpu_visible():
        pytest.skip("GPU visible")
    topk = wl.moe_routing(4, 8, 2, 8, 12)
    lay = nuna.A2ALayout(topk, 8)
    rows = lay.recv_rows()
    y = _bufs(4)
    out = _bufs(4, base=BASE + (1 << 32))
    cap = int(rows.max())
    assert nuna.all_to_all_combine_raw(y, out, lay.handle, 64, cap, nuna.BF16) == nuna.ERR_INVALID_ARG
    assert "upload" in nuna.last_error()
    assert nuna.all_to_all_combine_raw(y, out, lay.handle, 64, cap - 1, nuna.BF16) == nuna.ERR_INVALID_ARG
    assert "capacity" in nuna.last_error()
    assert nuna.all_to_all_combine_raw(y, out, lay.handle, 0, cap, nuna.BF16) == nuna.ERR_INVALID_ARG
    assert nuna.all_to_all_combine_raw(y, out, lay.handle, 64, cap, 7) == nuna.ERR_UNSUPPORTED
    assert nuna.all_to_all_combine_raw(y, out, lay.handle, 64, cap, nuna.BF16, place=5) == nuna.ERR_INVALID_ARG
    bad = list(y)
    bad[2] = y[2] + 2
    assert nuna.all_to_all_combine_raw(bad, out, lay.handle, 64, cap, nuna.BF16) == nuna.ERR_MISALIGNED
    bad[2] = 0
    assert nuna.all_to_all_combine_raw(bad, out, lay.handle, 64, cap, nuna.BF16) == nuna.ERR_INVALID_ARG
    clash = list(out)
    clash[3] = y[1] + 16
    assert nuna.all_to_all_combine_raw(y, clash, lay.handle, 64, cap, nuna.BF16) == nuna.ERR_OVERLAP
    clash = list(out)
    clash[3] = out[0] + 16
    assert nuna.all_to_all_combine_raw(y, clash, lay.handle, 64, cap, nuna.BF16) == nuna.ERR_OVERLAP
    assert nuna.all_to_all_combine_raw(y, out, None, 64, cap, nuna.BF16) == nuna.ERR_INVALID_ARG
    w0 = BASE + (2 << 32)
    assert nuna.all_to_all_combine_raw(y, out, lay.handle, 64, cap, nuna.BF16, weights_ptr=w0 + 2) == \
        nuna.ERR_MISALIGNED
    assert "weights" in nuna.last_error()
    assert nuna.all_to_all_combine_raw(y, out, lay.handle, 64, cap, nuna.BF16, weights_ptr=out[2] + 64) == \
        nuna.ERR_OVERLAP
    assert nuna.all_to_all_combine_raw(y, out, lay.handle, 64, cap, nuna.BF16, weights_ptr=w0) == \
        nuna.ERR_INVALID_ARG  # valid weights: still not uploaded
    assert "upload" in nuna.last_error()
    lay.close()


def test_combine_on_empty_layout_is_a_noop():
    lay = nuna.A2ALayout(np.zeros((4, 0, 2), dtype=np.int32), 8)
    assert nuna.all_to_all_combine_raw(_bufs(4), _bufs(4, base=BASE + (1 << 32)), lay.handle, 64, 0,
                                       nuna.BF16) == nuna.OK
    lay.close()


def test_a2a_layout_rejects_more_than_int32_tokens():
    topk = np.zeros((1, 1, 1), dtype=np.int32)  # not read: the size check comes first
    h = ctypes.c_void_p()
    st = nuna.lib().nuna_a2a_layout_create(64, (1 << 31) // 64, 1, 64, topk.ctypes.data, ctypes.byref(h))
    assert st == nuna.ERR_INVALID_ARG and "exceeds" in nuna.last_error()
    assert not h.value


def test_tunables_set_get_restore_and_reject():
    names = ["NUNA_MAX_GRID", "NUNA_WG_THREADS", "NUNA_VPT", "NUNA_LPR_MIN_RANKS", "NUNA_LPR_MAX_VECTORS",
             "NUNA_COMBINE_VPT", "NUNA_COMBINE_CHUNKS", "NUNA_TILE_V", "NUNA_COMBINE_LISTS",
             "NUNA_WRITE_THROUGH"]
    before = {n: nuna.get_tunable(n) for n in names}
    with nuna.tunables(NUNA_TILE_V=32, NUNA_WG_THREADS=128, NUNA_LPR_MAX_VECTORS=1 << 33, NUNA_COMBINE_CHUNKS=3,
                       NUNA_VPT=8, NUNA_COMBINE_LISTS=1, NUNA_WRITE_THROUGH=2):
        assert nuna.get_tunable("NUNA_COMBINE_LISTS") == 1
        assert nuna.get_tunable("NUNA_WRITE_THROUGH") == 2
        assert nuna.get_tunable("NUNA_VPT") == 8
        assert nuna.get_tunable("NUNA_TILE_V") == 32
        assert nuna.get_tunable("NUNA_WG_THREADS") == 128
        assert nuna.get_tunable("NUNA_LPR_MAX_VECTORS") == 1 << 33
        assert nuna.get_tunable("NUNA_COMBINE_CHUNKS") == 3
    assert {n: nuna.get_tunable(n) for n in names} == before
    for name, bad in [("NUNA_TILE_V", 8), ("NUNA_VPT", 3), ("NUNA_WG_THREADS", 32), ("NUNA_LPR_MIN_RANKS", 0),
                      ("NUNA_MAX_GRID", -1), ("NUNA_COMBINE_VPT", 8), ("NUNA_COMBINE_LISTS", 2),
                      ("NUNA_WRITE_THROUGH", 3),
                      ("NUNA_NOT_A_KNOB", 1)]:
        with pytest.raises(nuna.NunaError):
            nuna.set_tunable(name, bad)
    assert {n: nuna.get_tunable(n) for n in names} == before
    assert nuna.lib().nuna_get_tunable(b"NUNA_VPT", None) == nuna.ERR_INVALID_ARG


def test_tunables_from_environment_are_validated():
    """The environment is read once per process (here a fresh one): accepted values apply, 64-bit values
    parse, values outside a knob's set are ignored."""
    import subprocess
    import sys
    env = dict(os.environ, NUNA_TILE_V="32", NUNA_LPR_MAX_VECTORS=str(1 << 33), NUNA_WG_THREADS="33",
               NUNA_VPT="banana")
    code = ("import sys; sys.path.insert(0, %r); from paper_2608_00867_amd import nuna; "
            "print(nuna.get_tunable('NUNA_TILE_V'), nuna.get_tunable('NUNA_LPR_MAX_VECTORS'), "
            "nuna.get_tunable('NUNA_WG_THREADS'), nuna.get_tunable('NUNA_VPT'))" % ROOT)
    out = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, check=True)
    assert out.stdout.split() == ["32", str(1 << 33), "0", "0"]


# ---------------------------------------------------------------- placement map (host mirror)

def _map(place, G, groups, gsize):
    """item -> (workgroup, position in that workgroup's sequence)"""
    seen = {}
    for b in range(G):
        for pos, w in enumerate(nuna.placement_items(place, b, G, groups, gsize)):
            assert w not in seen, (place, G, groups, gsize, w)
            seen[w] = (b, pos)
    return seen


GEOMS = [(1, 1), (5, 1), (8, 1), (13, 1), (64, 1), (3, 8), (8, 8), (11, 3), (100, 1), (16384, 1), (50, 2), (4, 8),
         (9, 7)]


@pytest.mark.parametrize("groups,gsize", GEOMS)
def test_placement_covers_every_item_once(groups, gsize):
    W = groups * gsize
    for place in (nuna.LINEAR, nuna.XCD):
        G0 = nuna.placement_grid(place, groups, gsize)
        for G in sorted({G0, max(1, G0 // 3), 1, 7, 8}):
            if G > 4096 and G != G0:
                continue
            seen = _map(place, G, groups, gsize)
            assert sorted(seen) == list(range(W)), (place, G)


@pytest.mark.parametrize("groups,gsize", [g for g in GEOMS if g[0] * g[1] <= 4096])
def test_xcd_mode_deals_groups_round_robin_and_runs_members_together(groups, gsize):
    G = nuna.placement_grid(nuna.XCD, groups, gsize)
    assert G >= groups * gsize and (gsize == 1 or G % 8 == 0)
    seen = _map(nuna.XCD, G, groups, gsize)
    for g in range(groups):
        bs = [seen[g * gsize + m][0] for m in range(gsize)]
        # group g lives on XCD g mod 8 (workgroup b runs on XCD b mod 8) ...
        assert {b % 8 for b in bs} == {g % 8}, g
        # ... one item per workgroup, members on consecutive workgroup slots of that XCD
        assert all(seen[g * gsize + m][1] == 0 for m in range(gsize))
        ks = [b // 8 for b in bs]
        assert ks == list(range(ks[0], ks[0] + gsize)), (g, ks)


def test_xcd_mode_with_single_item_groups_equals_linear():
    for W in (8, 64, 1000):
        G = nuna.placement_grid(nuna.XCD, W, 1)
        lin = _map(nuna.LINEAR, G, W, 1)
        xcd = _map(nuna.XCD, G, W, 1)
        assert lin == xcd


def test_linear_mode_is_round_robin_and_spreads_groups():
    seen = _map(nuna.LINEAR, 16, 40, 1)
    assert all(b == w % 16 for w, (b, _) in seen.items())
    seen = _map(nuna.LINEAR, 64, 8, 8)
    for g in range(8):
        assert len({seen[g * 8 + m][0] % 8 for m in range(8)}) == 8


def test_status_codes_match_header():
    """The binding's status constants are the header's enum values."""
    text = open(os.path.join(ROOT, "include", "nuna.h")).read()
    enum = dict((m.group(1), int(m.group(2))) for m in re.finditer(r"\b(NUNA_(?:OK|ERR_[A-Z_]+)) = (\d+)", text))
    assert enum == {v: k for k, v in nuna.STATUS_NAMES.items()}
    assert enum["NUNA_ERR_NO_MEMORY"] == nuna.ERR_NO_MEMORY


def test_host_allocation_failure_is_a_status():
    """Host tables that cannot be allocated give NUNA_ERR_NO_MEMORY: no exception leaves the C ABI and
    the call does not end the process.  A child process caps its own address space 16 MiB above its
    use, then asks for a routing layout whose host tables need about 64 MiB."""
    import subprocess
    import sys
    code = (
        "import ctypes, resource, sys\n"
        "import numpy as np\n"
        "sys.path.insert(0, %r)\n"
        "from paper_2608_00867_amd import nuna\n"
        "L = nuna.lib()\n"
        "P, T = 8, 1 << 20\n"
        "topk = np.zeros((P, T, 1), dtype=np.int32)\n"
        "vm = int(open('/proc/self/statm').read().split()[0]) * resource.getpagesize()\n"
        "resource.setrlimit(resource.RLIMIT_AS, (vm + (16 << 20), resource.RLIM_INFINITY))\n"
        "h = ctypes.c_void_p()\n"
        "st = L.nuna_a2a_layout_create(P, T, 1, 8, topk.ctypes.data, ctypes.byref(h))\n"
        "print(st, h.value is None, nuna.last_error())\n" % ROOT)
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr[-2000:]
    st, null_handle, msg = out.stdout.strip().split(" ", 2)
    assert int(st) == nuna.ERR_NO_MEMORY and null_handle == "True", out.stdout
    assert "allocation" in msg


def test_last_error_is_per_thread():
    """Two threads fail with different errors at the same time; each reads back its own message."""
    import threading
    lib = nuna.lib()
    results = {}
    barrier = threading.Barrier(2)

    def worker(name, P):
        barrier.wait()
        msgs = set()
        for _ in range(2000):
            st = nuna.allreduce_raw([0x1000] * P if P > 0 else [], [0x2000] * max(P, 1), P, 16, nuna.BF16)
            msgs.add((st, lib.nuna_last_error_string().decode()))
        results[name] = msgs

    threads = [threading.Thread(target=worker, args=("bad_p", 0)), threading.Thread(target=worker, args=("bad_in", 8))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert results["bad_p"] == {(nuna.ERR_INVALID_ARG, "P=0 outside [1, 64]")}
    assert len(results["bad_in"]) == 1
    st, msg = next(iter(results["bad_in"]))
    assert st == nuna.ERR_OVERLAP and "overlap" in msg


def test_counter_summary_medians(tmp_path):
    """`bench.py --summarize-counters` reports per-kernel medians and keeps only the library's kernels."""
    import subprocess
    import sys
    rows = ["Kernel_Name,Grid_Size,Counter_Name,Counter_Value"]
    for v in (3, 1, 2):
        rows.append(f'"void k_copy<1>(uint4*, int)",4096,SQ_WAVES,{v}')
    rows.append('"void k_copy<1>(uint4*, int)",4096,GRBM_GUI_ACTIVE,10')
    rows.append('"at::native::elementwise_kernel",256,SQ_WAVES,7')
    csv_path = tmp_path / "c.csv"
    csv_path.write_text("\n".join(rows) + "\n")
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--summarize-counters", str(csv_path)],
                         capture_output=True, text=True, check=True).stdout
    lines = [ln for ln in out.splitlines() if ln.startswith("| `")]
    assert len(lines) == 1
    cells = [c.strip() for c in lines[0].strip("|").split("|")]
    assert cells[1:] == ["4096", "3", "10", "2"]


# ---------------------------------------------------------------- dispatch-map check behind nuna_init

def test_dispatch_map_check_accepts_b_mod_8_on_256_cus():
    for G in (64, 65, 2048):
        assert nuna.check_dispatch_map_raw(np.arange(G) % 8, 256) == nuna.OK, nuna.last_error()


@pytest.mark.parametrize("case", ["mod4", "one_off", "shifted", "one_xcd", "cus_80", "cus_304"])
def test_dispatch_map_check_rejects_other_maps(case):
    """What the library must not take for the MI355X map: fewer XCDs (a partition mode), one workgroup on
    the wrong XCD, a rotated map, a single-XCD partition, other compute-unit counts."""
    G, cus = 2048, 256
    x = np.arange(G) % 8
    if case == "mod4":
        x = np.arange(G) % 4
    elif case == "one_off":
        x[1234] = (x[1234] + 1) % 8
    elif case == "shifted":
        x = (np.arange(G) + 1) % 8
    elif case == "one_xcd":
        x = np.zeros(G, dtype=np.int64)
    elif case == "cus_80":
        cus = 80
    elif case == "cus_304":
        cus = 304
    assert nuna.check_dispatch_map_raw(x, cus) == nuna.ERR_UNSUPPORTED
    msg = nuna.last_error()
    assert ("compute units" in msg) if case.startswith("cus") else ("workgroup" in msg), msg


def test_dispatch_map_check_rejects_bad_arguments():
    assert nuna.check_dispatch_map_raw(np.arange(63) % 8, 256) == nuna.ERR_INVALID_ARG
    assert nuna.lib().nuna_check_dispatch_map(None, 2048, 256) == nuna.ERR_INVALID_ARG


def test_device_info_without_init_is_an_error():
    info = nuna.DeviceInfo()
    st = nuna.lib().nuna_get_device_info(ctypes.byref(info))
    assert st in (nuna.ERR_HIP, nuna.ERR_INVALID_ARG), nuna.last_error()
    assert nuna.lib().nuna_get_device_info(None) == nuna.ERR_INVALID_ARG


@no_gpu_only
def test_xcd_placement_without_a_device_never_launches():
    """XCD mode first asks for the verified dispatch map of the current device; without a device that is a
    HIP error, and LINEAR mode reaches the launch, which fails the same way."""
    for place in (nuna.XCD, nuna.LINEAR):
        st = nuna.allreduce_raw(_bufs(8), _bufs(8, base=BASE + (1 << 32)), 8, 4096, nuna.BF16, nuna.ALGO_TWO_SHOT,
                                place)
        assert st == nuna.ERR_HIP, nuna.last_error()


@no_gpu_only
@pytest.mark.parametrize("algo", [nuna.ALGO_TWO_SHOT, nuna.ALGO_TWO_SHOT_TWO_KERNELS])
def test_two_shot_forms_pass_validation(algo):
    P, n = 8, 8 * 4096
    ins, outs = _bufs(P, stride=1 << 24), _bufs(P, stride=1 << 24, base=BASE + (1 << 32))
    assert nuna.allreduce_raw(ins, outs, P, n, nuna.BF16, algo, nuna.LINEAR) == nuna.ERR_HIP
    assert nuna.allreduce_raw(ins, ins, P, n, nuna.BF16, algo, nuna.LINEAR) == nuna.ERR_HIP  # in place
    assert nuna.allreduce_raw(ins, outs, P, n, nuna.BF16, 5, nuna.LINEAR) == nuna.ERR_INVALID_ARG


# ---------------------------------------------------------------- page-grouped direct map (host mirror)

@pytest.mark.parametrize("items,chunk", [(1, 1024), (16, 1024), (64, 1024), (100, 1024), (1024, 1024),
                                         (64, 256), (1000, 256), (7, 512), (4096, 4096), (33, 8192), (4, 16)])
def test_direct_map_covers_every_item_once(items, chunk):
    for place in (nuna.LINEAR, nuna.XCD):
        with nuna.tunables(NUNA_PAGE_GROUPS=1):
            m = nuna.placement_direct(place, items, chunk)
        got = m[m >= 0]
        assert sorted(got.tolist()) == list(range(items)), (place, items, chunk)
        if place == nuna.LINEAR or chunk >= 4096:
            assert m.tolist() == list(range(items))


@pytest.mark.parametrize("items,chunk", [(16, 1024), (100, 1024), (1024, 1024), (1000, 256), (64, 16), (7, 512)])
def test_direct_map_keeps_each_page_on_one_xcd(items, chunk):
    """XCD mode: the chunks of one 4 KiB page run on one XCD (workgroup b runs on XCD b mod 8), pages are
    dealt round-robin to the XCDs, and a page's chunks run on consecutive workgroup slots of its XCD."""
    gp = 4096 // chunk
    with nuna.tunables(NUNA_PAGE_GROUPS=1):
        m = nuna.placement_direct(nuna.XCD, items, chunk)
    assert m.size % (8 * gp) == 0
    where = {int(w): b for b, w in enumerate(m) if w >= 0}
    for page in range((items + gp - 1) // gp):
        bs = [where[i] for i in range(page * gp, min(items, (page + 1) * gp))]
        assert {b % 8 for b in bs} == {page % 8}, page
        ks = [b // 8 for b in bs]
        assert ks == list(range(ks[0], ks[0] + len(bs))), (page, ks)
    lin = nuna.placement_direct(nuna.LINEAR, items, chunk)
    if gp > 1 and items >= 2 * gp:
        # the linear map splits a page over min(gp, 8) XCDs
        assert lin[:gp].tolist() == list(range(gp)) and len({b % 8 for b in range(gp)}) == min(gp, 8)


def test_direct_map_follows_the_page_groups_tunable():
    """Page groups are off by default (XCD mode runs the linear map for single-item launches)."""
    assert nuna.placement_direct(nuna.XCD, 64, 1024).tolist() == list(range(64))
    with nuna.tunables(NUNA_PAGE_GROUPS=1):
        assert nuna.placement_direct(nuna.XCD, 64, 1024).tolist() != list(range(64))


def test_direct_map_rejects_bad_geometry():
    g = ctypes.c_int64()
    for items, chunk in [(0, 1024), (8, 24), (8, 0), (8, 8)]:
        assert nuna.lib().nuna_placement_direct(nuna.XCD, items, chunk, None, 0, ctypes.byref(g)) == \
            nuna.ERR_INVALID_ARG
    assert nuna.lib().nuna_placement_direct(nuna.XCD, 64, 1024, None, 0, ctypes.byref(g)) == nuna.ERR_INVALID_ARG
    assert g.value == 64


# ---------------------------------------------------------------- binding checks before any C call

class _FakeTensor:
    def __init__(self, dtype, n):
        self.dtype, self._n = dtype, n

    def numel(self):
        return self._n


def test_output_count_and_dtype_checked_before_the_library():
    """An output list shorter than the inputs, or outputs of another dtype, would make the library read
    past the pointer array or write more bytes than an output holds: the binding refuses both."""
    ins = [_FakeTensor("f32", 64) for _ in range(4)]
    with pytest.raises(ValueError, match="one output per rank"):
        nuna._check_outs(ins, [_FakeTensor("f32", 64) for _ in range(3)], 64)
    with pytest.raises(ValueError, match="dtype"):
        nuna._check_outs(ins, [_FakeTensor("f32", 64)] * 3 + [_FakeTensor("bf16", 64)], 64)
    with pytest.raises(ValueError, match="elements"):
        nuna._check_outs(ins, [_FakeTensor("f32", 16) for _ in range(4)], 64)
    nuna._check_outs(ins, [_FakeTensor("f32", 64) for _ in range(4)], 64)


def test_new_tunables_accept_and_reject():
    with nuna.tunables(NUNA_PAGE_GROUPS=1, NUNA_DIRECT_MAX_GRID=16384, NUNA_TWO_SHOT_FORM=2):
        assert nuna.get_tunable("NUNA_PAGE_GROUPS") == 1
        assert nuna.get_tunable("NUNA_DIRECT_MAX_GRID") == 16384
        assert nuna.get_tunable("NUNA_TWO_SHOT_FORM") == 2
    assert nuna.get_tunable("NUNA_PAGE_GROUPS") == 0
    assert nuna.get_tunable("NUNA_TWO_SHOT_FORM") == 0
    for name, bad in [("NUNA_PAGE_GROUPS", 2), ("NUNA_DIRECT_MAX_GRID", -1), ("NUNA_DIRECT_MAX_GRID", (1 << 24) + 1),
                      ("NUNA_TWO_SHOT_FORM", 3)]:
        with pytest.raises(nuna.NunaError):
            nuna.set_tunable(name, bad)


def test_store_gap_tunable():
    """NUNA_STORE_GAP: -1 (by size, the default) or a fixed pause count 0..32."""
    assert nuna.get_tunable("NUNA_STORE_GAP") == -1
    with nuna.tunables(NUNA_STORE_GAP=0):
        assert nuna.get_tunable("NUNA_STORE_GAP") == 0
    with nuna.tunables(NUNA_STORE_GAP=32):
        assert nuna.get_tunable("NUNA_STORE_GAP") == 32
    assert nuna.get_tunable("NUNA_STORE_GAP") == -1
    for bad in (-2, 33):
        with pytest.raises(nuna.NunaError):
            nuna.set_tunable("NUNA_STORE_GAP", bad)


def test_last_launch_of_a_call_that_launched_nothing():
    """A call rejected by its argument checks, or with nothing to do, leaves an empty launch record."""
    assert nuna.allreduce_raw(None, None, 8, 16, nuna.BF16) == nuna.ERR_INVALID_ARG
    rec = nuna.last_launch()
    assert rec["launches"] == 0 and rec["kernels"] == "" and rec["map"] == "linear"
    assert nuna.lib().nuna_last_launch(None) == nuna.ERR_INVALID_ARG


@no_gpu_only
def test_routed_dispatch_validation():
    """The allocation-free dispatch rejects, before any HIP call, routing tables larger than its scratch,
    rows that are not whole 16-byte vectors, and the usual bad arguments."""
    P, H = 8, 64
    send, recv = _bufs(P, stride=1 << 24), _bufs(P, stride=1 << 24, base=BASE + (1 << 32))
    topk, rows = BASE + (1 << 34), BASE + (1 << 35)
    call = lambda **kw: nuna.all_to_all_routed_raw(  # noqa: E731
        kw.get("send", send), kw.get("recv", recv), kw.get("topk", topk), kw.get("P", P), kw.get("T", 16),
        kw.get("k", 8), kw.get("E", 64), kw.get("row", H), kw.get("cap", 64), kw.get("dtype", nuna.BF16),
        kw.get("rows", rows))
    assert call(T=40000) == nuna.ERR_INVALID_ARG and "scratch" in nuna.last_error()
    assert call(row=7) == nuna.ERR_UNSUPPORTED
    assert call(E=60) == nuna.ERR_INVALID_ARG
    assert call(k=0) == nuna.ERR_INVALID_ARG
    assert call(topk=None) == nuna.ERR_INVALID_ARG
    assert call(rows=None) == nuna.ERR_INVALID_ARG
    assert call(topk=topk + 2) == nuna.ERR_MISALIGNED
    assert call(rows=recv[0]) == nuna.ERR_OVERLAP
    assert call() == nuna.ERR_HIP  # valid: reaches the device lookup, and there is no device here
