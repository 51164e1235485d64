"""The allocation-free dispatch, nuna_all_to_all_routed, against nuna_all_to_all.

The routed dispatch reads the top-k table from device memory and builds its
routing in the library's static scratch array (at decode sizes, up to 256
tokens over all ranks, every workgroup recomputes the routing and no scratch
is used); the layout dispatch plans on the host and reads tables the library
allocated at upload.  Both must produce the oracle's receive buffers bit for
bit.  Two calls in a row share the one scratch array, the second smaller than
the first, so a table left from the first call must not leak into the second.
Rows past each rank's count (and past the caller's capacity) must stay
untouched.
"""
import numpy as np
import pytest

import oracle
from gpu_util import assert_bitwise, to_host
from paper_2608_00867_amd import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SENTINEL = 0x7FA5  # a NaN payload no routed row carries (rows are N(0,1) bf16)


@pytest.fixture(scope="module")
def nuna():
    from paper_2608_00867_amd import nuna as n
    n.init()
    return n


def _dev_rows(a):
    return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()


def _recv(P, cap, H):
    return [torch.full((cap, H), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16) for _ in range(P)]


def _routed(nuna, send, topk, E, cap, H, place, misalign=False):
    P = len(send)
    recv = _recv(P, cap, H)
    rows = torch.full((P + 1,), -1, dtype=torch.int64, device="cuda")
    flat = np.ascontiguousarray(topk, dtype=np.int32).reshape(-1)
    if misalign:  # the table 4 bytes past a 16-byte boundary: the 4-byte loads of the top-k entries
        buf = torch.zeros(flat.size + 1, dtype=torch.int32, device="cuda")
        buf[1:].copy_(torch.from_numpy(flat))
        topk_dev = buf[1:].view(topk.shape)
        assert topk_dev.data_ptr() % 16 == 4
    else:
        topk_dev = torch.from_numpy(flat).cuda().view(topk.shape)
    nuna.all_to_all_routed(send, recv, topk_dev, E, rows, placement=place)
    torch.cuda.synchronize()
    return recv, rows.cpu().numpy()


def _check_case(nuna, P, T, k, E, H, seed, place, cap_extra=8, topk_override=None, misalign=False):
    send_np = wl.moe_rows(P, T, H, seed)
    topk = wl.moe_routing(P, T, k, E, seed + 1) if topk_override is None else topk_override
    valid = np.where((topk >= 0) & (topk < E), topk, -1)
    # The oracle's routing: an out-of-range entry replaced by a valid expert of the same token routes the
    # same way (the routed dispatch ignores out-of-range entries; the oracle and the layout refuse them).
    fixed = topk.copy()
    for idx in zip(*np.nonzero(valid < 0)):
        s, t, _ = idx
        fixed[s, t, idx[2]] = valid[s, t][valid[s, t] >= 0][0]
    ref = oracle.all_to_all(send_np, fixed, E)
    want_rows = np.array([r.shape[0] for r in ref], dtype=np.int64)
    send = [_dev_rows(a.reshape(-1)).view(T, H) for a in send_np]
    cap = int(want_rows.max()) + cap_extra
    # the layout dispatch (allocating path) on the same routing
    lay = nuna.A2ALayout(fixed, E).upload()
    assert np.array_equal(lay.recv_rows(), want_rows)
    recv_l = _recv(P, max(cap, int(want_rows.max())), H)
    nuna.all_to_all(send, recv_l, lay, placement=place)
    recv_r, rows = _routed(nuna, send, topk, E, cap, H, place, misalign)
    assert np.array_equal(rows[:P], want_rows), (rows, want_rows)
    assert rows[P] == int(np.sum(valid < 0))
    for d in range(P):
        n = min(int(want_rows[d]), cap)
        got = to_host(recv_r[d])
        assert_bitwise(got[:n], ref[d][:n], f"routed P={P} T={T} {place} rank {d}")
        assert_bitwise(got[:n], to_host(recv_l[d])[:n], f"routed vs layout P={P} T={T} {place} rank {d}")
        assert np.all(got[n:].view(np.int16) == SENTINEL), f"rank {d}: rows past the count were written"
    lay.close()


@pytest.mark.parametrize("place", ["linear", "xcd"])
def test_routed_matches_layout_dispatch_twice(nuna, place):
    """The MoE shape (8 ranks, 512 tokens x 7168, top-8 of 256), then a smaller call on the same scratch
    (100 tokens per rank), then the decode shape (16 tokens per rank, no scratch)."""
    _check_case(nuna, 8, wl.MOE_TOKENS, 8, wl.MOE_EXPERTS, wl.HIDDEN_MOE, 21, place)
    _check_case(nuna, 8, 100, 8, wl.MOE_EXPERTS, wl.HIDDEN_MOE, 23, place)
    _check_case(nuna, 8, 16, 8, wl.MOE_EXPERTS, wl.HIDDEN_MOE, 22, place)


def test_routed_launch_record_names_the_map(nuna):
    """With XCD placement the copies of a token row run as one group per token (top-8 of 8 ranks: groups of 8);
    with LINEAR, in order.  Up to 256 tokens over all ranks one kernel routes and copies."""
    P, k, E, H = 8, 8, 256, 128
    for T, kernels in ((64, "k_route_count+k_route_copy"), (32, "k_route_small")):
        send = [_dev_rows(a.reshape(-1)).view(T, H) for a in wl.moe_rows(P, T, H, 51)]
        topk = wl.moe_routing(P, T, k, E, 52)
        for place, want in (("xcd", "xcd_groups"), ("linear", "linear")):
            _routed(nuna, send, topk, E, T * P, H, place)
            rec = nuna.last_launch()
            assert rec["kernels"] == kernels and rec["map"] == want, rec
            assert rec["grid"] == P * T * min(k, P), rec


@pytest.mark.parametrize("grid", [7, 24])
def test_routed_capped_grid_runs_several_items_per_workgroup(nuna, grid):
    """A capped grid hands every workgroup many (token, slot) items: the decode kernel's per-item counts
    alternate between two LDS buffers, and the copy kernel's prefix is reused across items.  7 workgroups
    run the linear map, 24 the XCD map."""
    with nuna.tunables(NUNA_MAX_GRID=grid):
        _check_case(nuna, 8, 30, 8, 256, 72, 61, "xcd")
        _check_case(nuna, 8, 120, 8, 256, 72, 62, "xcd")
        _check_case(nuna, 64, 4, 8, 256, 40, 63, "linear")

def test_routed_many_ranks_odd_rows_and_edges(nuna):
    """64 ranks; rows of one 16-byte vector and of several column passes; one token per rank; several passes
    of the routing kernel; no tokens."""
    _check_case(nuna, 64, 40, 8, 256, 64, 31, "xcd")
    _check_case(nuna, 3, 50, 2, 6, 8, 32, "linear")
    _check_case(nuna, 5, 7, 5, 10, 8 * 1100, 33, "xcd")
    _check_case(nuna, 8, 1, 8, 64, 128, 34, "linear")
    # the decode kernel at 64 ranks (256 tokens, 2048 entries: its largest table) and just past it
    _check_case(nuna, 64, 4, 8, 256, 64, 37, "xcd")
    _check_case(nuna, 64, 4, 9, 256, 64, 38, "xcd")
    _check_case(nuna, 8, 33, 8, 256, 64, 39, "linear")
    # copy kernel prefixes: 16 ranks (column loads) and 17 ranks (not a power of two)
    _check_case(nuna, 16, 100, 8, 256, 64, 43, "xcd")
    _check_case(nuna, 17, 80, 4, 34, 64, 44, "xcd")
    # a top-k table that is not 16-byte aligned, at top-8: decode kernel and routing kernel
    _check_case(nuna, 8, 16, 8, 256, 64, 50, "xcd", misalign=True)
    _check_case(nuna, 8, 100, 8, 256, 64, 51, "linear", misalign=True)
    # top-k longer than one load round (8 entries): 12 and 16 of 48 experts
    _check_case(nuna, 8, 20, 16, 48, 64, 52, "xcd")
    _check_case(nuna, 8, 100, 16, 48, 64, 53, "linear")
    _check_case(nuna, 8, 20, 12, 48, 64, 45, "xcd")
    _check_case(nuna, 8, 200, 12, 48, 64, 46, "linear")
    # more tokens than one pass of the routing kernel (1024): ranks carried across passes
    _check_case(nuna, 8, 3000, 8, 256, 64, 35, "xcd")
    _check_case(nuna, 4, 2500, 3, 16, 32, 36, "linear")
    P, H, E = 4, 64, 8
    send = [torch.zeros((1, H), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    recv = _recv(P, 4, H)
    rows = torch.full((P + 1,), -1, dtype=torch.int64, device="cuda")
    st = nuna.all_to_all_routed_raw([t.data_ptr() for t in send], [t.data_ptr() for t in recv], None, P, 0, 2, E, H,
                                    4, nuna.BF16, rows.data_ptr())
    assert st == nuna.OK, nuna.last_error()
    torch.cuda.synchronize()
    assert rows.cpu().tolist() == [0] * (P + 1)
    for d in range(P):
        assert np.all(to_host(recv[d]).view(np.int16) == SENTINEL)


def test_routed_out_of_range_experts_and_capacity(nuna):
    """Entries outside [0, E) route nowhere and are counted; rows past the capacity are not written
    while the counts still report every row."""
    P, T, k, E, H = 8, 100, 4, 64, 256
    topk = wl.moe_routing(P, T, k, E, 41)
    topk[0, 0, 0] = -1
    topk[3, 7, 2] = E
    topk[5, 9, 1] = 1 << 30
    _check_case(nuna, P, T, k, E, H, 40, "xcd", topk_override=topk)
    _check_case(nuna, P, T, k, E, H, 42, "linear", cap_extra=-20)
    # the same at decode size (one kernel, no scratch)
    T = 20
    topk = wl.moe_routing(P, T, k, E, 47)
    topk[0, 0, 0] = -1
    topk[3, 7, 2] = E
    topk[7, 19, 3] = -(1 << 30)
    _check_case(nuna, P, T, k, E, H, 48, "xcd", topk_override=topk)
    _check_case(nuna, P, T, k, E, H, 49, "linear", topk_override=topk, cap_extra=-6)


def test_routed_rejects_calls_beyond_the_scratch(nuna):
    P, H = 8, 64
    send = [torch.empty((1, H), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    recv = _recv(P, 4, H)
    rows = torch.zeros(P + 1, dtype=torch.int64, device="cuda")
    T = 40000  # 4 * 8 * 40000 * 8 bytes of records > 8 MiB
    st = nuna.all_to_all_routed_raw([t.data_ptr() for t in send], [t.data_ptr() for t in recv],
                                    rows.data_ptr() + 4096 * 64, P, T, 8, 64, H, 4, nuna.BF16, rows.data_ptr())
    assert st == nuna.ERR_INVALID_ARG and "scratch" in nuna.last_error(), nuna.last_error()
