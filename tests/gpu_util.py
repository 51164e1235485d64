"""Helpers for GPU tests: numpy <-> torch moves, bitwise comparison, and the MoE dispatch and combine
drivers (guarded device buffers around one library call each)."""
import numpy as np


def to_dev(a):
    """numpy (float32 or uint16 bf16 bits) -> CUDA tensor (float32 or bfloat16)."""
    import torch
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_host(t):
    """CUDA tensor -> numpy (float32 or uint16 bf16 bits)."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def bits(a):
    return a.view(np.uint16) if a.dtype == np.uint16 else a.view(np.uint32)


def assert_bitwise(got, exp, what=""):
    g, e = bits(got), bits(exp)
    if not np.array_equal(g, e):
        idx = np.flatnonzero(g.ravel() != e.ravel())
        i = int(idx[0])
        raise AssertionError(f"{what}: {idx.size} mismatches; first at {i}: got {hex(int(g.ravel()[i]))} "
                             f"expected {hex(int(e.ravel()[i]))}")


def is_nan_bits(a):
    b = bits(a).astype(np.uint64)
    if a.dtype == np.uint16:
        return (b & 0x7FFF) > 0x7F80
    return (b & 0x7FFFFFFF) > 0x7F800000


def assert_bitwise_nan_aware(got, exp, what=""):
    """Bitwise on non-NaN results; NaN results need only be NaN on both sides (IEEE-754 leaves the
    payload of an arithmetic NaN result to the implementation)."""
    gn, en = is_nan_bits(got), is_nan_bits(exp)
    assert np.array_equal(gn, en), f"{what}: NaN positions differ"
    assert_bitwise(got[~gn], exp[~en], what)


def run_a2a(nuna, send_np, topk, E, place, guard_rows=2):
    """Dispatch on the GPU.  Receive buffers hold `guard_rows` sentinel rows past the largest rank's
    rows; every row past a rank's own must keep its sentinel."""
    import torch
    P = len(send_np)
    lay = nuna.A2ALayout(topk, E).upload()
    rows = lay.recv_rows()
    send = [to_dev(a) for a in send_np]
    H = send_np[0].shape[1]
    cap = int(rows.max()) if rows.size else 0
    cap = max(cap, 1)
    recv_whole = [torch.full((cap + guard_rows, H), 0, dtype=send[0].dtype, device="cuda") for _ in range(P)]
    for w in recv_whole:
        w.view(torch.int16 if w.dtype == torch.bfloat16 else torch.int32).fill_(0x3C3C)
    recv = [w[:cap] for w in recv_whole]
    nuna.all_to_all(send, recv, lay, placement=place)
    torch.cuda.synchronize()
    out = []
    for d in range(P):
        whole = to_host(recv_whole[d])
        tailbits = whole[int(rows[d]):].view(np.uint16 if whole.dtype == np.uint16 else np.uint32)
        assert np.all(tailbits == 0x3C3C), f"rank {d}: write past its rows"
        out.append(whole[:int(rows[d])])
    lay.close()
    return out


def run_combine(nuna, y_np, topk, E, place, pad=64, weights=None):
    """Combine on the GPU.  Result buffers are padded past each rank's rows with NaN rows, so a
    read of a wrong row shows in the output; outputs have `pad` guard elements on both sides
    (64 elements keep the output 16-byte aligned)."""
    import torch
    P, T = int(topk.shape[0]), int(topk.shape[1])
    lay = nuna.A2ALayout(topk, E).upload()
    rows = lay.recv_rows()
    H = y_np[0].shape[1]
    tdt = torch.bfloat16 if y_np[0].dtype == np.uint16 else torch.float32
    ibits = torch.int16 if tdt == torch.bfloat16 else torch.int32
    nan = 0x7FC1 if tdt == torch.bfloat16 else 0x7FC00001
    cap = max(int(rows.max()), 1) + 1
    y = []
    for d in range(P):
        buf = torch.empty((cap, H), dtype=tdt, device="cuda")
        buf.view(ibits).fill_(nan)
        buf[:int(rows[d])] = to_dev(y_np[d])
        y.append(buf)
    out_whole = [torch.empty(T * H + 2 * pad, dtype=tdt, device="cuda") for _ in range(P)]
    for w in out_whole:
        w.view(ibits).fill_(0x3C3C)
    out = [w[pad:pad + T * H].view(T, H) for w in out_whole]
    w = to_dev(weights) if weights is not None else None
    nuna.all_to_all_combine(y, out, lay, placement=place, weights=w)
    torch.cuda.synchronize()
    got = []
    for s in range(P):
        whole = to_host(out_whole[s])
        band = np.concatenate([whole[:pad], whole[pad + T * H:]])
        assert np.all(band.view(np.uint16 if whole.dtype == np.uint16 else np.uint32) == 0x3C3C), \
            f"rank {s}: write outside its output rows"
        got.append(whole[pad:pad + T * H].reshape(T, H))
    lay.close()
    return got


def gate_weights(topk, E, seed):
    """Dense [P, T, P] weights: with E == P the router's gate of the token's expert on rank d,
    otherwise any positive weight per destination rank."""
    P, T, k = topk.shape
    g = np.random.default_rng(seed)
    w = np.zeros((P, T, P), dtype=np.float32)
    per = E // P
    for s in range(P):
        for t in range(T):
            for q in range(k):
                w[s, t, int(topk[s, t, q]) // per] = np.float32(g.random())
    return w
