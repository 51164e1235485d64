"""Helpers for GPU tests: numpy <-> torch moves and bitwise comparison."""
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
