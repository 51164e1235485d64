"""CPU oracle for the collective copy/reduce path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library (the HIP path) does
not import, link or call it, and this package imports nothing from the
product package.

The arithmetic lives in ``nuna_oracle.c`` (plain, element-at-a-time C).  This
module only marshals numpy arrays into it.  Buffers are numpy arrays:
``float32`` for fp32 data and ``uint16`` for bf16 bit patterns.

Semantics (Sec. 2.1 of the paper names all-gather, all-reduce and
all-to-all as the collectives AI relies on, with reduce-scatter/all-gather
in tensor-parallel traces; the accumulation rule -- fp32 accumulation, ranks
added in ascending order, one final rounding -- is the one fixed for this
path):

* all-reduce:     out[d][i] = narrow(((x0[i] + x1[i]) + x2[i]) + ... )  for all d
* reduce-scatter: out[r][j] = narrow(sum_q asc  in[q][r*m + j])
* all-gather:     out[d][r*m + j] = in[r][j]   (byte copy)
* all-to-all:     recv[d] = rows send[s][t] with d among the owner ranks of
                  token (s, t)'s top-k experts, ordered by (s, t) ascending.
* combine:        out[s][t] = narrow(sum over destination ranks d ascending of
                  y[d][j(s, t, d)]), the reverse of the dispatch (MoE result
                  collection); optionally each term is first scaled by
                  weights[s][t][d] (fp32 product, rounded once).
"""
import ctypes
import os

import numpy as np

from . import build as _build

F32, BF16 = 0, 1

_c_vpp = ctypes.POINTER(ctypes.c_void_p)


def _dtype_code(a):
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"oracle buffers are float32 or uint16 (bf16 bits), got {a.dtype}")


def _ptrs(arrs):
    return (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])


class Oracle:
    """ctypes front end over one build of ``nuna_oracle.c``."""

    def __init__(self, libpath):
        lib = ctypes.CDLL(libpath)
        self.lib = lib
        lib.oracle_allreduce.argtypes = [ctypes.c_int, ctypes.c_size_t, ctypes.c_int, _c_vpp, _c_vpp]
        lib.oracle_allreduce_acc_f32.argtypes = [ctypes.c_int, ctypes.c_size_t, ctypes.c_int, _c_vpp,
                                                 ctypes.c_void_p]
        lib.oracle_reduce_scatter.argtypes = [ctypes.c_int, ctypes.c_size_t, ctypes.c_int, _c_vpp, _c_vpp]
        lib.oracle_all_gather.argtypes = [ctypes.c_int, ctypes.c_size_t, ctypes.c_int, _c_vpp, _c_vpp]
        lib.oracle_a2a_counts.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p, ctypes.c_void_p]
        lib.oracle_a2a_map.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p, ctypes.c_int,
                                                            ctypes.c_void_p, ctypes.c_void_p]
        lib.oracle_a2a_map.restype = ctypes.c_int64
        lib.oracle_all_to_all.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p, ctypes.c_size_t,
                                                                _c_vpp, _c_vpp]
        lib.oracle_a2a_combine.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int,
                                                                 ctypes.c_void_p, _c_vpp, _c_vpp]
        lib.oracle_f32_to_bf16_array.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t]
        lib.oracle_f32_to_bf16.argtypes = [ctypes.c_float]
        lib.oracle_f32_to_bf16.restype = ctypes.c_uint16
        lib.oracle_bf16_to_f32.argtypes = [ctypes.c_uint16]
        lib.oracle_bf16_to_f32.restype = ctypes.c_float

    # -- helpers ----------------------------------------------------------
    @staticmethod
    def _check_ranks(ins):
        if len(ins) < 1:
            raise ValueError("need at least one rank buffer")
        d0 = ins[0].dtype
        n0 = ins[0].size
        for a in ins:
            if a.dtype != d0 or a.size != n0 or not a.flags.c_contiguous:
                raise ValueError("rank buffers must share dtype and size and be contiguous")
        return _dtype_code(ins[0]), n0

    # -- collectives ------------------------------------------------------
    def allreduce(self, ins, outs=None):
        dt, n = self._check_ranks(ins)
        if outs is None:
            outs = [np.empty_like(ins[0]) for _ in ins]
        rc = self.lib.oracle_allreduce(len(ins), n, dt, _ptrs(ins), _ptrs(outs))
        assert rc == 0
        return outs

    def allreduce_acc(self, ins):
        dt, n = self._check_ranks(ins)
        acc = np.empty(n, dtype=np.float32)
        rc = self.lib.oracle_allreduce_acc_f32(len(ins), n, dt, _ptrs(ins), acc.ctypes.data)
        assert rc == 0
        return acc

    def reduce_scatter(self, ins):
        dt, n = self._check_ranks(ins)
        P = len(ins)
        if n % P:
            raise ValueError("reduce-scatter input size must be a multiple of P")
        m = n // P
        outs = [np.empty(m, dtype=ins[0].dtype) for _ in ins]
        rc = self.lib.oracle_reduce_scatter(P, m, dt, _ptrs(ins), _ptrs(outs))
        assert rc == 0
        return outs

    def all_gather(self, ins):
        dt, m = self._check_ranks(ins)
        P = len(ins)
        outs = [np.empty(P * m, dtype=ins[0].dtype) for _ in ins]
        rc = self.lib.oracle_all_gather(P, m, dt, _ptrs(ins), _ptrs(outs))
        assert rc == 0
        return outs

    def a2a_counts(self, topk, num_experts):
        topk = np.ascontiguousarray(topk, dtype=np.int32)
        P, T, k = topk.shape
        rows = np.zeros(P, dtype=np.int64)
        rc = self.lib.oracle_a2a_counts(P, T, k, num_experts, topk.ctypes.data, rows.ctypes.data)
        assert rc == 0
        return rows

    def a2a_map(self, topk, num_experts, d):
        topk = np.ascontiguousarray(topk, dtype=np.int32)
        P, T, k = topk.shape
        cap = P * T
        sr = np.empty(cap, dtype=np.int32)
        st = np.empty(cap, dtype=np.int32)
        j = self.lib.oracle_a2a_map(P, T, k, num_experts, topk.ctypes.data, d, sr.ctypes.data,
                                    st.ctypes.data)
        return sr[:j].copy(), st[:j].copy()

    def all_to_all(self, send, topk, num_experts):
        """send: list of P arrays shaped [T, row]; returns list of P recv arrays [rows_d, row]."""
        topk = np.ascontiguousarray(topk, dtype=np.int32)
        P, T, k = topk.shape
        if len(send) != P:
            raise ValueError("one send buffer per rank")
        for a in send:
            if a.shape[0] != T or a.shape != send[0].shape or a.dtype != send[0].dtype:
                raise ValueError("send buffers must be [T, row] of one dtype")
            if not a.flags.c_contiguous:
                raise ValueError("send buffers must be contiguous")
        row_bytes = send[0][0].nbytes if T else 0
        rows = self.a2a_counts(topk, num_experts)
        recv = [np.zeros((int(rows[d]),) + send[0].shape[1:], dtype=send[0].dtype) for d in range(P)]
        rc = self.lib.oracle_all_to_all(P, T, k, num_experts, topk.ctypes.data, row_bytes,
                                        _ptrs(send), _ptrs(recv))
        assert rc == 0
        return recv

    def combine(self, y, topk, num_experts, weights=None):
        """y: list of P arrays [rows_d, row] (one result row per received row); returns list of P
        arrays [T, row] with each token's results summed over its destination ranks (ascending).
        weights: optional float32 [P, T, P]; weights[s, t, d] scales rank d's row for token (s, t)."""
        topk = np.ascontiguousarray(topk, dtype=np.int32)
        P, T, k = topk.shape
        if weights is not None:
            weights = np.ascontiguousarray(weights, dtype=np.float32)
            if weights.shape != (P, T, P):
                raise ValueError("weights must be [P, T, P]")
        if len(y) != P:
            raise ValueError("one result buffer per rank")
        row = y[0].shape[1]
        for a in y:
            if a.ndim != 2 or a.shape[1] != row or a.dtype != y[0].dtype or not a.flags.c_contiguous:
                raise ValueError("result buffers must be contiguous [rows, row] of one dtype")
        dt = _dtype_code(y[0])
        out = [np.zeros((T, row), dtype=y[0].dtype) for _ in range(P)]
        ys = [a if a.size else np.zeros((1, row), dtype=a.dtype) for a in y]
        wp = weights.ctypes.data if weights is not None and weights.size else None
        rc = self.lib.oracle_a2a_combine(P, T, k, num_experts, topk.ctypes.data, row, dt, wp, _ptrs(ys), _ptrs(out))
        assert rc == 0
        return out

    # -- rounding ---------------------------------------------------------
    def f32_to_bf16(self, x):
        x = np.ascontiguousarray(x, dtype=np.float32)
        y = np.empty(x.shape, dtype=np.uint16)
        self.lib.oracle_f32_to_bf16_array(x.ctypes.data, y.ctypes.data, x.size)
        return y


_default = None


def get():
    """The oracle built from ``nuna_oracle.c``; builds it once if absent."""
    global _default
    if _default is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _default = Oracle(_build.LIB)
    return _default


def allreduce(ins, outs=None):
    return get().allreduce(ins, outs)


def allreduce_acc(ins):
    return get().allreduce_acc(ins)


def reduce_scatter(ins):
    return get().reduce_scatter(ins)


def all_gather(ins):
    return get().all_gather(ins)


def a2a_counts(topk, num_experts):
    return get().a2a_counts(topk, num_experts)


def a2a_map(topk, num_experts, d):
    return get().a2a_map(topk, num_experts, d)


def all_to_all(send, topk, num_experts):
    return get().all_to_all(send, topk, num_experts)


def combine(y, topk, num_experts, weights=None):
    return get().combine(y, topk, num_experts, weights)


def f32_to_bf16(x):
    return get().f32_to_bf16(x)
