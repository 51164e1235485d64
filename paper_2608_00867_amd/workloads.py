"""Seeded synthetic inputs shared by the oracle side and the HIP side.

This module holds input generation only -- none of the collective arithmetic.
Values are produced on the host with numpy's PCG64 (``default_rng``) from a
fixed seed per workload, so the oracle and the GPU see identical bits.

Buffers are numpy arrays: ``float32`` for fp32 data, ``uint16`` for bf16 bit
patterns.  N(0,1) bf16 data is drawn in fp32 and converted to bf16 with
torch's CPU conversion (round-to-nearest-even), a library routine.

Workload shapes (inference-shaped messages; hidden 8192 is the Llama-70B
class the paper uses for its tensor-parallel example in Sec. 6.7, hidden 7168
with 256 experts and top-8 routing is the DeepSeek-V3 class MoE named in
Sec. 5.2):

* ``ar_f32_int``   one-shot all-reduce, P=8, 2048 fp32 elements per rank,
                    integers uniform in [-8, 8] (inclusive).
* ``ar_bf16_decode`` one-shot all-reduce bf16, P=8, [T, 8192], T in {1,4,16,64}.
* ``ar_bf16_prefill`` two-shot all-reduce bf16, P=8, [T, 8192],
                    T in {256, 1024, 4096}.
* ``a2a_moe``      all-to-all dispatch bf16, P=8, 512 tokens x 7168 per rank,
                    top-8 distinct experts of 256 chosen uniformly, 32 experts
                    per rank.
* ``ar_bf16_p64``  one-shot all-reduce bf16, P=64, {16..256} KiB per rank.
* ``a2a_moe`` combine: the same routing, with N(0,1) bf16 result rows in
                    place of the expert outputs (``result_rows``).
"""
import numpy as np

BASE_SEED = 0x4E554E41

HIDDEN_DENSE = 8192
HIDDEN_MOE = 7168

DECODE_TOKENS = (1, 4, 16, 64)
PREFILL_TOKENS = (256, 1024, 4096)
P64_KIB = (16, 32, 64, 128, 256)

MOE_TOKENS = 512
MOE_TOPK = 8
MOE_EXPERTS = 256


def seed_for(workload_id, sub=0):
    """One fixed seed per (workload, sub-case)."""
    return BASE_SEED + 1000 * int(workload_id) + int(sub)


def _rng(seed):
    return np.random.default_rng(seed)


def int_uniform_f32(P, n, lo, hi, seed):
    """P fp32 buffers of integers uniform in [lo, hi] (inclusive)."""
    g = _rng(seed)
    return [g.integers(lo, hi, size=n, endpoint=True).astype(np.float32) for _ in range(P)]


def int_uniform_bf16(P, n, lo, hi, seed):
    """P bf16 buffers of small integers (exact in bf16 while |x| <= 256)."""
    import torch
    out = []
    for a in int_uniform_f32(P, n, lo, hi, seed):
        out.append(torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy())
    return out


def f32_to_bf16_bits(a):
    """Convert an fp32 array to bf16 bit patterns with torch's CPU conversion."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def normal_f32(P, n, seed):
    g = _rng(seed)
    return [g.standard_normal(n, dtype=np.float32) for _ in range(P)]


def normal_bf16(P, n, seed):
    """P bf16 buffers of N(0,1) values (drawn fp32, rounded to bf16)."""
    g = _rng(seed)
    return [f32_to_bf16_bits(g.standard_normal(n, dtype=np.float32)) for _ in range(P)]


def random_bits(P, n, dtype, seed):
    """Arbitrary bit patterns (NaN payloads, infinities, denormals included)."""
    g = _rng(seed)
    if dtype == np.uint16:
        return [g.integers(0, 1 << 16, size=n, dtype=np.uint32).astype(np.uint16) for _ in range(P)]
    return [g.integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32).view(np.float32)
            for _ in range(P)]


def moe_routing(P, T, k, E, seed):
    """top-k distinct experts per token, chosen uniformly without replacement.

    Returns int32 [P, T, k].  Each token's expert set is the first k entries
    of a uniformly random permutation of the E experts.
    """
    g = _rng(seed)
    keys = g.random((P, T, E))
    return np.argsort(keys, axis=-1, kind="stable")[..., :k].astype(np.int32)


def moe_rows(P, T, hidden, seed):
    """P send buffers [T, hidden] of N(0,1) bf16 token rows."""
    g = _rng(seed)
    return [f32_to_bf16_bits(g.standard_normal(T * hidden, dtype=np.float32)).reshape(T, hidden)
            for _ in range(P)]


def result_rows(rows, hidden, dtype, seed):
    """One buffer per rank of N(0,1) result rows, rows[d] x hidden (expert outputs to combine).
    fp32 values are scaled by 2^u, u uniform in [-12, 12], so that the order in which a
    token's results are added changes the rounded sum."""
    g = _rng(seed)
    out = []
    for r in rows:
        n = int(r) * hidden
        if dtype == np.uint16:
            out.append(f32_to_bf16_bits(g.standard_normal(n, dtype=np.float32)).reshape(int(r), hidden))
        else:
            v = g.standard_normal(n) * np.exp2(g.integers(-12, 12, size=n, endpoint=True))
            out.append(v.astype(np.float32).reshape(int(r), hidden))
    return out


def gate_weights(topk, num_experts, seed):
    """fp32 [P, T, P] combine weights: for each token, a uniform (0, 1) weight for every destination
    rank that owns one of its experts, 0 for the other ranks."""
    P, T, k = topk.shape
    g = _rng(seed)
    w = np.zeros((P, T, P), dtype=np.float32)
    ranks = np.asarray(topk) // (num_experts // P)
    np.put_along_axis(w, ranks, g.random((P, T, k)).astype(np.float32), axis=2)
    return w


# ---- named workloads ------------------------------------------------------

def ar_f32_int(seed=None, P=8, n=2048):
    seed = seed_for(1) if seed is None else seed
    return int_uniform_f32(P, n, -8, 8, seed)


def ar_bf16_decode(T, seed=None, P=8):
    seed = seed_for(2, T) if seed is None else seed
    return normal_bf16(P, T * HIDDEN_DENSE, seed)


def ar_bf16_prefill(T, seed=None, P=8):
    seed = seed_for(3, T) if seed is None else seed
    return normal_bf16(P, T * HIDDEN_DENSE, seed)


def a2a_moe(seed=None, P=8, T=MOE_TOKENS, hidden=HIDDEN_MOE, k=MOE_TOPK, E=MOE_EXPERTS):
    seed = seed_for(4) if seed is None else seed
    topk = moe_routing(P, T, k, E, seed)
    send = moe_rows(P, T, hidden, seed + 1)
    return send, topk


def ar_bf16_p64(kib, seed=None, P=64):
    seed = seed_for(5, kib) if seed is None else seed
    n = kib * 1024 // 2
    return normal_bf16(P, n, seed)
