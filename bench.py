#!/usr/bin/env python3
"""Benchmark of the collective copy/reduce path on one MI355X.

Default workload (one JSON line on stdout): the two-shot all-reduce, bf16 data
with fp32 accumulation, P=8 simulated ranks, prefill-shaped messages [T, 8192]
for T in {256, 1024, 4096} (4, 16 and 64 MiB per rank).  One step = one
two-shot all-reduce at each of the three sizes.  Calls are captured in HIP
graphs and replayed; the buffers sit in a 3 GiB pool and every call meets
inputs that are not resident in L2 or the 256 MB Infinity Cache (cold).
NUNA-aware (XCD) and locality-unaware (LINEAR) placement are timed
interleaved A/B; ``value`` is the XCD-placement throughput.  The same line
carries per-size figures of the fused and the two-kernel two-shot and of the
one-shot, the decode all-reduce sweep, the MoE dispatch, the dominant
kernel's roofline and the oracle timed on the host.

Throughput = algorithmic bytes / time.  Algorithmic bytes of an all-reduce
call are (P reads + P writes) * n * element size.

``--full`` instead sweeps every workload (fp32 integer all-reduce, decode and
prefill all-reduce, MoE all-to-all dispatch and combine, P=64 all-reduce,
standalone reduce-scatter and all-gather) in both modes, cold and warm, and
writes JSONL to ``--out``.  ``--set NAME=VALUE`` applies a launch-shape
tunable to any run (shape sweeps).
"""
import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

METRIC = ("collective latency (µs) + effective HBM GB/s vs msg size, NUNA-aware vs unaware, 1 GPU")
HBM_PEAK_GBPS = 8000.0
POOL_BYTES_MAIN = 3 << 30  # 3 GiB
ALIGN = 4096


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1280, help="timed steps per placement mode")
    ap.add_argument("--warmup", type=int, default=3, help="untimed graph replays before timing")
    ap.add_argument("--reps", type=int, default=15, help="timed replays per size in the sweeps")
    ap.add_argument("--full", action="store_true", help="sweep every workload and write JSONL")
    ap.add_argument("--out", default=None, help="JSONL output file of --full and --interference (required there)")
    ap.add_argument("--only", default=None, metavar="PREFIX",
                    help="with --full: only the workloads whose name starts with PREFIX")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="oracle timing budget (cpu_baseline)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV", default=None,
                    help="print a markdown summary of a rocprofv3 --kernel-trace CSV (per kernel and grid)")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"), default=None,
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of --profile into HBM traffic "
                         "per launch of the dominant kernel, scaled by the reference copy; writes "
                         "profiles/dominant_traffic.json and prints markdown")
    ap.add_argument("--interference", action="store_true",
                    help="all-gather (P=8, 1 MiB per output) and split all-reduce (P=8, [64, 8192]) timed while a "
                         "hipBLASLt GEMM with about 100 output tiles runs on another stream, K swept, LINEAR vs XCD; "
                         "writes JSONL to --out")
    ap.add_argument("--affinity", action="store_true",
                    help="probe which die (XCDs 0-3 or 4-7) is near each 8 KiB block of an all-reduce's 16 rank "
                         "buffers (decode T=64 and prefill T=1024 layouts of the pool) and print how well the "
                         "buffers agree offset by offset")
    ap.add_argument("--cu-affinity", action="store_true",
                    help="per-compute-unit cold-load latency from every CU of every XCD to every 8 KiB block of a "
                         "64 MiB buffer; prints a JSON summary and a markdown table")
    ap.add_argument("--profile", type=int, default=0, metavar="N",
                    help="profiling run: N cold launches each of the dominant kernel (fused two-shot all-reduce, "
                         "P=8, [4096, 8192] bf16, XCD), the 64 MiB reference copy, the two-kernel two-shot at "
                         "[256, 8192], the split all-reduce (decode T=64), the MoE dispatch and combine, eager, "
                         "then exit")
    ap.add_argument("--summarize-counters", metavar="CSV", default=None,
                    help="print per-kernel medians of every counter in one rocprofv3 --pmc CSV")
    ap.add_argument("--summarize-l2", nargs=2, metavar=("LINEAR_CSV", "XCD_CSV"), default=None,
                    help="markdown table of TCC_HIT_sum / TCC_MISS_sum from two --profile runs (LINEAR, XCD)")
    ap.add_argument("--xcc-counter-defs", metavar="YAML", default=None,
                    help="write rocprofv3 counter definitions TCC_HIT_XCC<x> / TCC_MISS_XCC<x> (L2 hits and misses of "
                         "one XCD, summed over its 16 channels) for `rocprofv3 -E`, then exit")
    ap.add_argument("--summarize-l2-xcc", nargs="+", metavar="PLACE=CSV", default=None,
                    help="markdown table of per-XCD L2 hit rates from --profile runs with the --xcc-counter-defs "
                         "counters, e.g. linear=a.csv linear=b.csv xcd=c.csv ...")
    ap.add_argument("--profile-place", choices=("linear", "xcd"), default="xcd",
                    help="placement of the split all-reduce and MoE kernels in --profile")
    ap.add_argument("--set", action="append", default=[], metavar="NAME=VALUE",
                    help="launch-shape tunable for this run (repeatable), e.g. NUNA_VPT=2")
    ap.add_argument("--kernel-json", metavar="JSON", default=None,
                    help="with --summarize-trace: also write the dominant kernel's traced average duration to JSON")
    ap.add_argument("--summarize-phases", metavar="KERNEL_TRACE_CSV", default=None,
                    help="per-phase durations and the gap between the phases of the two-kernel two-shot, from a "
                         "rocprofv3 --kernel-trace CSV of the default bench")
    return ap.parse_args()


# ---------------------------------------------------------------------------------------------- buffers

class Pool:
    """One big device allocation carved into 4 KiB-aligned buffer sets at rotating offsets."""

    def __init__(self, torch, nbytes):
        self.torch = torch
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        self.nbytes = nbytes
        self.off = 0

    def take(self, nbytes):
        nbytes = (nbytes + ALIGN - 1) // ALIGN * ALIGN
        if self.off + nbytes > self.nbytes:
            self.off = 0
        v = self.buf[self.off:self.off + nbytes]
        self.off += nbytes
        return v

    def rank_views(self, P, nelem, dtype, region):
        es = 2 if dtype == self.torch.bfloat16 else 4
        per = (nelem * es + ALIGN - 1) // ALIGN * ALIGN
        return [region[r * per:r * per + nelem * es].view(dtype) for r in range(P)]


def ar_footprint(P, n, es):
    per = (n * es + ALIGN - 1) // ALIGN * ALIGN
    return 2 * P * per


# ---------------------------------------------------------------------------------------------- timing

def time_graphs(torch, graphs, calls_per_graph, reps, warmup):
    """Replay each graph `warmup` times, then `reps` rounds interleaving all graphs (A/B/A/B).
    Returns {name: [us per call, ...]} from HIP events on the current stream."""
    for _ in range(warmup):
        for g in graphs.values():
            g.replay()
    torch.cuda.synchronize()
    res = {k: [] for k in graphs}
    names = list(graphs)
    for rep in range(reps):
        for k in (names if rep % 2 == 0 else names[::-1]):  # A/B then B/A
            g = graphs[k]
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            g.replay()
            b.record()
            b.synchronize()
            res[k].append(a.elapsed_time(b) * 1e3 / calls_per_graph)
    return res


def capture(torch, fn, ncalls):
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn(0)  # warm-up launch outside capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(ncalls):
            fn(i)
    torch.cuda.synchronize()
    return g


def stats(v):
    v = sorted(v)
    q = lambda p: v[min(len(v) - 1, max(0, int(round(p * (len(v) - 1)))))]  # noqa: E731
    return {"median": statistics.median(v), "p10": q(0.1), "p90": q(0.9), "mean": statistics.mean(v)}


# ---------------------------------------------------------------------------------------------- workloads

COLD_SPAN = 512 << 20  # bytes a graph's buffer rotation must sweep to leave L2 and the Infinity Cache cold
GRAPH_BYTES = 8 << 30  # bytes one timed graph moves (calls_for)


def dev_copy_of(torch, a):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def ar_sets(torch, pool, x_np, nsets, src=None):
    """`nsets` (ins, outs) buffer sets at rotating pool offsets, inputs filled with x."""
    P, n = len(x_np), x_np[0].size
    dt = torch.bfloat16 if x_np[0].dtype == np.uint16 else torch.float32
    es = 2 if dt == torch.bfloat16 else 4
    if src is None:
        src = [dev_copy_of(torch, a) for a in x_np]
    sets = []
    for _ in range(nsets):
        region = pool.take(ar_footprint(P, n, es))
        half = region.numel() // 2
        ins = pool.rank_views(P, n, dt, region[:half])
        outs = pool.rank_views(P, n, dt, region[half:])
        for a, b in zip(ins, src):
            a.copy_(b)
        sets.append((ins, outs))
    return sets


def oracle_check_ar(nuna, torch, x_np, algo, place, ref=None):
    """One call on fresh buffers compared bit for bit with the oracle (`ref`: its result, if known)."""
    import oracle
    ref = oracle.allreduce(x_np) if ref is None else ref
    dt = torch.bfloat16 if x_np[0].dtype == np.uint16 else torch.float32
    ins = [dev_copy_of(torch, a) for a in x_np]
    outs = nuna.allreduce(ins, algo=algo, placement=place)
    torch.cuda.synchronize()
    for d, o in enumerate(outs):
        g = o.cpu()
        g = g.view(torch.int16).numpy().view(np.uint16) if dt == torch.bfloat16 else g.numpy()
        if not np.array_equal(g.view(ref[d].dtype), ref[d]):
            return False
    return True


def calls_for(fp, max_calls=4096):
    """Calls per captured graph, each call moving `fp` bytes: enough that one graph moves GRAPH_BYTES
    (at least 4 calls, at most max_calls).  The timer stops when the graph's last kernel ends, while
    up to 256 MB of its writes can still sit in the Infinity Cache and drain in the gap before the
    next replay; over several GiB per graph that gap and the replay's own launch stay a few percent.
    Graphs of 4 calls at 64-576 MiB each moved the figures both ways on MI355X: most large calls
    ran 2-8 % slower per call than back to back, and one write-heavy all-gather variant ran 1.5x
    faster."""
    return int(min(max_calls, max(4, math.ceil(GRAPH_BYTES / fp))))


def bench_allreduce(nuna, torch, pool, x_np, algo, reps, warmup, cold=True, places=("linear", "xcd"),
                    max_calls=4096):
    P, n = len(x_np), x_np[0].size
    es = 2 if x_np[0].dtype == np.uint16 else 4
    fp = ar_footprint(P, n, es)
    calls = calls_for(fp, max_calls)
    nsets = max(1, min(calls, pool.nbytes // fp)) if cold else 1
    pool.off = 0
    sets = ar_sets(torch, pool, x_np, nsets)
    graphs = {}
    for place in places:
        graphs[place] = capture(torch, lambda i, place=place: nuna.allreduce(
            sets[i % nsets][0], sets[i % nsets][1], algo=algo, placement=place), calls)
    t = time_graphs(torch, graphs, calls, reps, warmup)
    alg_bytes = 2 * P * n * es
    out = {}
    for place in places:
        st = stats(t[place])
        out[place] = {"us": st, "gbps": alg_bytes / (st["median"] * 1e-6) / 1e9}
    del graphs, sets
    return alg_bytes, out, calls


def bench_rs_ag(nuna, torch, pool, kind, x_np, reps, warmup, cold=True, places=("linear", "xcd")):
    """Standalone reduce-scatter (kind "rs": in[r] holds P*m elements, out[r] m) or all-gather
    (kind "ag": in[r] holds m, out[d] P*m), timed like the all-reduce.  Returns algorithmic bytes
    (P inputs read + P outputs written), per-placement results, calls per graph and parity."""
    import oracle
    P, n_in = len(x_np), x_np[0].size
    es = 2 if x_np[0].dtype == np.uint16 else 4
    dt = torch.bfloat16 if es == 2 else torch.float32
    n_out = n_in // P if kind == "rs" else n_in * P
    per_in = (n_in * es + ALIGN - 1) // ALIGN * ALIGN
    per_out = (n_out * es + ALIGN - 1) // ALIGN * ALIGN
    fp = P * (per_in + per_out)
    calls = calls_for(fp)
    nsets = max(1, min(calls, pool.nbytes // fp)) if cold else 1
    pool.off = 0
    src = [dev_copy_of(torch, a) for a in x_np]
    sets = []
    for _ in range(nsets):
        region = pool.take(fp)
        ins = [region[r * per_in:r * per_in + n_in * es].view(dt) for r in range(P)]
        base = P * per_in
        outs = [region[base + r * per_out:base + r * per_out + n_out * es].view(dt) for r in range(P)]
        for a, b in zip(ins, src):
            a.copy_(b)
        sets.append((ins, outs))
    op = nuna.reduce_scatter if kind == "rs" else nuna.all_gather
    ref = oracle.reduce_scatter(x_np) if kind == "rs" else oracle.all_gather(x_np)
    ok = True
    launches = {}
    for place in places:
        op(sets[0][0], sets[0][1], placement=place)
        launches[place] = nuna.last_launch()
        torch.cuda.synchronize()
        for d in range(P):
            g = sets[0][1][d].cpu()
            g = g.view(torch.int16).numpy().view(np.uint16) if es == 2 else g.numpy()
            ok = ok and np.array_equal(g, ref[d])
    graphs = {p: capture(torch, lambda i, p=p: op(sets[i % nsets][0], sets[i % nsets][1], placement=p), calls)
              for p in places}
    t = time_graphs(torch, graphs, calls, reps, warmup)
    alg_bytes = P * (n_in + n_out) * es
    out = {}
    for place in places:
        st = stats(t[place])
        out[place] = {"us": st, "gbps": alg_bytes / (st["median"] * 1e-6) / 1e9, "launch": launches[place]}
    del graphs, sets
    return alg_bytes, out, calls, ok


RS_AG_KIB = (16, 128, 1024, 4096, 8192)  # bytes per rank of the all-gather input / reduce-scatter output


# ---------------------------------------------------------------------------------------------- main line

def steps_per_graph(ksteps, step_bytes):
    """Steps captured per graph: the largest divisor of the timed step count that keeps one graph
    within GRAPH_BYTES, so that whole replays time exactly `ksteps` steps.  When that divisor is a
    small fraction of the target (a step count with few divisors), the graph holds the target and
    the last replay may run past `ksteps`."""
    target = max(1, math.ceil(GRAPH_BYTES / step_bytes))
    best = max(d for d in range(1, min(ksteps, target) + 1) if ksteps % d == 0)
    return best if best * 4 >= min(ksteps, target) else min(ksteps, target)


def steps_timed(nuna, torch, pool, args, xs, algo):
    """The timed region: K steps per placement mode, a step being one all-reduce (`algo`) of each input
    set in `xs`.  Steps are replayed from graphs of `steps_per_graph` steps (several GiB each); step i
    uses buffer region i mod R of the pool, R as many step regions as the pool holds.  With one region,
    each call is still cold: between two uses of a buffer set, the other sets of the step (and the
    set's own larger part) stream more bytes than the 256 MB Infinity Cache holds."""
    step_fp = sum(ar_footprint(len(x), x[0].size, 2) for x in xs)
    step_bytes = sum(2 * len(x) * x[0].size * 2 for x in xs)
    nsteps = steps_per_graph(args.steps, step_bytes)
    nreg = max(1, min(nsteps, pool.nbytes // step_fp))
    assert step_fp * nreg <= pool.nbytes
    pool.off = 0
    srcs = [[dev_copy_of(torch, a) for a in x] for x in xs]
    sets = [[ar_sets(torch, pool, x, 1, src)[0] for x, src in zip(xs, srcs)] for _ in range(nreg)]
    del srcs

    def step(i, place):
        for ins, outs in sets[i % nreg]:
            nuna.allreduce(ins, outs, algo=algo, placement=place)

    graphs = {p: capture(torch, lambda i, p=p: step(i, p), nsteps) for p in ("linear", "xcd")}
    reps = max(1, math.ceil(args.steps / nsteps))
    for _ in range(args.warmup):
        for g in graphs.values():
            g.replay()
    torch.cuda.synchronize()
    ev = {p: [] for p in graphs}
    names = list(graphs)
    for rep in range(reps):
        for p in (names if rep % 2 == 0 else names[::-1]):  # A/B then B/A
            g = graphs[p]
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            g.replay()
            b.record()
            b.synchronize()
            ev[p].append(a.elapsed_time(b))
    torch.cuda.synchronize()
    out = {}
    for p in graphs:
        ms = sum(ev[p]) / (reps * nsteps)
        out[p] = {"ms_per_step": ms, "gbps": step_bytes / (ms * 1e-3) / 1e9,
                  "replay_ms": stats(ev[p])}
    del graphs, sets
    torch.cuda.empty_cache()
    return step_bytes, reps * nsteps, nsteps, out


def launch_of(nuna, torch, x, algo, place):
    """Kernels and map of one call (nuna_last_launch) on scratch buffers."""
    ins = [dev_copy_of(torch, a) for a in x]
    outs = [torch.empty_like(t) for t in ins]
    nuna.allreduce(ins, outs, algo=algo, placement=place)
    info = nuna.last_launch()
    torch.cuda.synchronize()
    del ins, outs
    return info


def same_map(li_linear, li_xcd):
    """True when both placements ran identical launches: same kernels, same grid, the linear map."""
    return (li_linear["kernels"] == li_xcd["kernels"] and li_linear["grid"] == li_xcd["grid"]
            and li_linear["map"] == li_xcd["map"] == "linear")


def ar_sweep(nuna, torch, pool, args, cases, algos, max_calls=4096):
    """Per size and algorithm: µs per call (median, p10, p90, mean) and GB/s in both placements, from
    graph replays on cold buffers; bit-for-bit parity of both placements with the oracle; the launches
    each placement ran and whether they are the same map."""
    import oracle
    rows = []
    for label, x in cases:
        P, n = len(x), x[0].size
        es = 2 if x[0].dtype == np.uint16 else 4
        ref = oracle.allreduce(x)
        for algo in algos:
            ok = all(oracle_check_ar(nuna, torch, x, algo, p, ref) for p in ("linear", "xcd"))
            li = {p: launch_of(nuna, torch, x, algo, p) for p in ("linear", "xcd")}
            nbytes, res, calls = bench_allreduce(nuna, torch, pool, x, algo, args.reps, args.warmup,
                                                 max_calls=max_calls)
            rows.append({**label, "algo": algo, "bytes_per_rank": n * es, "alg_bytes": nbytes, "parity": ok,
                         "calls_per_graph": calls,
                         "xcd_us": {k: round(v, 3) for k, v in res["xcd"]["us"].items()},
                         "linear_us": {k: round(v, 3) for k, v in res["linear"]["us"].items()},
                         "xcd_gbps": round(res["xcd"]["gbps"], 1), "linear_gbps": round(res["linear"]["gbps"], 1),
                         "xcd_frac_hbm": round(res["xcd"]["gbps"] / HBM_PEAK_GBPS, 4),
                         "linear_over_xcd_time": round(res["linear"]["us"]["median"] / res["xcd"]["us"]["median"], 4),
                         "same_map": same_map(li["linear"], li["xcd"]),
                         "xcd_launch": {k: li["xcd"][k] for k in ("kernels", "map", "group_size", "grid", "threads",
                                                                   "vectors_per_thread")},
                         "linear_launch": {k: li["linear"][k] for k in ("kernels", "map", "grid")}})
            annotate_targets(rows[-1])
        del ref
    return rows


def prefill_sweep(nuna, torch, pool, args, xs):
    from paper_2608_00867_amd import workloads as wl
    cases = [({"tokens": T}, x) for T, x in zip(wl.PREFILL_TOKENS, xs)]
    return ar_sweep(nuna, torch, pool, args, cases, ["two_shot", "two_shot_two_kernels", "one_shot"])


def decode_sweep(nuna, torch, pool, args):
    from paper_2608_00867_amd import workloads as wl
    cases = [({"tokens": T}, wl.ar_bf16_decode(T)) for T in wl.DECODE_TOKENS]
    return ar_sweep(nuna, torch, pool, args, cases, ["auto"], max_calls=1024)


DOMINANT_JSON = os.path.join(ROOT, "profiles", "dominant_kernel.json")


def profiled_dominant():
    """The dominant kernel's traced average duration from the committed kernel-trace summary, or None
    when the kernel sources have changed since the trace was taken."""
    try:
        rec = json.load(open(DOMINANT_JSON))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_sha():
        return None
    return rec


def roofline_dominant(sweep):
    """Dominant kernel of the step: the fused two-shot all-reduce at T=4096 (64 MiB per rank), one
    kernel per call, XCD placement.  Its average duration per launch comes from HIP events around
    graph replays of back-to-back cold launches on the launching stream (the mean over the replays of
    replay time / launches).  The committed rocprofv3 kernel-trace average of the same kernel, from a
    run of this bench command on the same sources, is carried beside it."""
    row = [r for r in sweep if r["tokens"] == 4096 and r["algo"] == "two_shot"][0]
    us = row["xcd_us"]["mean"]
    achieved = row["alg_bytes"] / (us * 1e-6) / 1e9
    roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": measured_traffic(),
            "kernel": row["xcd_launch"]["kernels"], "grid_workgroups": row["xcd_launch"]["grid"],
            "threads": row["xcd_launch"]["threads"], "vectors_per_thread": row["xcd_launch"]["vectors_per_thread"],
            "workload": "two-shot all-reduce, P=8, [4096, 8192] bf16 per rank (64 MiB), XCD placement, cold",
            "alg_bytes_per_launch": row["alg_bytes"],
            "alg_bytes_rule": "2 * P * n * 2 B: each element read from P inputs and written to P outputs",
            "kernel_us_events_mean": us}
    prof = profiled_dominant()
    if prof is not None:
        pa = row["alg_bytes"] / (prof["avg_us"] * 1e-6) / 1e9
        roof["profile"] = {"kernel": prof["kernel"], "avg_us": prof["avg_us"], "dispatches": prof["dispatches"],
                           "frac": round(pa / HBM_PEAK_GBPS, 4), "source": prof["source"],
                           "events_over_profile": round(us / prof["avg_us"], 4)}
    return roof


def moe_dispatch_summary(nuna, torch, pool, args):
    """The MoE dispatch (8 ranks, 512 tokens x 7168 bf16 per rank, top-8 of 256 experts), cold."""
    recs = []
    a2a_case(nuna, torch, pool, args, recs.append, None, colds=(True,))
    r, routed = recs
    annotate_targets(r)
    r["routed"] = {"workload": routed["workload"], "parity": routed["parity"], "same_map": routed["same_map"],
                   "xcd_us": routed["xcd_us"], "linear_us": routed["linear_us"], "xcd_gbps": routed["xcd_gbps"],
                   "xcd_frac_hbm": routed["xcd_frac_hbm"],
                   "layout_xcd_over_routed_time": routed["layout_xcd_over_routed_time"]}
    r["parity"] = bool(r["parity"] and routed["parity"])
    return r


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(seconds, xs):
    """The oracle (single-threaded C) on the same step (one all-reduce of each input set in `xs`),
    repeated for about `seconds`; then the same oracle on all host cores, each thread running it on a
    contiguous element range of every rank buffer (each element still adds its ranks in ascending
    order, so the bits are the same; checked).  The oracle call releases the interpreter lock while it
    runs.  Inputs are already in host memory; their generation is not timed."""
    import concurrent.futures
    import oracle
    step_bytes = sum(2 * len(x) * x[0].size * 2 for x in xs)
    outs = [[np.empty_like(a) for a in x] for x in xs]
    oracle.get()

    def timed(run_step, budget):
        steps = 0
        t0 = time.perf_counter()
        while True:
            run_step()
            steps += 1
            el = time.perf_counter() - t0
            if el >= budget:
                return steps, el

    def single():
        for x, o in zip(xs, outs):
            oracle.allreduce(x, o)

    steps, el = timed(single, seconds)
    shape = "all-reduce bf16 P=8 at [T, 8192], T=" + ",".join(str(x[0].size // 8192) for x in xs)
    res = {"value": round(step_bytes * steps / el / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
           "sample": f"{steps} steps ({shape}) in {el:.1f} s, single thread, inputs resident in host memory; "
                     f"host reports {os.cpu_count()} CPUs",
           "cpu_model": cpu_model(), "ms_per_step": round(el / steps * 1e3, 3)}
    nthreads = max(1, min(os.cpu_count() or 1, 16))
    outs_mt = [[np.empty_like(a) for a in x] for x in xs]
    parts = []
    for x, o in zip(xs, outs_mt):
        n = x[0].size
        bounds = [n * k // nthreads for k in range(nthreads + 1)]
        parts += [([a[lo:hi] for a in x], [b[lo:hi] for b in o]) for lo, hi in zip(bounds, bounds[1:]) if hi > lo]
    with concurrent.futures.ThreadPoolExecutor(nthreads) as ex:
        def multi():
            list(ex.map(lambda io: oracle.allreduce(io[0], io[1]), parts))
        multi()
        same = all(np.array_equal(a, b) for o1, o2 in zip(outs, outs_mt) for a, b in zip(o1, o2))
        steps, el = timed(multi, seconds / 2)
    res["all_cores"] = {"value": round(step_bytes * steps / el / 1e9, 3), "unit": "GB/s", "threads": nthreads,
                        "same_bits_as_single": bool(same),
                        "sample": f"{steps} steps in {el:.1f} s, element ranges split over {nthreads} threads"}
    return res


# ---------------------------------------------------------------------------------------------- --full sweep

MOE_DECODE_TOKENS = (128, 16)  # decode-shaped MoE steps beside the 512-token shape
NO_SLOWER_TOL = 1.02   # XCD counts as no slower within 2 % of LINEAR's median
TARGET_FRAC = 0.70     # of the HBM peak, for messages of 4 MiB per rank and more
TARGET_MIN_BYTES = 4 << 20


def message_bytes_per_rank(rec):
    """Bytes one rank contributes to the collective: its all-reduce buffer, its reduce-scatter input
    (P shards), its all-gather output (P shards), or its MoE token rows."""
    if "bytes_per_rank" in rec:
        return rec["bytes_per_rank"]
    if "shard_bytes" in rec:
        return rec["shard_bytes"] * rec["P"]
    if "tokens_per_rank" in rec:
        return rec["tokens_per_rank"] * rec["hidden"] * 2
    return None


def annotate_targets(rec):
    """Per-record verdicts on the two comparative targets.  xcd_no_slower: XCD's median within 2 % of
    LINEAR's, or the two distributions overlap (XCD's p10 at or below LINEAR's p90).  meets_70pct: at
    4 MiB per rank and more, XCD reaches 70 % of the HBM peak."""
    lx, xx = rec.get("linear_us"), rec.get("xcd_us")
    if isinstance(lx, dict) and isinstance(xx, dict):
        rec["xcd_no_slower"] = bool(xx["median"] <= NO_SLOWER_TOL * lx["median"] or xx["p10"] <= lx["p90"])
    mb = message_bytes_per_rank(rec)
    if mb is not None and mb >= TARGET_MIN_BYTES and "xcd_frac_hbm" in rec:
        rec["meets_70pct"] = bool(rec["xcd_frac_hbm"] >= TARGET_FRAC)


def full_sweep(nuna, torch, pool, args):
    from paper_2608_00867_amd import workloads as wl
    os.makedirs(os.path.dirname(args.out), exist_ok=True)
    f = open(args.out, "w")

    def emit(rec):
        annotate_targets(rec)
        f.write(json.dumps(rec) + "\n")
        f.flush()
        print(json.dumps(rec), flush=True)

    def want(name):
        return args.only is None or name.startswith(args.only)

    def ar_case(name, make, algos):
        if not want(name):
            return
        x = make()
        P, n = len(x), x[0].size
        es = 2 if x[0].dtype == np.uint16 else 4
        for algo in algos:
            ok = all(oracle_check_ar(nuna, torch, x, algo, p) for p in ("linear", "xcd"))
            li = {p: launch_of(nuna, torch, x, algo, p) for p in ("linear", "xcd")}
            for cold in (True, False):
                nb, res, calls = bench_allreduce(nuna, torch, pool, x, algo, args.reps, args.warmup, cold=cold)
                emit({"workload": name, "P": P, "bytes_per_rank": n * es, "algo": algo,
                      "cache": "cold" if cold else "warm", "alg_bytes": nb, "calls_per_graph": calls,
                      "parity": ok, "same_map": same_map(li["linear"], li["xcd"]),
                      "xcd_kernels": li["xcd"]["kernels"], "xcd_map": li["xcd"]["map"],
                      **{f"{p}_us": {k: round(v, 3) for k, v in res[p]["us"].items()} for p in res},
                      **{f"{p}_gbps": round(res[p]["gbps"], 1) for p in res},
                      **{f"{p}_frac_hbm": round(res[p]["gbps"] / HBM_PEAK_GBPS, 4) for p in res},
                      "linear_over_xcd_time": round(res["linear"]["us"]["median"] / res["xcd"]["us"]["median"], 4)})

    ar_case("ar_f32_int_p8", wl.ar_f32_int, ["one_shot", "one_shot_split", "two_shot", "two_shot_two_kernels"])
    for T in wl.DECODE_TOKENS:
        ar_case(f"ar_bf16_decode_T{T}", lambda T=T: wl.ar_bf16_decode(T), ["one_shot", "one_shot_split", "two_shot",
                                                                           "two_shot_two_kernels"])
    for T in wl.PREFILL_TOKENS:
        ar_case(f"ar_bf16_prefill_T{T}", lambda T=T: wl.ar_bf16_prefill(T), ["two_shot", "two_shot_two_kernels",
                                                                             "one_shot"])
    for kib in wl.P64_KIB:
        ar_case(f"ar_bf16_p64_{kib}KiB", lambda kib=kib: wl.ar_bf16_p64(kib), ["one_shot", "one_shot_split",
                                                                             "two_shot"])
    if want("ar_bf16_decode_eager"):
        eager_case(nuna, torch, pool, args, emit)
    for kind in ("rs", "ag"):
        for kib in RS_AG_KIB:
            name = f"{kind}_bf16_p8_{kib}KiB"
            if not want(name):
                continue
            m = kib * 1024 // 2
            x = wl.normal_bf16(8, 8 * m if kind == "rs" else m, wl.seed_for(7 if kind == "rs" else 8, kib))
            for cold in (True, False):
                nb, res, calls, ok = bench_rs_ag(nuna, torch, pool, kind, x, args.reps, args.warmup, cold=cold)
                emit({"workload": name, "P": 8, "shard_bytes": kib * 1024, "algo": "standalone",
                      "cache": "cold" if cold else "warm", "alg_bytes": nb, "calls_per_graph": calls, "parity": ok,
                      "same_map": same_map(res["linear"]["launch"], res["xcd"]["launch"]),
                      "xcd_kernels": res["xcd"]["launch"]["kernels"], "xcd_map": res["xcd"]["launch"]["map"],
                      **{f"{p}_us": {k: round(v, 3) for k, v in res[p]["us"].items()} for p in res},
                      **{f"{p}_gbps": round(res[p]["gbps"], 1) for p in res},
                      **{f"{p}_frac_hbm": round(res[p]["gbps"] / HBM_PEAK_GBPS, 4) for p in res},
                      "linear_over_xcd_time": round(res["linear"]["us"]["median"] / res["xcd"]["us"]["median"], 4)})
    if want("a2a_moe_dispatch"):
        for T_tok in (None,) + MOE_DECODE_TOKENS:
            a2a_case(nuna, torch, pool, args, emit, T_tok)
    if want("a2a_moe_combine"):
        for T_tok in (None,) + MOE_DECODE_TOKENS:
            combine_case(nuna, torch, pool, args, emit, T_tok)
    size_sweep(nuna, torch, pool, args, emit, want)  # each size checks want() itself
    if want("copy_reference"):
        copy_case(nuna, torch, pool, args, emit)
    if want("ref_stream"):
        ref_stream_case(nuna, torch, pool, args, emit)
    if want("moe_step"):
        moe_step_case(nuna, torch, args, emit)
    if want("launch_floor"):
        launch_floor_case(nuna, torch, args, emit)
    f.close()


def a2a_case(nuna, torch, pool, args, emit, T_tokens=None, colds=(True, False)):
    """MoE dispatch at T_tokens per rank (default: the 512-token shape); decode-shaped token counts
    measure the latency regime."""
    import oracle
    from paper_2608_00867_amd import workloads as wl
    send_np, topk = wl.a2a_moe() if T_tokens is None else wl.a2a_moe(T=T_tokens)
    E = wl.MOE_EXPERTS
    lay = nuna.A2ALayout(topk, E).upload()
    rows = lay.recv_rows()
    P, T, H = len(send_np), send_np[0].shape[0], send_np[0].shape[1]
    cap = int(rows.max())
    rb = H * 2
    alg_bytes = int(P * T * rb + rows.sum() * rb)
    set_bytes = P * T * rb + P * cap * rb
    src = [dev_copy_of(torch, a.reshape(-1)) for a in send_np]
    for cold in colds:
        nsets = max(1, min(pool.nbytes // (set_bytes + 16 * ALIGN), math.ceil(COLD_SPAN / set_bytes) + 1)) \
            if cold else 1
        pool.off = 0
        sets = []
        for _ in range(nsets):
            send = [pool.take(T * rb)[:T * rb].view(torch.bfloat16).view(T, H) for _ in range(P)]
            recv = [pool.take(cap * rb)[:cap * rb].view(torch.bfloat16).view(cap, H) for _ in range(P)]
            for a, b in zip(send, src):
                a.view(-1).copy_(b)
            sets.append((send, recv))
        calls = max(nsets, calls_for(set_bytes))
        ref = oracle.all_to_all(send_np, topk, E)
        ok = True
        for p in ("linear", "xcd"):
            nuna.all_to_all(sets[0][0], sets[0][1], lay, placement=p)
            torch.cuda.synchronize()
            for d in range(P):
                g = sets[0][1][d][:int(rows[d])].cpu().view(torch.int16).numpy().view(np.uint16)
                ok = ok and np.array_equal(g, ref[d])
        graphs = {p: capture(torch, lambda i, p=p: nuna.all_to_all(sets[i % nsets][0], sets[i % nsets][1], lay,
                                                                    placement=p), calls)
                  for p in ("linear", "xcd")}
        t = time_graphs(torch, graphs, calls, args.reps, args.warmup)
        res = {p: stats(t[p]) for p in t}
        li = {}
        for p in ("linear", "xcd"):
            nuna.all_to_all(sets[0][0], sets[0][1], lay, placement=p)
            li[p] = nuna.last_launch()
        torch.cuda.synchronize()
        emit({"workload": "a2a_moe_dispatch_bf16_p8" + ("" if T_tokens is None else f"_T{T}"), "P": P,
              "same_map": same_map(li["linear"], li["xcd"]), "xcd_kernels": li["xcd"]["kernels"],
              "xcd_map": li["xcd"]["map"], "tokens_per_rank": T, "hidden": H,
              "rows_received": int(rows.sum()), "cache": "cold" if cold else "warm", "alg_bytes": alg_bytes,
              "calls_per_graph": calls, "parity": bool(ok),
              **{f"{p}_us": {k: round(v, 3) for k, v in res[p].items()} for p in res},
              **{f"{p}_gbps": round(alg_bytes / (res[p]["median"] * 1e-6) / 1e9, 1) for p in res},
              **{f"{p}_frac_hbm": round(alg_bytes / (res[p]["median"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
                 for p in res},
              "linear_over_xcd_time": round(res["linear"]["median"] / res["xcd"]["median"], 4)})
        del graphs
        # The allocation-free dispatch on the same buffers: the routing computed on the device from the
        # top-k table, one work item per (token, destination slot), a token's slots grouped on one XCD
        # with XCD placement (one kernel up to 256 tokens over all ranks, else a routing kernel and a
        # copy kernel).
        topk_dev = torch.from_numpy(np.ascontiguousarray(topk, dtype=np.int32)).cuda()
        rows_dev = torch.zeros(P + 1, dtype=torch.int64, device="cuda")
        ok_r = True
        for p in ("linear", "xcd"):
            for d in range(P):
                sets[0][1][d].zero_()
            nuna.all_to_all_routed(sets[0][0], sets[0][1], topk_dev, E, rows_dev, placement=p)
            torch.cuda.synchronize()
            ok_r = ok_r and rows_dev.cpu().tolist() == [int(r) for r in rows] + [0]
            for d in range(P):
                g = sets[0][1][d][:int(rows[d])].cpu().view(torch.int16).numpy().view(np.uint16)
                ok_r = ok_r and np.array_equal(g, ref[d])
        graphs = {p: capture(torch, lambda i, p=p: nuna.all_to_all_routed(sets[i % nsets][0], sets[i % nsets][1],
                                                                           topk_dev, E, rows_dev, placement=p), calls)
                  for p in ("linear", "xcd")}
        t = time_graphs(torch, graphs, calls, args.reps, args.warmup)
        rr = {p: stats(t[p]) for p in t}
        for p in ("linear", "xcd"):
            nuna.all_to_all_routed(sets[0][0], sets[0][1], topk_dev, E, rows_dev, placement=p)
            li[p] = nuna.last_launch()
        torch.cuda.synchronize()
        emit({"workload": "a2a_moe_dispatch_routed_bf16_p8" + ("" if T_tokens is None else f"_T{T}"), "P": P,
              "same_map": same_map(li["linear"], li["xcd"]), "xcd_kernels": li["xcd"]["kernels"],
              "xcd_map": li["xcd"]["map"], "tokens_per_rank": T, "hidden": H,
              "rows_received": int(rows.sum()), "cache": "cold" if cold else "warm", "alg_bytes": alg_bytes,
              "calls_per_graph": calls, "parity": bool(ok_r),
              **{f"{p}_us": {k: round(v, 3) for k, v in rr[p].items()} for p in rr},
              **{f"{p}_gbps": round(alg_bytes / (rr[p]["median"] * 1e-6) / 1e9, 1) for p in rr},
              **{f"{p}_frac_hbm": round(alg_bytes / (rr[p]["median"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
                 for p in rr},
              "linear_over_xcd_time": round(rr["linear"]["median"] / rr["xcd"]["median"], 4),
              "layout_xcd_over_routed_time": round(res["xcd"]["median"] / rr["xcd"]["median"], 4)})
        del graphs, sets
    lay.close()


EAGER_CALLS = 200


MOE_STEP_CALLS = 200


def moe_step_case(nuna, torch, args, emit):
    """One MoE dispatch per serving step with a new routing each step, the top-k table produced on the
    device (as a gate kernel leaves it), timed on the host per step including a device synchronize:
    - layout-driven: the table copied to the host, planned (nuna_a2a_layout_create), uploaded (which
      allocates and copies), dispatched, and the layout freed;
    - routed: the allocation-free dispatch reading the table where it is.
    Both give the same receive buffers (checked on the first step)."""
    from paper_2608_00867_amd import workloads as wl
    E, H = wl.MOE_EXPERTS, wl.HIDDEN_MOE
    for T_tok in MOE_DECODE_TOKENS:
        send_np, _ = wl.a2a_moe(T=T_tok)
        P, T = len(send_np), send_np[0].shape[0]
        tables = [wl.moe_routing(P, T, 8, E, wl.seed_for(4, 100 + i)) for i in range(16)]
        topk_dev = [torch.from_numpy(np.ascontiguousarray(t, dtype=np.int32)).cuda() for t in tables]
        send = [dev_copy_of(torch, a.reshape(-1)).view(torch.bfloat16).view(T, H) for a in send_np]
        cap = P * T
        recv_l = [torch.zeros((cap, H), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
        recv_r = [torch.zeros((cap, H), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
        rows_dev = torch.zeros(P + 1, dtype=torch.int64, device="cuda")

        def layout_step(i, out):
            host = topk_dev[i % len(topk_dev)].cpu().numpy()
            lay = nuna.A2ALayout(host, E).upload()
            nuna.all_to_all(send, out, lay, placement="xcd")
            torch.cuda.synchronize()
            rows = lay.recv_rows()
            lay.close()
            return rows

        def routed_step(i, out):
            nuna.all_to_all_routed(send, out, topk_dev[i % len(topk_dev)], E, rows_dev, placement="xcd")
            torch.cuda.synchronize()

        rows = layout_step(0, recv_l)
        routed_step(0, recv_r)
        ok = rows_dev.cpu().tolist() == [int(r) for r in rows] + [0] and all(
            torch.equal(recv_l[d][:int(rows[d])].view(torch.int16), recv_r[d][:int(rows[d])].view(torch.int16))
            for d in range(P))
        per = {"layout": [], "routed": []}
        for rep in range(MOE_STEP_CALLS):
            for kind in (("layout", "routed") if rep % 2 == 0 else ("routed", "layout")):
                t0 = time.perf_counter()
                if kind == "layout":
                    layout_step(rep, recv_l)
                else:
                    routed_step(rep, recv_r)
                per[kind].append((time.perf_counter() - t0) * 1e6)
        res = {k: stats(v) for k, v in per.items()}
        emit({"workload": f"moe_step_bf16_p8_T{T}", "P": P, "tokens_per_rank": T, "hidden": H, "parity": bool(ok),
              "steps": MOE_STEP_CALLS, "placement": "xcd",
              **{f"{k}_step_us": {q: round(v, 2) for q, v in r.items()} for k, r in res.items()},
              "layout_over_routed_step": round(res["layout"]["median"] / res["routed"]["median"], 2)})


def eager_case(nuna, torch, pool, args, emit):
    """The launch arm: decode all-reduces launched one at a time, each followed by a device
    synchronize, timed on the host (what a caller without graphs sees per call).  Compared with the
    graph-replay figure of the same size, the difference is the launch and synchronization cost."""
    from paper_2608_00867_amd import workloads as wl
    for T in wl.DECODE_TOKENS:
        x = wl.ar_bf16_decode(T)
        P, n = len(x), x[0].size
        fp = ar_footprint(P, n, 2)
        nsets = max(1, min(EAGER_CALLS, pool.nbytes // fp))
        pool.off = 0
        sets = ar_sets(torch, pool, x, nsets)
        res = {}
        for place in ("linear", "xcd"):
            for i in range(10):
                nuna.allreduce(sets[i % nsets][0], sets[i % nsets][1], algo="auto", placement=place)
            torch.cuda.synchronize()
        per = {"linear": [], "xcd": []}
        for rep in range(EAGER_CALLS):
            for place in (("linear", "xcd") if rep % 2 == 0 else ("xcd", "linear")):
                ins, outs = sets[rep % nsets]
                t0 = time.perf_counter()
                nuna.allreduce(ins, outs, algo="auto", placement=place)
                torch.cuda.synchronize()
                per[place].append((time.perf_counter() - t0) * 1e6)
        for place in per:
            res[place] = stats(per[place])
        # Host cost of one call alone: back-to-back enqueues (Python binding + C ABI + launch), no sync.
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(EAGER_CALLS):
            nuna.allreduce(sets[i % nsets][0], sets[i % nsets][1], algo="auto", placement="xcd")
        enqueue_us = (time.perf_counter() - t0) * 1e6 / EAGER_CALLS
        torch.cuda.synchronize()
        # The same with the call prepared once (no per-call Python checks or marshalling).
        calls = [nuna.prepare_allreduce(ins, outs, algo="auto", placement="xcd") for ins, outs in sets[:16]]
        handle = torch.cuda.current_stream().cuda_stream
        t0 = time.perf_counter()
        for i in range(EAGER_CALLS):
            calls[i % len(calls)](handle)
        prepared_us = (time.perf_counter() - t0) * 1e6 / EAGER_CALLS
        torch.cuda.synchronize()
        emit({"workload": "ar_bf16_decode_eager", "P": P, "tokens": T, "bytes_per_rank": n * 2,
              "timing": "host clock per eager call + device synchronize", "calls": EAGER_CALLS,
              **{f"{p}_us": {k: round(v, 3) for k, v in res[p].items()} for p in res},
              "enqueue_only_us": round(enqueue_us, 3), "prepared_enqueue_only_us": round(prepared_us, 3)})
        del sets


def combine_case(nuna, torch, pool, args, emit, T_tokens=None):
    """MoE combine at the dispatch's shape: every received row comes back as a result row and is
    summed into its token (reads: all result rows; writes: every token row once), unweighted and with
    one gate weight per (token, destination rank)."""
    import oracle
    from paper_2608_00867_amd import workloads as wl
    _, topk = wl.a2a_moe() if T_tokens is None else wl.a2a_moe(T=T_tokens)
    E, H = wl.MOE_EXPERTS, wl.HIDDEN_MOE
    P, T = int(topk.shape[0]), int(topk.shape[1])
    lay = nuna.A2ALayout(topk, E).upload()
    rows = lay.recv_rows()
    cap = int(rows.max())
    rb = H * 2
    set_bytes = P * cap * rb + P * T * rb
    y_np = wl.result_rows(rows, H, np.uint16, wl.seed_for(4, 7))
    src = [dev_copy_of(torch, a.reshape(-1)) for a in y_np]
    w_np = wl.gate_weights(topk, E, wl.seed_for(4, 8))
    w_dev = torch.from_numpy(w_np).cuda()
    for weighted in (False, True):
        ref = oracle.combine(y_np, topk, E, w_np if weighted else None)
        wt = w_dev if weighted else None
        alg_bytes = int(rows.sum() * rb + P * T * rb + (w_np.nbytes if weighted else 0))
        name = ("a2a_moe_combine_weighted_bf16_p8" if weighted else "a2a_moe_combine_bf16_p8") + \
            ("" if T_tokens is None else f"_T{T}")
        for cold in (True, False):
            nsets = max(1, min(pool.nbytes // (set_bytes + 16 * ALIGN), math.ceil(COLD_SPAN / set_bytes) + 1)) \
                if cold else 1
            pool.off = 0
            sets = []
            for _ in range(nsets):
                y = [pool.take(cap * rb)[:cap * rb].view(torch.bfloat16).view(cap, H) for _ in range(P)]
                out = [pool.take(T * rb)[:T * rb].view(torch.bfloat16).view(T, H) for _ in range(P)]
                for d in range(P):
                    y[d][:int(rows[d])].view(-1).copy_(src[d])
                sets.append((y, out))
            calls = max(nsets, calls_for(set_bytes))
            ok = True
            li = {}
            for p in ("linear", "xcd"):
                nuna.all_to_all_combine(sets[0][0], sets[0][1], lay, placement=p, weights=wt)
                li[p] = nuna.last_launch()
                torch.cuda.synchronize()
                for d in range(P):
                    g = sets[0][1][d].cpu().view(torch.int16).numpy().view(np.uint16)
                    ok = ok and np.array_equal(g, ref[d])
            graphs = {p: capture(torch, lambda i, p=p: nuna.all_to_all_combine(
                sets[i % nsets][0], sets[i % nsets][1], lay, placement=p, weights=wt), calls)
                for p in ("linear", "xcd")}
            t = time_graphs(torch, graphs, calls, args.reps, args.warmup)
            res = {p: stats(t[p]) for p in t}
            emit({"workload": name, "P": P, "tokens_per_rank": T, "hidden": H,
                  "result_rows": int(rows.sum()), "cache": "cold" if cold else "warm", "alg_bytes": alg_bytes,
                  "calls_per_graph": calls, "parity": bool(ok), "same_map": same_map(li["linear"], li["xcd"]),
                  "xcd_kernels": li["xcd"]["kernels"], "xcd_map": li["xcd"]["map"],
                  **{f"{p}_us": {k: round(v, 3) for k, v in res[p].items()} for p in res},
                  **{f"{p}_gbps": round(alg_bytes / (res[p]["median"] * 1e-6) / 1e9, 1) for p in res},
                  **{f"{p}_frac_hbm": round(alg_bytes / (res[p]["median"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
                     for p in res},
                  "linear_over_xcd_time": round(res["linear"]["median"] / res["xcd"]["median"], 4)})
            del graphs, sets
    lay.close()


def launch_floor_case(nuna, torch, args, emit):
    """Per-call time of the library's smallest kernel (the dispatch probe: one argument load and one
    4-byte store per workgroup) in the same graph replay as the collectives: the floor that launch
    and completion put under every call."""
    calls = 2048
    for G in (1, 256):
        xcc = torch.empty(G, dtype=torch.int32, device="cuda")

        def fn(i, G=G, xcc=xcc):
            st = nuna.lib().nuna_probe_xcc(G, xcc.data_ptr(), None, torch.cuda.current_stream().cuda_stream)
            assert st == 0, nuna.last_error()
        g = {"probe": capture(torch, fn, calls)}
        t = stats(time_graphs(torch, g, calls, args.reps, args.warmup)["probe"])
        emit({"workload": "launch_floor", "kernel": "k_probe_xcc", "workgroups": G, "threads_per_workgroup": 64,
              "calls_per_graph": calls, "us": {k: round(v, 3) for k, v in t.items()}})


def copy_case(nuna, torch, pool, args, emit):
    """Plain streaming copy: the bandwidth ceiling a read+write kernel reaches on this GPU.  32, 128
    and 512 MiB copied move what the prefill all-reduces move at 4, 16 and 64 MiB per rank."""
    for mib in (16, 32, 64, 128, 256, 512):
        nb = mib << 20
        nsets = max(1, min(pool.nbytes // (2 * nb), math.ceil(COLD_SPAN / (2 * nb))))
        pool.off = 0
        pairs = [(pool.take(nb), pool.take(nb)) for _ in range(nsets)]
        calls = max(nsets, calls_for(2 * nb))
        s = torch.cuda.current_stream()

        def fn(i):
            a, b = pairs[i % nsets]
            nuna.lib().nuna_copy(b.data_ptr(), a.data_ptr(), nb, torch.cuda.current_stream().cuda_stream)

        g = {"copy": capture(torch, fn, calls)}
        t = stats(time_graphs(torch, g, calls, args.reps, args.warmup)["copy"])
        emit({"workload": "copy_reference", "bytes": nb, "cache": "cold", "us": {k: round(v, 3) for k, v in t.items()},
              "gbps_read_plus_write": round(2 * nb / (t["median"] * 1e-6) / 1e9, 1)})
        del g, pairs
        del s


SIZE_SWEEP_AR_KIB = (16, 64, 256, 1024, 4096, 16384, 65536, 131072)  # bytes per rank of the all-reduce
SIZE_SWEEP_AG_KIB = (2, 8, 32, 128, 512, 2048, 8192, 16384)            # shard bytes of the all-gather (x8 out)


def size_sweep(nuna, torch, pool, args, emit, want):
    """Latency and HBM GB/s against message size, both placements, cold, 8 ranks of bf16: the all-reduce
    (AUTO, the destination-split one-shot and the two-shot) from 16 KiB to 128 MiB per rank, and the
    all-gather from 2 KiB to 16 MiB shards (16 KiB to 128 MiB received per rank), in steps of 4x."""
    import oracle
    from paper_2608_00867_amd import workloads as wl
    for kib in SIZE_SWEEP_AR_KIB:
        name = f"size_ar_bf16_p8_{kib}KiB"
        if not want(name):
            continue
        n = kib * 1024 // 2
        x = wl.normal_bf16(8, n, wl.seed_for(11, kib))
        ref = oracle.allreduce(x)
        for algo in ("auto", "one_shot_split", "two_shot"):
            ok = all(oracle_check_ar(nuna, torch, x, algo, p, ref) for p in ("linear", "xcd"))
            li = {p: launch_of(nuna, torch, x, algo, p) for p in ("linear", "xcd")}
            nb, res, calls = bench_allreduce(nuna, torch, pool, x, algo, args.reps, args.warmup)
            emit({"workload": name, "P": 8, "bytes_per_rank": kib * 1024, "algo": algo, "cache": "cold",
                  "alg_bytes": nb, "calls_per_graph": calls, "parity": ok,
                  "same_map": same_map(li["linear"], li["xcd"]),
                  "xcd_kernels": li["xcd"]["kernels"], "xcd_map": li["xcd"]["map"],
                  **{f"{p}_us": {k: round(v, 3) for k, v in res[p]["us"].items()} for p in res},
                  **{f"{p}_gbps": round(res[p]["gbps"], 1) for p in res},
                  **{f"{p}_frac_hbm": round(res[p]["gbps"] / HBM_PEAK_GBPS, 4) for p in res},
                  "linear_over_xcd_time": round(res["linear"]["us"]["median"] / res["xcd"]["us"]["median"], 4)})
        del x, ref
    for kib in SIZE_SWEEP_AG_KIB:
        name = f"size_ag_bf16_p8_{kib}KiB"
        if not want(name):
            continue
        m = kib * 1024 // 2
        x = wl.normal_bf16(8, m, wl.seed_for(12, kib))
        nb, res, calls, ok = bench_rs_ag(nuna, torch, pool, "ag", x, args.reps, args.warmup)
        emit({"workload": name, "P": 8, "shard_bytes": kib * 1024, "bytes_per_rank": 8 * kib * 1024,
              "algo": "standalone", "cache": "cold", "alg_bytes": nb, "calls_per_graph": calls, "parity": ok,
              "same_map": same_map(res["linear"]["launch"], res["xcd"]["launch"]),
              "xcd_kernels": res["xcd"]["launch"]["kernels"], "xcd_map": res["xcd"]["launch"]["map"],
              **{f"{p}_us": {k: round(v, 3) for k, v in res[p]["us"].items()} for p in res},
              **{f"{p}_gbps": round(res[p]["gbps"], 1) for p in res},
              **{f"{p}_frac_hbm": round(res[p]["gbps"] / HBM_PEAK_GBPS, 4) for p in res},
              "linear_over_xcd_time": round(res["linear"]["us"]["median"] / res["xcd"]["us"]["median"], 4)})
        del x


REF_STREAMS = (("read", 1, 512), ("read", 8, 64), ("write", 1, 512), ("write", 8, 64), ("copy", 1, 512),
               ("copy", 2, 256), ("copy", 4, 128), ("copy", 8, 64))  # (kind, buffers, MiB per buffer)


def ref_stream_case(nuna, torch, pool, args, emit):
    """The plain access patterns that bound the collectives (nuna_ref_stream), cold, one 4 KiB item of every
    buffer per workgroup: reads only, writes only, and copies of 1 to 8 buffers at once.  The 8-buffer rows
    have the 8-rank all-reduce's streams at 64 MiB per rank (8 inputs and 8 outputs at one offset) without
    the reduction; the 1-buffer rows, the same bytes in one stream."""
    for kind, n, mib in REF_STREAMS:
        nb = mib << 20
        items = (nb + 4095) // 4096
        per = {"read": n * nb + items * 16, "write": n * nb, "copy": 2 * n * nb}[kind]
        moved = {"read": n * nb, "write": n * nb, "copy": 2 * n * nb}[kind]
        nsets = max(1, min(pool.nbytes // per, math.ceil(COLD_SPAN / per)))
        pool.off = 0
        sets = []
        for _ in range(nsets):
            region = pool.take(per)
            u8 = region.view(torch.uint8)
            if kind == "read":
                srcs = [u8[r * nb:(r + 1) * nb] for r in range(n)]
                dsts = [u8[n * nb:n * nb + items * 16]]
            elif kind == "write":
                srcs, dsts = None, [u8[r * nb:(r + 1) * nb] for r in range(n)]
            else:
                srcs = [u8[r * nb:(r + 1) * nb] for r in range(n)]
                dsts = [u8[(n + r) * nb:(n + r + 1) * nb] for r in range(n)]
            sets.append((srcs, dsts))
        calls = max(nsets, calls_for(moved))

        def fn(i):
            srcs, dsts = sets[i % nsets]
            nuna.ref_stream(kind, srcs, dsts)

        g = {"ref": capture(torch, fn, calls)}
        t = stats(time_graphs(torch, g, calls, args.reps, args.warmup)["ref"])
        gbps = moved / (t["median"] * 1e-6) / 1e9
        emit({"workload": "ref_stream", "kind": kind, "buffers": n, "bytes_per_buffer": nb, "bytes_moved": moved,
              "cache": "cold", "calls_per_graph": calls, "us": {k: round(v, 3) for k, v in t.items()},
              "gbps": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)})
        del g, sets


# ---------------------------------------------------------------------------------------------- --interference

INTERF_M = 2560                      # M = N: about 100 output tiles of 256 x 256
INTERF_K = (0, 2048, 8192, 32768, 131072)
INTERF_AG_ELEMS = 65536              # bf16 per rank: 128 KiB in, 1 MiB out per rank with P = 8
INTERF_AR_TOKENS = 64                # split all-reduce: [64, 8192] bf16 per rank (1 MiB)
INTERF_MOE_TOKENS = 128              # MoE dispatch: 128 tokens x 7168 bf16 per rank, top-8 of 256 experts
INTERF_CALLS = 200
INTERF_MAX_SLOWDOWN = 30.0           # the GEMM window covers the collective's graph even this much slower


def interference_cases(wl, oracle):
    """The collectives run beside the GEMM.  The all-gather is the paper's setup (1 MB per output);
    at that size its default map is the same in both placements.  The split all-reduce (each chunk's
    8 destination groups are separate work items) and the MoE dispatch (the copies of a token row
    form one group) are maps the placement changes.  Inputs and outputs are flat bf16 buffers; `ref`
    holds each rank's expected leading elements (the dispatch's receive buffers have spare rows,
    which must stay untouched)."""
    P, m = 8, INTERF_AG_ELEMS
    x = wl.normal_bf16(P, m, wl.seed_for(6))
    yield {"workload": "all_gather_bf16_p8_1MiB_beside_gemm", "ins": x, "out_elems": P * m,
           "ref": oracle.all_gather(x),
           "call": lambda nuna, ins, outs, p: nuna.all_gather(ins, outs, placement=p)}
    x = wl.ar_bf16_decode(INTERF_AR_TOKENS)
    yield {"workload": f"allreduce_split_bf16_p8_T{INTERF_AR_TOKENS}_beside_gemm", "ins": x,
           "out_elems": x[0].size, "ref": oracle.allreduce(x),
           "call": lambda nuna, ins, outs, p: nuna.allreduce(ins, outs, algo="one_shot_split", placement=p)}
    T, H, E = INTERF_MOE_TOKENS, wl.HIDDEN_MOE, wl.MOE_EXPERTS
    send, topk = wl.a2a_moe(T=T)
    ref = oracle.all_to_all(send, topk, E)
    cap = max(r.shape[0] for r in ref)
    held = {}

    def dispatch(nuna, ins, outs, p):
        nuna.all_to_all([t.view(T, H) for t in ins], [o.view(cap, H) for o in outs], held["layout"], placement=p)

    yield {"workload": f"a2a_moe_dispatch_bf16_p8_T{T}_beside_gemm", "ins": [a.ravel() for a in send],
           "out_elems": cap * H, "ref": [r.ravel() for r in ref], "call": dispatch,
           "prepare": lambda nuna: held.update(layout=nuna.A2ALayout(topk, E).upload()),
           "release": lambda: held.pop("layout").close()}


def interference(nuna, torch, args):
    """Each collective beside an unrelated GEMM (the paper's concurrent-GEMM experiment): per K, the
    collective's per-call time from a graph of INTERF_CALLS calls replayed on its own stream while
    GEMMs keep the other stream busy for the whole window; LINEAR and XCD interleaved A/B.  Two cache
    states: warm (one buffer set used over and over) and cold (the calls rotate over buffer sets
    whose total exceeds the Infinity Cache).  Both streams have the default priority.  After the timed
    runs every output is checked bit for bit against the oracle."""
    import oracle
    from paper_2608_00867_amd import workloads as wl
    os.makedirs(os.path.dirname(args.out), exist_ok=True)
    f = open(args.out, "w")
    s_coll, s_gemm = torch.cuda.Stream(), torch.cuda.Stream()
    for case in interference_cases(wl, oracle):
        x, ref, call = case["ins"], case["ref"], case["call"]
        P, m, mo = len(x), x[0].size, case["out_elems"]
        if "prepare" in case:
            case["prepare"](nuna)
        src = [dev_copy_of(torch, a) for a in x]
        set_bytes = P * (m + mo) * 2
        for cache in ("warm", "cold"):
            nsets = 1 if cache == "warm" else math.ceil(COLD_SPAN / set_bytes) + 1
            # Both placements run on the same buffers, so that only the map differs between them.
            sets = []
            for _ in range(nsets):
                ins = [torch.empty(m, dtype=torch.bfloat16, device="cuda") for _ in range(P)]
                for a, b in zip(ins, src):
                    a.copy_(b)
                sets.append((ins, [torch.empty(mo, dtype=torch.bfloat16, device="cuda") for _ in range(P)]))
            graphs = {}
            for p in ("linear", "xcd"):
                with torch.cuda.stream(s_coll):
                    call(nuna, sets[0][0], sets[0][1], p)
                torch.cuda.synchronize()
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=s_coll):
                    for i in range(INTERF_CALLS):
                        ins, outs = sets[i % nsets]
                        call(nuna, ins, outs, p)
                graphs[p] = g
            torch.cuda.synchronize()
            alone = {}
            for K in INTERF_K:
                gemm_us = None
                if K:
                    a = torch.randn(INTERF_M, K, dtype=torch.bfloat16, device="cuda")
                    b = torch.randn(K, INTERF_M, dtype=torch.bfloat16, device="cuda")
                    c = torch.empty(INTERF_M, INTERF_M, dtype=torch.bfloat16, device="cuda")
                    with torch.cuda.stream(s_gemm):
                        for _ in range(2):
                            torch.matmul(a, b, out=c)
                        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                        e0.record()
                        for _ in range(5):
                            torch.matmul(a, b, out=c)
                        e1.record()
                    torch.cuda.synchronize()
                    gemm_us = e0.elapsed_time(e1) * 1e3 / 5
                    # us: bound on the graph's duration beside the GEMM, from the slower mode alone
                    window = INTERF_MAX_SLOWDOWN * INTERF_CALLS * max(alone.values()) + 50.0
                    ngemm = max(2, math.ceil(window / gemm_us))
                res = {p: [] for p in graphs}
                gemm_conc = []
                covered = True
                for rep in range(args.reps):
                    for p in (("linear", "xcd") if rep % 2 == 0 else ("xcd", "linear")):
                        torch.cuda.synchronize()
                        if K:
                            g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                            with torch.cuda.stream(s_gemm):
                                g0.record()
                                for _ in range(ngemm):
                                    torch.matmul(a, b, out=c)
                                g1.record()
                        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                        with torch.cuda.stream(s_coll):
                            c0.record()
                            graphs[p].replay()
                            c1.record()
                        torch.cuda.synchronize()
                        res[p].append(c0.elapsed_time(c1) * 1e3 / INTERF_CALLS)
                        if K:
                            gemm_conc.append(g0.elapsed_time(g1) * 1e3 / ngemm)
                            # the GEMMs started first; they must also still run when the last call ends
                            covered = covered and g0.elapsed_time(c1) <= g0.elapsed_time(g1)
                ok = True
                for p in graphs:
                    for o in range(min(2, nsets)):
                        for d in range(P):
                            sets[o][1][d].zero_()
                    torch.cuda.synchronize()
                    graphs[p].replay()
                    torch.cuda.synchronize()
                    for _, outs in sets[:2]:
                        for d in range(P):
                            got = outs[d].cpu().view(torch.int16).numpy().view(np.uint16)
                            n_d = ref[d].size
                            ok = ok and np.array_equal(got[:n_d], ref[d]) and not got[n_d:].any()
                st = {p: stats(res[p]) for p in res}
                if not K:
                    alone = {p: st[p]["median"] for p in st}
                rec = {"workload": case["workload"], "cache": cache, "gemm_m": INTERF_M,
                       "gemm_n": INTERF_M, "gemm_k": K,
                       "gemm_us_alone": None if gemm_us is None else round(gemm_us, 1),
                       "gemm_us_beside_collective": round(statistics.median(gemm_conc), 1) if gemm_conc else None,
                       "calls": INTERF_CALLS, "buffer_sets": nsets, "parity": bool(ok),
                       "gemm_covers_collective": bool(covered) if K else None,
                       **{f"{p}_us": {k: round(v, 3) for k, v in st[p].items()} for p in st},
                       **{f"{p}_slowdown": round(st[p]["median"] / alone[p], 3) for p in st},
                       "linear_over_xcd_time": round(st["linear"]["median"] / st["xcd"]["median"], 4)}
                f.write(json.dumps(rec) + "\n")
                f.flush()
                print(json.dumps(rec), flush=True)
                if K:
                    del a, b, c
            del graphs, sets
            torch.cuda.empty_cache()
        if "release" in case:
            case["release"]()
    f.close()


# ---------------------------------------------------------------------------------------------- --affinity

def affinity(nuna, torch, pool):
    """Memory-side NUNA across an all-reduce's buffers.  For the first buffer set of a layout, every
    8 KiB block's near die is probed twice (from XCD 0 and XCD 4, caches evicted between passes);
    each rank buffer's labels are compared with rank 0's input at equal offsets."""
    for T in (64, 1024):
        P, n = 8, T * 8192
        fp = ar_footprint(P, n, 2)
        pool.off = 0
        region = pool.take(fp)
        per = (n * 2 + ALIGN - 1) // ALIGN * ALIGN
        words = region.view(torch.int32)
        passes = [nuna.memory_affinity(words, stride=8192, xcds=(0, 4))[1].cpu().numpy() for _ in range(2)]
        nb = per // 8192
        lab = np.stack([passes[0][v * nb:(v + 1) * nb] for v in range(2 * P)])
        maj = (lab.mean(axis=0) >= 0.5).astype(int)
        print(json.dumps({"layout": f"all-reduce bf16 P=8 [{T},8192]: 16 buffers of {per >> 10} KiB",
                          "blocks_per_buffer": nb,
                          "probe_repeatability": round(float(np.mean(passes[0] == passes[1])), 3),
                          "agreement_with_rank0_input": [round(float(np.mean(lab[v] == lab[0])), 3)
                                                         for v in range(2 * P)],
                          "near_fraction_on_majority_die": round(float(np.mean(lab == maj[None, :])), 3)}),
              flush=True)


CU_PROBE_BYTES = 64 << 20


def cu_affinity(nuna, torch):
    """The paper's latency profiling over every compute unit and target address (Sec. 3.2), on one GPU:
    every CU of every XCD times one cold load per 8 KiB block of a 64 MiB buffer.  Each block is labelled
    by the XCD group (0-3 or 4-7) whose CUs load it faster on average; the summary gives, per XCD, the
    CUs reached, the spread of the per-CU median latencies to near and to far blocks, how often a single
    CU's own near/far call agrees with the block's label, and the spread over addresses."""
    buf = torch.zeros(CU_PROBE_BYTES // 4, dtype=torch.int32, device="cuda")
    res = nuna.cu_latency_map(buf, stride=8192)
    lat = {x: res[x][0].numpy() for x in res}
    group_a = np.concatenate([lat[x] for x in range(4)]).mean(axis=0)
    group_b = np.concatenate([lat[x] for x in range(4, 8)]).mean(axis=0)
    near_a = group_a < group_b  # block is near XCDs 0-3
    rows = []
    for x in sorted(lat):
        L = lat[x]
        near = near_a if x < 4 else ~near_a
        med_near = np.median(L[:, near], axis=1)
        med_far = np.median(L[:, ~near], axis=1)
        thr = (med_near + med_far)[:, None] / 2
        own = L < thr  # each CU's own near call per block
        agree = np.mean(own == near[None, :], axis=1)
        q = np.percentile(L, [10, 50, 90], axis=1)
        rows.append({"xcd": x, "cus_seen": int(res[x][2]), "cus_probed": int(L.shape[0]),
                     "distinct_cu_keys": int(np.unique(res[x][1].numpy()).size),
                     "near_median_cycles": [round(float(med_near.min()), 1), round(float(np.median(med_near)), 1),
                                            round(float(med_near.max()), 1)],
                     "far_median_cycles": [round(float(med_far.min()), 1), round(float(np.median(med_far)), 1),
                                           round(float(med_far.max()), 1)],
                     "cu_spread_near": round(float(med_near.max() / med_near.min()), 3),
                     "far_over_near": round(float(np.median(med_far) / np.median(med_near)), 3),
                     "own_call_agreement": [round(float(agree.min()), 3), round(float(np.median(agree)), 3)],
                     "address_p10_p50_p90": [round(float(np.median(q[0])), 1), round(float(np.median(q[1])), 1),
                                             round(float(np.median(q[2])), 1)],
                     "address_max_over_min": round(float(np.median(L.max(axis=1) / np.maximum(L.min(axis=1), 1))), 3)})
    summary = {"buffer_bytes": CU_PROBE_BYTES, "block_bytes": 8192, "blocks": int(near_a.size),
               "near_group_0_3_fraction": round(float(near_a.mean()), 3), "per_xcd": rows}
    print(json.dumps({"cu_affinity": summary}), flush=True)
    print("\n| XCD | CUs probed (distinct) | near: per-CU median cycles min / median / max | far: min / median / max | "
          "CU spread (near, max/min) | far / near | CU's own near call agrees with the block label (min, median) | "
          "one CU over addresses: p10 / p50 / p90 | max / min over addresses |")
    print("|---|---|---|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['xcd']} | {r['cus_probed']} ({r['distinct_cu_keys']}) | "
              f"{' / '.join(str(v) for v in r['near_median_cycles'])} | "
              f"{' / '.join(str(v) for v in r['far_median_cycles'])} | {r['cu_spread_near']} | {r['far_over_near']} | "
              f"{r['own_call_agreement'][0]}, {r['own_call_agreement'][1]} | "
              f"{' / '.join(str(v) for v in r['address_p10_p50_p90'])} | {r['address_max_over_min']} |")


# ---------------------------------------------------------------------------------------------- --profile

PROFILE_COPY_BYTES = 64 << 20


PROFILE_PHASE_TOKENS = 256  # the two-kernel two-shot traced per phase (4 MiB per rank)


def profile_run(nuna, torch, pool, n, place="xcd"):
    """Short eager run for rocprofv3 counter passes, in dispatch order: the dominant kernel (fused
    two-shot, [4096, 8192] bf16 per rank, XCD) on cold buffers; the reference copy of
    PROFILE_COPY_BYTES (the calibration kernel for the traffic counters); the two-kernel two-shot at
    [256, 8192] (its reduce-scatter and all-gather phases); then the kernels whose map the placement
    changes (split all-reduce at decode T=64, MoE dispatch; the combine too) in placement `place`."""
    from paper_2608_00867_amd import workloads as wl

    def run(x, algo, plc):
        pool.off = 0
        sets = ar_sets(torch, pool, x, max(1, min(n, pool.nbytes // ar_footprint(8, x[0].size, 2))))
        torch.cuda.synchronize()
        for i in range(n):
            ins, outs = sets[i % len(sets)]
            nuna.allreduce(ins, outs, algo=algo, placement=plc)
        torch.cuda.synchronize()
        del sets

    xd = wl.ar_bf16_prefill(4096)
    run(xd, "two_shot", "xcd")
    del xd
    pool.off = 0
    a = pool.take(PROFILE_COPY_BYTES)
    b = pool.take(PROFILE_COPY_BYTES)
    for _ in range(n):
        nuna.copy(b, a)
    torch.cuda.synchronize()
    run(wl.ar_bf16_prefill(PROFILE_PHASE_TOKENS), "two_shot_two_kernels", "xcd")
    # The split all-reduce: 8 destination groups per chunk, the placement under study.
    run(wl.ar_bf16_decode(64), "one_shot_split", place)
    moe = profile_moe(nuna, torch, pool, n, place)
    print(json.dumps({"profile": {"place": place, "dominant_launches": n, "dominant_alg_bytes": DOMINANT_ALG_BYTES,
                                  "copy_launches": n, "copy_bytes": PROFILE_COPY_BYTES, **moe}}), flush=True)


def moe_alg_bytes():
    """Algorithmic bytes of one MoE dispatch and of one combine at the full shape (equal: every
    received row is read or written once, every token row written or read once)."""
    import oracle
    from paper_2608_00867_amd import workloads as wl
    _, topk = wl.a2a_moe()
    rows = oracle.a2a_counts(topk, wl.MOE_EXPERTS)
    rb = wl.HIDDEN_MOE * 2
    return int(rows.sum() * rb + topk.shape[0] * topk.shape[1] * rb)


def route_count_bytes():
    """Algorithmic bytes of the routed dispatch's routing kernel at the MoE shape: the int32 top-k
    table read once, then min(k, P) 4-byte records per token and the P x P counts and P invalid-entry
    counts written."""
    from paper_2608_00867_amd import workloads as wl
    _, topk = wl.a2a_moe()
    P, T, k = (int(v) for v in topk.shape)
    return 4 * P * T * k + 4 * P * T * min(k, P) + 4 * P * P + 4 * P


def profile_moe(nuna, torch, pool, n, place="xcd"):
    """`n` dispatches, `n` combines, then `n` allocation-free (routed) dispatches at the MoE shape,
    rotating over buffer sets that together exceed the caches."""
    from paper_2608_00867_amd import workloads as wl
    send_np, topk = wl.a2a_moe()
    E, H = wl.MOE_EXPERTS, wl.HIDDEN_MOE
    P, T = int(topk.shape[0]), int(topk.shape[1])
    lay = nuna.A2ALayout(topk, E).upload()
    cap = int(lay.recv_rows().max())
    rb = H * 2
    set_bytes = P * T * rb + P * cap * rb
    nsets = max(1, min(3, pool.nbytes // (set_bytes + 16 * ALIGN)))
    pool.off = 0
    sets = []
    for _ in range(nsets):
        tok = [pool.take(T * rb)[:T * rb].view(torch.bfloat16).view(T, H) for _ in range(P)]
        rec = [pool.take(cap * rb)[:cap * rb].view(torch.bfloat16).view(cap, H) for _ in range(P)]
        for t, a in zip(tok, send_np):
            t.copy_(dev_copy_of(torch, a))
        sets.append((tok, rec))
    torch.cuda.synchronize()
    for i in range(n):
        tok, rec = sets[i % nsets]
        nuna.all_to_all(tok, rec, lay, placement=place)
    torch.cuda.synchronize()
    for i in range(n):
        tok, rec = sets[i % nsets]
        nuna.all_to_all_combine(rec, tok, lay, placement=place)
    torch.cuda.synchronize()
    topk_dev = torch.from_numpy(np.ascontiguousarray(topk, dtype=np.int32)).cuda()
    rows_dev = torch.zeros(P + 1, dtype=torch.int64, device="cuda")
    for i in range(n):
        tok, rec = sets[i % nsets]
        nuna.all_to_all_routed(tok, rec, topk_dev, E, rows_dev, placement=place)
    torch.cuda.synchronize()
    lay.close()
    return {"moe_launches": n, "moe_alg_bytes": moe_alg_bytes(), "routed_launches": n}


# ---------------------------------------------------------------------------------------------- rocprofv3 summaries

TRAFFIC_JSON = os.path.join(ROOT, "profiles", "dominant_traffic.json")
# Sources the dominant kernel is compiled from (its kernel file and the headers it includes).
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_00867_amd", "csrc", f)
                  for f in ("nuna_allreduce.hip", "device_common.h", "placement.h", "kernels.h", "shapes.h")]


def kernel_source_text(text):
    """Source text as the compiler sees it for the traffic check: comments, trailing blanks and empty
    lines removed, so that a comment edit does not invalidate counters taken with the same code."""
    import re
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(line.rstrip() for line in text.splitlines() if line.strip())


def kernel_source_sha(texts=None):
    """SHA-256 over the dominant kernel's sources (comments and blank lines removed).  `texts` maps a
    file name to its text; by default the files are read from the tree."""
    import hashlib
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        name = os.path.basename(path)
        text = texts[name] if texts is not None else open(path).read()
        h.update(name.encode() + b"\0")
        h.update(kernel_source_text(text).encode())
    return h.hexdigest()


def _short(name):
    name = name.replace("nuna::(anonymous namespace)::", "")
    name = name[5:] if name.startswith("void ") else name
    return name.split("(")[0] if "(" in name else name


def _trace_rows(path):
    import csv
    rows = []
    for r in csv.DictReader(open(path)):
        rows.append({"name": _short(r["Kernel_Name"]), "start": int(r["Start_Timestamp"]),
                     "end": int(r["End_Timestamp"]), "grid": int(r["Grid_Size_X"]),
                     "grid_y": int(r.get("Grid_Size_Y") or 1), "wg": int(r["Workgroup_Size_X"]),
                     "queue": r.get("Queue_Id", "")})
    rows.sort(key=lambda r: r["start"])
    return rows


def summarize_trace(path, kernel_json=None):
    """Per (kernel, grid) durations of a rocprofv3 --kernel-trace CSV, as markdown.  With kernel_json,
    also write the dominant kernel's average (the fused two-shot kernel with the most total time: the
    64 MiB-per-rank launch of the default bench) for the bench line's cross-check."""
    import collections
    by = collections.defaultdict(list)
    for r in _trace_rows(path):
        by[(r["name"], r["grid"] * r["grid_y"], r["wg"])].append((r["end"] - r["start"]) / 1e3)
    print("| kernel | grid (threads) | workgroup | dispatches | avg µs | median µs | p10 µs | p90 µs |")
    print("|---|---|---|---|---|---|---|---|")
    for (k, g, w), v in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        v = sorted(v)
        print(f"| `{k}` | {g} | {w} | {len(v)} | {statistics.mean(v):.3f} | {statistics.median(v):.3f} | "
              f"{v[len(v) // 10]:.3f} | {v[(9 * len(v)) // 10]:.3f} |")
    if kernel_json:
        cands = [(sum(v), k, v) for k, v in by.items() if k[0].startswith("k_two_shot")]
        _, (k, g, w), v = max(cands)
        rec = {"kernel": k, "grid_threads": g, "workgroup": w, "dispatches": len(v),
               "avg_us": round(statistics.mean(v), 3), "median_us": round(statistics.median(v), 3),
               "source": os.path.relpath(kernel_json, ROOT).replace(".json", ".md"),
               "kernel_source_sha256": kernel_source_sha()}
        json.dump(rec, open(kernel_json, "w"), indent=1)
        print(f"\nDominant kernel: `{k}`, grid {g} threads, {len(v)} dispatches, average "
              f"{rec['avg_us']:.3f} µs (written to {os.path.basename(kernel_json)}).")


def _template_args(name):
    inner = name[name.index("<") + 1:name.rindex(">")]
    return [a.strip() for a in inner.split(",")]


def summarize_phases(path):
    """The two-kernel two-shot all-reduce from a kernel trace: each reduce-scatter launch that keeps
    its shards in cache (`k_reduce_scatter_direct<P, dtype, VPT, true>`) followed on its queue by an
    all-gather reading them (`k_all_gather_direct<P, VPT, true, WT>`).  Per message size: the two
    kernels' durations, the gap from the end of the first to the start of the second, and each
    phase's rate against its own bytes (reduce-scatter (P + 1) * n * s, all-gather P * n * s with the
    in-place shard skipped) and the call's against the collective's 2 * P * n * s."""
    import collections
    rows = _trace_rows(path)
    by_q = collections.defaultdict(list)
    for r in rows:
        by_q[r["queue"]].append(r)
    pairs = collections.defaultdict(list)
    for q in by_q.values():
        for a, b in zip(q, q[1:]):
            if not (a["name"].startswith("k_reduce_scatter_direct") and a["name"].endswith("true>")):
                continue
            if not b["name"].startswith("k_all_gather_direct") or _template_args(b["name"])[2] != "true":
                continue
            ta = _template_args(a["name"])
            P, es, vpt = int(ta[0]), (2 if ta[1] == "1" else 4), int(ta[2])
            shard = a["grid"] * vpt * 16  # bytes per shard (whole chunks at these sizes)
            pairs[(P, es, shard)].append(((a["end"] - a["start"]) / 1e3, (b["start"] - a["end"]) / 1e3,
                                          (b["end"] - b["start"]) / 1e3, a["name"], b["name"]))
    print("| P | bytes per rank | pairs | reduce-scatter µs | % of peak | gap µs | all-gather µs | % of peak | "
          "call µs (first start to last end) | % of peak (2·P·n·s) |")
    print("|---|---|---|---|---|---|---|---|---|---|")
    for (P, es, shard), v in sorted(pairs.items()):
        nb = P * shard
        rs = statistics.mean(x[0] for x in v)
        gap = statistics.mean(x[1] for x in v)
        ag = statistics.mean(x[2] for x in v)
        call = rs + gap + ag
        pct = lambda b, us: 100 * b / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS  # noqa: E731
        print(f"| {P} | {nb >> 20} MiB | {len(v)} | {rs:.3f} | {pct((P + 1) * nb, rs):.1f} | {gap:.3f} | "
              f"{ag:.3f} | {pct(P * nb, ag):.1f} | {call:.3f} | {pct(2 * P * nb, call):.1f} |")
    kinds = sorted({(x[3], x[4]) for v in pairs.values() for x in v})
    print("\nKernels: " + "; ".join(f"`{a}` then `{b}`" for a, b in kinds))


DOMINANT_ALG_BYTES = 2 * 8 * 4096 * 8192 * 2  # fused two-shot, P=8, [4096, 8192] bf16 per rank


def summarize_traffic(fetch_csv, write_csv):
    """FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the --profile run.  The reference copy moves
    PROFILE_COPY_BYTES each way; its readings give the scale factor of each counter.  The dominant
    kernel is the first collective kernel dispatched (after the dispatch probe of nuna_init)."""
    import csv
    import collections

    def read(path):
        by = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            by[(_short(r["Kernel_Name"]), int(r["Grid_Size"]))].append(float(r["Counter_Value"]))
        return by

    f, w = read(fetch_csv), read(write_csv)
    dom = [k for k in f if k[0].startswith("k_two_shot")][:1]  # dispatched first of the collectives
    cpy = [k for k in f if k[0].startswith("k_copy")]
    assert len(dom) == 1 and dom[0][0].startswith("k_two_shot") and len(cpy) == 1, (dom, cpy)
    kib = PROFILE_COPY_BYTES / 1024
    ff = kib / statistics.median(f[cpy[0]])
    wf = kib / statistics.median(w[cpy[0]])
    fetch = statistics.median(f[dom[0]]) * ff * 1024
    write = statistics.median(w[dom[0]]) * wf * 1024
    alg = DOMINANT_ALG_BYTES
    rec = {"kernel": dom[0][0], "grid": dom[0][1], "fetch_bytes": round(fetch), "write_bytes": round(write),
           "traffic_bytes": round(fetch + write), "alg_bytes": alg, "fetch_scale": round(ff, 4),
           "write_scale": round(wf, 4), "kernel_source_sha256": kernel_source_sha(),
           "kernel_source_sha256_covers": ", ".join(os.path.basename(p) for p in KERNEL_SOURCES)
           + " with comments and blank lines removed"}
    os.makedirs(os.path.dirname(TRAFFIC_JSON), exist_ok=True)
    json.dump(rec, open(TRAFFIC_JSON, "w"), indent=1)
    print("| counter | reference copy (KiB/dispatch, moves %d KiB each way) | scale | dominant kernel (KiB/dispatch) | "
          "scaled bytes |" % kib)
    print("|---|---|---|---|---|")
    print(f"| FETCH_SIZE | {statistics.median(f[cpy[0]]):.1f} | {ff:.4f} | {statistics.median(f[dom[0]]):.1f} | "
          f"{fetch:.0f} |")
    print(f"| WRITE_SIZE | {statistics.median(w[cpy[0]]):.1f} | {wf:.4f} | {statistics.median(w[dom[0]]):.1f} | "
          f"{write:.0f} |")
    print(f"\nTraffic per launch {fetch + write:.0f} B vs algorithmic {alg} B: ratio {(fetch + write) / alg:.4f}.")
    others = [k for k in f if k not in dom and k[0].startswith("k_") and not k[0].startswith(("k_copy", "k_probe"))]
    if others:
        malg = moe_alg_bytes()
        nb = PROFILE_PHASE_TOKENS * 8192 * 2  # bytes per rank of the traced two-kernel two-shot
        dec = 2 * 8 * 64 * 8192 * 2           # split all-reduce, decode T=64

        def alg_of(name):
            if name.startswith("k_reduce_scatter"):
                return 9 * nb, "(P + 1) n s"
            if name.startswith("k_all_gather"):
                return 8 * nb, "P n s (in-place shard skipped: (P - 1) n s written, n s read)"
            if name.startswith("k_allreduce"):
                return dec, "2 P n s"
            if name.startswith("k_route_count"):
                return route_count_bytes(), "top-k table read + routing records and counts written"
            return malg, "rows read + rows written"
        print("\nOther kernels of the same runs: the two-kernel two-shot at [256, 8192] bf16 per rank (its "
              "reduce-scatter and all-gather phases), the split all-reduce (decode T=64, 8 destination groups "
              "per chunk) and the MoE kernels (8 ranks, 512 tokens x 7168 bf16 per rank, top-8 of 256 "
              f"experts; the dispatch, the combine and the allocation-free dispatch's routing and copy):\n")
        print("| kernel | grid (threads) | FETCH_SIZE (KiB) | WRITE_SIZE (KiB) | scaled fetch B | scaled write B | "
              "algorithmic B | traffic / algorithmic |")
        print("|---|---|---|---|---|---|---|---|")
        for k in others:
            a, rule = alg_of(k[0])
            fk, wk = statistics.median(f[k]), statistics.median(w.get(k, [0.0]))
            fb, wb = fk * ff * 1024, wk * wf * 1024
            print(f"| `{k[0]}` | {k[1]} | {fk:.1f} | {wk:.1f} | {fb:.0f} | {wb:.0f} | {a} ({rule}) | "
                  f"{(fb + wb) / a:.4f} |")


def summarize_counters(path):
    """Per-kernel medians over dispatches of every counter in one rocprofv3 --pmc CSV (the library's
    kernels only)."""
    import csv
    import collections
    by = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in csv.DictReader(open(path)):
        by[(_short(r["Kernel_Name"]), int(r["Grid_Size"]))][r["Counter_Name"]].append(float(r["Counter_Value"]))
    names = sorted({c for v in by.values() for c in v})
    print("| kernel | grid (threads) | dispatches | " + " | ".join(names) + " |")
    print("|---|---|---|" + "---|" * len(names))
    for k, v in by.items():
        if not k[0].startswith(("k_", "nuna")):
            continue
        n = max(len(x) for x in v.values())
        cells = [f"{statistics.median(v[c]):.0f}" if c in v else "" for c in names]
        print(f"| `{k[0]}` | {k[1]} | {n} | " + " | ".join(cells) + " |")


def summarize_l2(linear_csv, xcd_csv):
    """TCC_HIT_sum / TCC_MISS_sum (L2 requests per dispatch, summed over the 8 XCDs' L2s) of two
    --profile runs, one per placement: the kernels whose map the placement changes."""
    import csv
    import collections

    def read(path):
        by = collections.defaultdict(lambda: collections.defaultdict(list))
        for r in csv.DictReader(open(path)):
            by[(_short(r["Kernel_Name"]), int(r["Grid_Size"]))][r["Counter_Name"]].append(float(r["Counter_Value"]))
        return by

    runs = {"LINEAR": read(linear_csv), "XCD": read(xcd_csv)}
    keys = []  # every kernel of either run, in dispatch order; a placement's grid may differ
    for run in runs.values():
        keys += [k for k in run if k not in keys and k[0].startswith(("k_allreduce", "k_all_to_all", "k_combine",
                                                                       "k_route"))]
    keys.sort(key=lambda k: (k[0], k[1]))
    print("| kernel | grid (threads) | placement | L2 hits | L2 misses | hit rate |")
    print("|---|---|---|---|---|---|")
    for k in keys:
        for mode, run in runs.items():
            if k not in run:
                continue
            h = statistics.median(run[k]["TCC_HIT_sum"])
            m = statistics.median(run[k]["TCC_MISS_sum"])
            print(f"| `{k[0]}` | {k[1]} | {mode} | {h:.0f} | {m:.0f} | {h / (h + m):.3f} |")


def write_xcc_counter_defs(path):
    """rocprofv3 extra counters: TCC_HIT and TCC_MISS of one XCC (the 16 L2 channels of that XCD)."""
    lines = ["rocprofiler-sdk:", "  counters-schema-version: 1", "  counters:"]
    for x in range(8):
        for c in ("HIT", "MISS"):
            lines += [f"  - name: TCC_{c}_XCC{x}",
                      f"    description: TCC_{c} summed over the 16 L2 channels of XCC {x}.",
                      "    properties: []",
                      "    definitions:",
                      "    - architectures:",
                      "      - gfx950",
                      f"      expression: reduce(select(TCC_{c},[DIMENSION_XCC=[{x}]]),sum)"]
    d = os.path.dirname(path)
    if d:
        os.makedirs(d, exist_ok=True)
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def summarize_l2_xcc(specs):
    """Per-XCD L2 hit rate (median over the dispatches of each pass) of the kernels whose map the placement
    changes, from passes that each collected some of the TCC_HIT_XCC<x> / TCC_MISS_XCC<x> counters."""
    import csv
    import collections
    vals = collections.defaultdict(list)  # (place, kernel, grid, counter) -> values
    for spec in specs:
        place, path = spec.split("=", 1)
        for r in csv.DictReader(open(path)):
            vals[(place.upper(), _short(r["Kernel_Name"]), int(r["Grid_Size"]), r["Counter_Name"])].append(
                float(r["Counter_Value"]))
    places = sorted({k[0] for k in vals})
    kernels = sorted({(k[1], k[2]) for k in vals
                      if k[1].startswith(("k_allreduce", "k_all_to_all", "k_combine", "k_route"))})
    print("| kernel | grid (threads) | placement | " + " | ".join(f"XCD {x}" for x in range(8)) + " | min–max |")
    print("|---|---|---|" + "---|" * 9)
    for kern, grid in kernels:
        for place in places:
            rates = []
            for x in range(8):
                h = vals.get((place, kern, grid, f"TCC_HIT_XCC{x}"))
                m = vals.get((place, kern, grid, f"TCC_MISS_XCC{x}"))
                if not h or not m:
                    rates.append(None)
                    continue
                hh, mm = statistics.median(h), statistics.median(m)
                rates.append(hh / (hh + mm) if hh + mm else None)
            if all(r is None for r in rates):
                continue
            got = [r for r in rates if r is not None]
            cells = " | ".join("—" if r is None else f"{r:.2f}" for r in rates)
            print(f"| `{kern}` | {grid} | {place} | {cells} | {min(got):.2f}–{max(got):.2f} |")


def measured_traffic():
    """HBM bytes per launch of the dominant kernel from the committed counter summary, or None when the
    kernel source has changed since the counters were taken."""
    try:
        rec = json.load(open(TRAFFIC_JSON))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_sha():
        return None
    return rec["traffic_bytes"]


# ---------------------------------------------------------------------------------------------- main

def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.kernel_json)
        return
    if args.summarize_phases:
        summarize_phases(args.summarize_phases)
        return
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic)
        return
    if args.xcc_counter_defs:
        write_xcc_counter_defs(args.xcc_counter_defs)
        return
    if args.summarize_l2_xcc:
        summarize_l2_xcc(args.summarize_l2_xcc)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return
    if args.summarize_l2:
        summarize_l2(*args.summarize_l2)
        return
    if (args.full or args.interference) and not args.out:
        print("--full and --interference need --out FILE.jsonl", file=sys.stderr)
        sys.exit(2)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (the path runs all P "
              f"simulated ranks on one GPU, and no figure across GPUs is produced).", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2608_00867_amd import nuna
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    nuna.init()
    for kv in args.set:
        name, _, val = kv.partition("=")
        nuna.set_tunable(name, int(val))
    pool = Pool(torch, POOL_BYTES_MAIN)

    if args.full:
        full_sweep(nuna, torch, pool, args)
        return
    if args.profile:
        profile_run(nuna, torch, pool, args.profile, args.profile_place)
        return
    if args.affinity:
        affinity(nuna, torch, pool)
        return
    if args.cu_affinity:
        cu_affinity(nuna, torch)
        return
    if args.interference:
        interference(nuna, torch, args)
        return

    from paper_2608_00867_amd import workloads as wl
    xs = [wl.ar_bf16_prefill(T) for T in wl.PREFILL_TOKENS]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    step_bytes, ksteps, per_graph, main_res = steps_timed(nuna, torch, pool, args, xs, "two_shot")
    t_timed = time.perf_counter() - t0
    sweep = prefill_sweep(nuna, torch, pool, args, xs)
    roof = roofline_dominant(sweep)
    x = main_res["xcd"]
    step_launch = [r for r in sweep if r["algo"] == "two_shot"]
    line = {
        "metric": METRIC,
        "value": round(x["gbps"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": ksteps,
        "warmup": args.warmup,
        "ms_per_step": round(x["ms_per_step"], 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "allreduce_two_shot_bf16_p8_prefill", "ranks": 8, "tokens": list(wl.PREFILL_TOKENS),
                   "hidden": 8192, "bytes_per_rank": [T * 8192 * 2 for T in wl.PREFILL_TOKENS], "data_dtype": "bf16",
                   "accumulate": "fp32", "placement": "xcd", "algo": "two_shot",
                   "cache": "cold (each call's inputs evicted from L2 and the Infinity Cache by the other calls)",
                   "timing": f"HIP graphs of {per_graph} steps replayed, LINEAR and XCD interleaved; HIP events"},
        "step_alg_bytes": step_bytes,
        "step_alg_bytes_rule": "sum over T of 2 * P * T * 8192 * 2 B (P reads and P writes per element)",
        "linear": {"value": round(main_res["linear"]["gbps"], 2),
                   "ms_per_step": round(main_res["linear"]["ms_per_step"], 6)},
        "linear_over_xcd_time": round(main_res["linear"]["ms_per_step"] / x["ms_per_step"], 4),
        "step_same_map": all(r["same_map"] for r in step_launch),
        "sweep": sweep,
        "roofline": roof,
        "parity": all(r["parity"] for r in sweep),
        "timed_region_s": round(t_timed, 3),
    }
    dec = decode_sweep(nuna, torch, pool, args)
    line["decode_sweep"] = dec
    line["moe_dispatch"] = moe_dispatch_summary(nuna, torch, pool, args)
    line["parity"] = line["parity"] and all(r["parity"] for r in dec) and bool(line["moe_dispatch"]["parity"])
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(args.cpu_seconds, xs)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
