"""Host logic of bench.py on synthetic inputs, no GPU: the kernel-trace, phase and traffic summaries that
the committed profiles come from, the per-record target verdicts, the graph sizing of the timed steps,
and the source hash that decides whether committed profiles still describe the kernel."""
import csv
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

TRACE_COLS = ["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X", "Grid_Size_Y", "Workgroup_Size_X",
              "Queue_Id"]


def _write_csv(path, cols, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=cols)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(cols, r)))


def _mangled(name):
    return f"void nuna::(anonymous namespace)::{name}(nuna::(anonymous namespace)::Ptrs<8>, long)"


def test_summarize_trace_takes_the_two_shot_with_most_time(tmp_path, capsys):
    """Rows per (kernel, total grid, workgroup), sorted by total time; the dominant kernel is the fused
    two-shot grid with the most total time, and its record carries the current source hash."""
    rows, t = [], 0
    for d_ns in (177000, 178000, 176000):  # the 64 MiB-per-rank fused two-shot: three dispatches
        rows.append([_mangled("k_two_shot<8, 1, 1, false, false>"), t, t + d_ns, 4194304, 1, 256, 1])
        t += d_ns + 1000
    for _ in range(10):  # a smaller two-shot grid with less total time
        rows.append([_mangled("k_two_shot_direct<8, 1, 4, false, false>"), t, t + 11500, 8192, 8, 128, 1])
        t += 12500
    rows.append([_mangled("k_allreduce_direct<8, 1, 1, false>"), t, t + 2500, 1024, 1, 64, 1])
    trace = tmp_path / "trace.csv"
    _write_csv(trace, TRACE_COLS, rows)
    kj = tmp_path / "dominant_kernel.json"
    bench.summarize_trace(str(trace), str(kj))
    out = capsys.readouterr().out
    rec = json.load(open(kj))
    assert rec["kernel"] == "k_two_shot<8, 1, 1, false, false>"
    assert rec["dispatches"] == 3 and rec["grid_threads"] == 4194304 and rec["workgroup"] == 256
    assert rec["avg_us"] == pytest.approx(177.0) and rec["median_us"] == pytest.approx(177.0)
    assert rec["kernel_source_sha256"] == bench.kernel_source_sha()
    lines = [line for line in out.splitlines() if line.startswith("| `")]
    assert lines[0].startswith("| `k_two_shot<8, 1, 1, false, false>` | 4194304 | 256 | 3 |")
    # the direct kernel's grid is x times y (8192 x 8), its total time 115 us
    assert lines[1].startswith("| `k_two_shot_direct<8, 1, 4, false, false>` | 65536 | 128 | 10 | 11.500 |")
    assert lines[2].startswith("| `k_allreduce_direct<8, 1, 1, false>` | 1024 | 64 | 1 | 2.500 |")


def test_summarize_phases_pairs_each_kept_reduce_scatter_with_the_next_all_gather(tmp_path, capsys):
    """Only a reduce-scatter that keeps its shards in cache, followed on the same queue by an all-gather
    that reads them through the cache, forms a pair; rates are against each phase's own bytes."""
    rs_keep = _mangled("k_reduce_scatter_direct<8, 1, 4, true>")
    rs_stream = _mangled("k_reduce_scatter_direct<8, 1, 4, false>")
    ag_cached = _mangled("k_all_gather_direct<8, 1, true, false>")
    rows = [
        # queue 1: a pair (16 MiB per rank: shards of 32768 x 4 vectors), gap 10 ns
        [rs_keep, 0, 26000, 32768, 8, 256, 1], [ag_cached, 26010, 46010, 131072, 8, 256, 1],
        # queue 1: a streaming reduce-scatter is no two-shot phase
        [rs_stream, 50000, 76000, 32768, 8, 256, 1], [ag_cached, 76010, 96010, 131072, 8, 256, 1],
        # queue 2: all-gather first, then a reduce-scatter with nothing after it
        [ag_cached, 0, 20000, 131072, 8, 256, 2], [rs_keep, 20010, 46010, 32768, 8, 256, 2],
    ]
    trace = tmp_path / "trace.csv"
    _write_csv(trace, TRACE_COLS, rows)
    bench.summarize_phases(str(trace))
    out = [line for line in capsys.readouterr().out.splitlines() if line.startswith("| 8 |")]
    assert len(out) == 1
    cells = [c.strip() for c in out[0].strip("|").split("|")]
    nb = 8 * 32768 * 4 * 16  # bytes per rank
    assert cells[1] == "16 MiB" and cells[2] == "1"
    assert float(cells[3]) == pytest.approx(26.0) and float(cells[5]) == pytest.approx(0.010)
    assert float(cells[6]) == pytest.approx(20.0) and float(cells[8]) == pytest.approx(46.01)
    pct = lambda b, us: 100 * b / (us * 1e-6) / 1e9 / bench.HBM_PEAK_GBPS  # noqa: E731
    assert float(cells[4]) == pytest.approx(pct(9 * nb, 26.0), abs=0.05)
    assert float(cells[7]) == pytest.approx(pct(8 * nb, 20.0), abs=0.05)
    assert float(cells[9]) == pytest.approx(pct(16 * nb, 46.01), abs=0.05)


def test_summarize_traffic_scales_each_counter_by_the_reference_copy(tmp_path, capsys, monkeypatch):
    """FETCH_SIZE and WRITE_SIZE are scaled so that the 64 MiB reference copy reads as 64 MiB each way;
    the dominant kernel is the first fused two-shot dispatched; the dispatch probe is left out."""
    monkeypatch.setattr(bench, "TRAFFIC_JSON", str(tmp_path / "dominant_traffic.json"))
    cols = ["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"]
    kib = bench.PROFILE_COPY_BYTES / 1024
    fetch = [["k_probe_xcc", 131072, "FETCH_SIZE", 1.0]]
    write = [["k_probe_xcc", 131072, "WRITE_SIZE", 1.0]]
    for v in (262100.0, 262200.0, 262150.0):
        fetch.append([_mangled("k_two_shot<8, 1, 1, false, false>"), 4194304, "FETCH_SIZE", v])
        write.append([_mangled("k_two_shot<8, 1, 1, false, false>"), 4194304, "WRITE_SIZE", 2 * v])
    for _ in range(3):
        fetch.append(["void nuna::(anonymous namespace)::k_copy<1>(uint4*)", 4194304, "FETCH_SIZE", kib / 2])
        write.append(["void nuna::(anonymous namespace)::k_copy<1>(uint4*)", 4194304, "WRITE_SIZE", kib])
    _write_csv(tmp_path / "f.csv", cols, fetch)
    _write_csv(tmp_path / "w.csv", cols, write)
    bench.summarize_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"))
    rec = json.load(open(tmp_path / "dominant_traffic.json"))
    assert rec["kernel"] == "k_two_shot<8, 1, 1, false, false>" and rec["grid"] == 4194304
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    assert rec["fetch_bytes"] == round(262150.0 * 2 * 1024) and rec["write_bytes"] == round(2 * 262150.0 * 1024)
    assert rec["traffic_bytes"] == rec["fetch_bytes"] + rec["write_bytes"]
    assert rec["alg_bytes"] == bench.DOMINANT_ALG_BYTES == 2 * 8 * 4096 * 8192 * 2
    assert rec["kernel_source_sha256"] == bench.kernel_source_sha()
    out = capsys.readouterr().out
    assert f"ratio {rec['traffic_bytes'] / rec['alg_bytes']:.4f}" in out and "k_probe_xcc" not in out


def test_summarize_l2_lists_kernels_of_either_placement(tmp_path, capsys):
    """A kernel whose grid differs between the placements (the layout-driven dispatch sizes its XCD grid
    for the longest per-XCD list) is listed under each placement; a kernel of neither family is not."""
    cols = ["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"]

    def rows(grid_a2a, hit):
        out = []
        for name, grid in (("k_all_to_all<8, 4>", grid_a2a), ("k_route_copy<8>", 8388608), ("k_copy<1>", 4096)):
            out.append([_mangled(name), grid, "TCC_HIT_sum", hit])
            out.append([_mangled(name), grid, "TCC_MISS_sum", 100.0 - hit])
        return out

    _write_csv(tmp_path / "lin.csv", cols, rows(5544704, 34.0))
    _write_csv(tmp_path / "xcd.csv", cols, rows(5548032, 60.0))
    bench.summarize_l2(str(tmp_path / "lin.csv"), str(tmp_path / "xcd.csv"))
    out = capsys.readouterr().out
    assert "| `k_all_to_all<8, 4>` | 5544704 | LINEAR | 34 | 66 | 0.340 |" in out
    assert "| `k_all_to_all<8, 4>` | 5548032 | XCD | 60 | 40 | 0.600 |" in out
    assert "| `k_route_copy<8>` | 8388608 | LINEAR |" in out and "| `k_route_copy<8>` | 8388608 | XCD |" in out
    assert "k_copy" not in out


def test_route_count_bytes_at_the_moe_shape():
    """The routing kernel's algorithmic bytes at 8 ranks x 512 tokens, top-8: the table read (4 B per entry),
    min(k, P) = 8 records per token and the 8 x 8 + 8 counts written."""
    assert bench.route_count_bytes() == 4 * 8 * 512 * 8 + 4 * 8 * 512 * 8 + 4 * 64 + 4 * 8


def test_target_verdicts():
    """No slower: XCD's median within 2 % of LINEAR's, or XCD's p10 at or below LINEAR's p90.  The 70 %
    verdict applies from 4 MiB per rank only."""
    def rec(x, lx, **kw):
        return {"xcd_us": {"median": x[0], "p10": x[1]}, "linear_us": {"median": lx[0], "p90": lx[1]}, **kw}
    r = rec((10.15, 10.1), (10.0, 10.05), bytes_per_rank=1 << 20, xcd_frac_hbm=0.5)
    bench.annotate_targets(r)
    assert r["xcd_no_slower"] is True and "meets_70pct" not in r
    r = rec((11.0, 10.9), (10.0, 10.5), bytes_per_rank=4 << 20, xcd_frac_hbm=0.71)
    bench.annotate_targets(r)
    assert r["xcd_no_slower"] is False and r["meets_70pct"] is True
    r = rec((10.5, 10.2), (10.0, 10.3), shard_bytes=1 << 20, P=8, xcd_frac_hbm=0.69)
    bench.annotate_targets(r)
    assert r["xcd_no_slower"] is True and r["meets_70pct"] is False  # 8 MiB per rank, distributions overlap
    assert bench.message_bytes_per_rank({"tokens_per_rank": 512, "hidden": 7168}) == 512 * 7168 * 2


@pytest.mark.parametrize("ksteps,step_bytes,want", [(20, 1409286144, 5), (20, 1 << 20, 20), (7, 2 << 30, 1),
                                                      (1, 1 << 40, 1), (12, 1 << 30, 6), (13, 1 << 30, 8)])
def test_steps_per_graph(ksteps, step_bytes, want):
    """A graph holds the largest divisor of the timed steps within the 8 GiB target, or the target itself
    when that divisor is under a quarter of it."""
    assert bench.steps_per_graph(ksteps, step_bytes) == want


def test_source_hash_ignores_comments_but_not_code():
    """Committed profiles stay valid across comment edits and go stale on any code change."""
    texts = {os.path.basename(p): open(p).read() for p in bench.KERNEL_SOURCES}
    base = bench.kernel_source_sha(texts)
    assert base == bench.kernel_source_sha()
    edited = dict(texts)
    edited["nuna_allreduce.hip"] = "// a new note\n/* and a\n   block */\n" + texts["nuna_allreduce.hip"] + "\n\n"
    assert bench.kernel_source_sha(edited) == base
    edited["shapes.h"] = texts["shapes.h"] + "\nconstexpr int kUnused = 1;\n"
    assert bench.kernel_source_sha(edited) != base


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused(n):
    """bench.py measures one GPU: --gpus above 1 exits with status 2 and says why, before touching a GPU."""
    import subprocess
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert f"--gpus {n} is not supported" in r.stderr and "one GPU" in r.stderr
    assert r.stdout == ""
