"""Host logic of bench.py (no GPU): the traffic model, the gate on the
committed hardware counters, the refusal of several GPUs, and the oracle's CPU
baseline on a bounded sample."""

import os
import subprocess
import sys

import numpy as np

import bench
import oracle
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_traffic_model_by_hand():
    # 3 rows, 10 entries of which 4 in halo rows, F = 6: row pointers 24 B,
    # entries 80 B, 6 local rows of 24 B, 4 halo rows of 6 code bytes + 8 B
    # (8-bit) or 2 + 8 B (2-bit), outputs 3 x 24 B
    assert bench.model_bytes(3, 10, 4, 6, 8) == 24 + 80 + 144 + 56 + 72
    assert bench.model_bytes(3, 10, 4, 6, 2) == 24 + 80 + 144 + 40 + 72
    assert bench.model_bytes(3, 10, 0, 6) == 24 + 80 + 240 + 72


def _counters_file(path, sha, kernel="agg_pieces", sym="k_pieces<4, 32, SrcQ<4, 8, false> >"):
    with open(path, "w") as f:
        f.write("# table\n")
        f.write("# %-40s %16s %16s %14s %14s %8s\n" % ("kernel", "F", "W", "f", "w", "L2_hit"))
        f.write("# %-40s %16.6g %16.6g %14.2f %14.2f %7.1f%%\n" % (sym, 1.0, 1.0, 1.0, 1.0, 61.5))
        f.write("kernel: %s\nkernel_symbol: %s\nsource_sha256: %s\n" % (kernel, sym, sha))
        f.write("fetch_bytes_per_dispatch: 1000\nwrite_bytes_per_dispatch: 234\n")


def test_counters_gate_on_source_hash(tmp_path, monkeypatch):
    src = tmp_path / "kernels.hip"
    src.write_text("// kernels\n")
    monkeypatch.setattr(bench, "AGG_SOURCES", [str(src)])
    cfile = tmp_path / "counters.txt"
    monkeypatch.setattr(bench, "COUNTERS", str(cfile))
    assert bench.read_counters("agg_pieces") == (None, None)  # no file
    _counters_file(cfile, bench.sources_sha256([str(src)]))
    assert bench.read_counters("agg_pieces") == (1234.0, 0.615)
    assert bench.read_counters("agg_short") == (None, None)  # another kernel
    src.write_text("// kernels, edited\n")  # counters taken on other sources
    assert bench.read_counters("agg_pieces") == (None, None)


def test_several_gpus_are_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_cpu_baseline_small_graph_repeats_and_threads():
    n = 512
    src, dst = synth.rmat_edges(71, n, 8 * n, perm_seed=72)
    w = synth.Workload("rmat512", n, n, src, dst, synth.SYMMETRIZE | synth.ADD_SELF_LOOPS, 16)
    X = synth.normal(73, n, 16)
    before = oracle.num_threads()
    try:
        b = bench.cpu_baseline(w, X, None, 16, 0.3, 8, threads=1)
        assert b["cores"] == 1 and b["kind"] == "oracle" and b["unit"] == "GB/s"
        assert b["value"] > 0 and b["edge_features_per_s"] > 0
        # the whole graph is far below 0.3 s of work: it is run repeatedly
        assert "%d uniformly sampled rows" % n in b["sample"] and "repeated" in b["sample"]
        assert "median of 3 such batches" in b["sample"]
        q = bench.cpu_baseline(w, X, 3 * n // 4, 16, 0.1, 8, threads=1)
        assert "8-bit halo dequantized" in q["sample"] and q["value"] > 0
    finally:
        oracle.set_num_threads(before)
    assert oracle.num_threads() == before
    assert np.isfinite(b["seconds"])
