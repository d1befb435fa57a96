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


def _counters_file(path, sha):
    with open(path, "w") as f:
        f.write("# table\n")
        f.write("source_sha256: %s\nfetch_scale: 2.0\n" % sha)
        f.write("counted: agg_pieces fwd 1000 234 0.615\n")
        f.write("counted: agg_pieces bwd 1100 300 0.6\n")
        f.write("counted: agg_short fwd 50 5 0.2\n")


def test_counters_gate_on_source_hash(tmp_path, monkeypatch):
    src = tmp_path / "kernels.hip"
    src.write_text("// kernels\n")
    monkeypatch.setattr(bench, "AGG_SOURCES", [str(src)])
    cfile = tmp_path / "counters.txt"
    assert bench.read_counters(str(cfile)) is None  # no file
    _counters_file(cfile, bench.sources_sha256([str(src)]))
    c = bench.read_counters(str(cfile))
    assert c["rows"][("agg_pieces", "fwd")] == (1000.0, 234.0, 0.615)
    assert c["rows"][("agg_pieces", "bwd")] == (1100.0, 300.0, 0.6)
    assert c["rows"][("agg_short", "fwd")] == (50.0, 5.0, 0.2)
    assert c["fetch_scale"] == "2.0"
    src.write_text("// kernels, edited\n")  # counters taken on other sources
    assert bench.read_counters(str(cfile)) is None


def test_counters_path_per_workload():
    assert bench.counters_path("rmat24_q8").endswith("profiles/agg_counters_rmat24_q8.txt")
    assert bench.counters_path("rmat24_q8", 2).endswith("profiles/agg_counters_rmat24_q8_int2.txt")


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
        b = bench.cpu_baseline(w, X, None, 16, 0.3, 8, threads=1, G_h=X)
        assert b["cores"] == 1 and b["kind"] == "oracle" and b["unit"] == "GB/s"
        assert b["value"] > 0 and b["edge_features_per_s"] > 0
        assert b["fwd"]["GBps"] > 0 and b["bwd"]["GBps"] > 0
        # the whole graph is far below 0.3 s of work: it is run repeatedly
        assert "%d rows of A " % n in b["sample"] and "repeated" in b["sample"]
        assert "%d rows of A^T" % n in b["sample"]
        assert "median of 3 such batches" in b["sample"]
        q = bench.cpu_baseline(w, X, 3 * n // 4, 16, 0.1, 8, threads=1)
        assert "8-bit halo dequantized" in q["sample"] and q["value"] > 0
    finally:
        oracle.set_num_threads(before)
    assert oracle.num_threads() == before
    assert np.isfinite(b["seconds"])
