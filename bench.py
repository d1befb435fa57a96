#!/usr/bin/env python
"""Benchmark of the GCN aggregation hot path on one MI355X.

One step = one forward aggregation Y = A_hat x and one backward aggregation
dX = A_hat^T g over the same graph, where the last quarter of the node ids
are halo rows held as uint8 codes with a per-row (min, scale) that the
kernels dequantize on read (fused dequantize + aggregate). The default
workload is the RMAT graph of scale 24 (16,777,216 nodes, 32 draws per
node, quadrant probabilities .57/.19/.19/.05, relabelled by a seeded
permutation, symmetrized, deduplicated, one self-loop per node), F = 128,
fp32 inputs drawn from N(0, 1).

Reported: modeled bytes per second for the whole step under the traffic
model (CSR bytes + gathered-row bytes + output bytes, where every stored
entry brings its source row: the algorithm's traffic without cache reuse,
so caches that serve repeated rows can put it above the 8 TB/s HBM peak),
the bytes the L2 actually moved to and from the memory fabric (hardware
counters committed under profiles/, scaled by a factor checked on a gather
of known size), the compulsory traffic (every input row once), edge-features
per second, the dominant kernel's roofline figures from per-launch HIP
events, and the CPU oracle timed on a bounded row sample of the same
workload.

The graph build (sort, deduplication, transpose, binning) and the
normalization run once per graph; they are timed separately and are not
part of a step.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "aggregation GB/s (% of HBM peak) + edge-features/s, fwd Â·X and bwd Âᵀ·G"
HBM_PEAK_GBS = 8000.0
# the kernels and the plan that decides their work: counters taken on other
# sources do not describe the library being timed
AGG_SOURCES = [os.path.join(ROOT, "paper_2411_16025_amd", "csrc", f)
               for f in ("aggregate.hip", "build.hip")]
MODEL_NOTE = ("no-reuse gather model: every stored entry brings its source row, so cache hits "
              "on repeated rows are priced as HBM traffic and frac can exceed 1; the counted "
              "fabric bytes are the hardware figure")

# kernel name -> row-length classes whose rows it processes
KERNEL_CLASSES = {"agg_zero_rows": [0], "agg_tiny": [1, 2], "agg_short": [3, 4, 5, 6, 7],
                  "agg_chunk": [8], "agg_pieces": [9]}


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="rmat24_q8",
                    choices=["rmat24_q8", "rmat24", "rmat20", "er4096", "product", "partition",
                             "perm22", "gcn_step", "sage_step", "prepost", "producer", "gemm"])
    ap.add_argument("--halo-bits", type=int, default=8, choices=[8, 2],
                    help="code width of the halo rows (8: one byte per feature; 2: four per byte)")
    ap.add_argument("--senders", type=int, default=7,
                    help="prepost: number of workers that own the halo nodes")
    ap.add_argument("--cpu-target-s", type=float, default=12.0,
                    help="approximate seconds of oracle work for the CPU baseline")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="threads of the oracle for the CPU baseline (0: all it sees)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=2,
                    help="extra steps with per-kernel HIP event timing")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="first run one plain device copy of this size (a known-size kernel "
                         "for scaling hardware byte counters)")
    return ap.parse_args()


def code_bytes(F, bits=8):
    return F if bits == 8 else (F + 3) // 4


def model_bytes(rows, entries, halo_entries, F, bits=8):
    """Modeled bytes of one pass with no reuse of gathered rows: row pointer
    (8 B/row), column + value (8 B/entry), every gathered row at full cost (4F B
    for fp32; the code bytes + 8 B for a quantized halo row with its min and
    scale), output rows (4F B). Rows gathered more than once are charged each
    time, so this exceeds the compulsory bytes and a rate over it can exceed
    the HBM peak; the counted fabric bytes are the physical figure."""
    local = entries - halo_entries
    return (8 * rows + 8 * entries + 4 * F * local + (code_bytes(F, bits) + 8) * halo_entries
            + 4 * F * rows)


def sources_sha256(paths):
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def counters_path(workload, bits=8):
    tag = workload + ("_int2" if bits == 2 else "")
    return os.path.join(ROOT, "profiles", "agg_counters_%s.txt" % tag)


def read_counters(path):
    """Per (library kernel name, pass): counted L2-to-fabric bytes read and
    written per pass and the L2 hit rate, from a committed rocprofv3 summary,
    only if it was taken on the current aggregation source; else None."""
    if not os.path.exists(path):
        return None
    kv, rows = {}, {}
    for line in open(path).read().splitlines():
        if line.startswith("#") or ":" not in line:
            continue
        k, v = line.split(":", 1)
        if k.strip() == "counted":
            name, op, fetch, write, hit = v.split()
            rows[(name, op)] = (float(fetch), float(write), float(hit))
        else:
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != sources_sha256(AGG_SOURCES) or not rows:
        return None
    return {"rows": rows, "fetch_scale": kv.get("fetch_scale"), "path": os.path.relpath(path, ROOT)}


FP32_MFMA_PEAK_TFLOPS = 157.3
OVERLAP_NOTE = ("per-kernel times are HIP events around each launch; the weight-gradient products "
                "run on a second stream and overlap other kernels, so the parts add up to more "
                "than ms_per_step and the rates derived from them are lower bounds")


def run_gcn_step(args):
    """One training step of the 2-layer GCN (F_in 100, hidden 256, 47 classes)
    on the product-shaped graph, all in the library: three aggregations (the
    100-wide inputs, the 47-wide logits forward and their gradient backward;
    layer 1 aggregates before its transform, so its backward needs none), five
    GEMMs (the first with the ReLU in its epilogue) and softmax cross-entropy."""
    import torch
    import synth
    import paper_2411_16025_amd as G

    dev = torch.device("cuda:0")
    w = synth.product_like()
    g = G.gcn_build_csr(w.n_rows, w.n_cols, torch.from_numpy(w.src).to(dev),
                        torch.from_numpy(w.dst).to(dev), w.flags)
    G.gcn_normalize(g)
    n, f_in, hidden, ncls = w.n_rows, 100, 256, 47
    X = torch.from_numpy(synth.normal(3003, n, f_in)).to(dev)
    W1 = torch.from_numpy(synth.glorot(5003, f_in, hidden)).to(dev)
    W2 = torch.from_numpy(synth.glorot(5103, hidden, ncls)).to(dev)
    y = torch.from_numpy(synth.labels(5203, n, ncls)).to(dev)
    step = lambda: G.gcn_gcn2_step(g, X, W1, W2, y)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ts = time.time()
    for _ in range(args.steps):
        out = step()
    torch.cuda.synchronize()
    step_ms = (time.time() - ts) * 1e3 / args.steps
    G.gcn_profile_enable(True)
    for _ in range(max(1, args.profile_steps)):
        step()
    torch.cuda.synchronize()
    prof = G.gcn_profile_read()
    G.gcn_profile_enable(False)
    ps = max(1, args.profile_steps)
    gemm_flop = 2 * n * (f_in * hidden * 2 + hidden * ncls * 3)
    gemm_ms = sum(v[1] for k, v in prof.items() if k.startswith("gemm")) / ps
    agg_ms = sum(v[1] for k, v in prof.items() if k.startswith("agg")) / ps
    bins = G.gcn_graph_bins(g, 0)
    rows = sum(b["rows"] for b in bins)
    ents = sum(b["entries"] for b in bins)
    agg_bytes = model_bytes(rows, ents, 0, f_in) + 2 * model_bytes(rows, ents, 0, ncls)
    out_json = {
        "metric": "2-layer GCN training step (fwd + bwd), product-shaped graph",
        "value": round(step_ms, 3), "unit": "ms", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(step_ms, 3), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "nodes": n, "nnz": g.nnz, "f_in": f_in, "hidden": hidden,
                   "classes": ncls},
        "loss": float(out[0]),
        "aggregation_ms_per_step": round(agg_ms, 3),
        "aggregation_modeled_GBps": round(agg_bytes / (agg_ms * 1e-3) / 1e9, 1),
        "gemm_ms_per_step": round(gemm_ms, 3),
        "gemm_TFLOPs": round(gemm_flop / (gemm_ms * 1e-3) / 1e12, 2),
        "gemm_frac_of_fp32_mfma_peak": round(gemm_flop / (gemm_ms * 1e-3) / 1e12
                                             / FP32_MFMA_PEAK_TFLOPS, 4),
        "kernels_ms_per_step": {k: round(v[1] / ps, 4) for k, v in prof.items()},
        "breakdown_note": OVERLAP_NOTE,
        "roofline": {"bound": "hbm", "kernel": "aggregation (3 passes)",
                     "achieved": round(agg_bytes / (agg_ms * 1e-3) / 1e9, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(agg_bytes / (agg_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": None},
    }
    print(json.dumps(out_json), flush=True)


def run_sage_step(args):
    """One training step of the 3-layer GraphSAGE model of the evaluation
    (LayerNorm before each layer, mean aggregation, F_in 100, hidden 256, 47
    classes) on the product-shaped graph without self-loops, with the labels
    of half of the nodes embedded (masked label propagation)."""
    import torch
    import synth
    import paper_2411_16025_amd as G

    dev = torch.device("cuda:0")
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    w = synth.product_like()
    n, f_in, hidden, C = w.n_rows, 100, 256, 47
    g = G.gcn_build_csr(n, n, d(w.src), d(w.dst), synth.SYMMETRIZE)
    G.gcn_normalize_mean(g)
    X = d(synth.normal(3003, n, f_in))
    params = []
    for k, (a, b) in enumerate([(f_in, hidden), (hidden, hidden), (hidden, C)]):
        params += [d(synth.glorot(5003 + 3 * k, a, b)), d(synth.glorot(5004 + 3 * k, a, b)),
                   d(0.1 * synth.uniform(5005 + 3 * k, 1, b)[0])]
    y = d(synth.labels(5203, n, C))
    mask = d((synth.uniform(5204, n, 1)[:, 0] < 0.0).astype(np.uint8))
    E = d(0.5 * synth.normal(5205, C, f_in))
    step = lambda: G.gcn_sage3_step(g, X, params, y, mask, E)  # noqa: E731
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ts = time.time()
    for _ in range(args.steps):
        out = step()
    torch.cuda.synchronize()
    step_ms = (time.time() - ts) * 1e3 / args.steps
    G.gcn_profile_enable(True)
    for _ in range(max(1, args.profile_steps)):
        step()
    torch.cuda.synchronize()
    prof = G.gcn_profile_read()
    G.gcn_profile_enable(False)
    ps = max(1, args.profile_steps)
    dims = [(f_in, hidden), (hidden, hidden), (hidden, C)]
    # algorithmic flops: Y W_self + Z W_neigh (forward), the weight gradients,
    # and the input gradients of all three layers (label propagation needs layer 1's)
    flop = sum(2 * n * 2 * f * fo * 3 for f, fo in dims)
    gemm_ms = sum(v[1] for k, v in prof.items() if k.startswith("gemm")) / ps
    agg_ms = sum(v[1] for k, v in prof.items() if k.startswith("agg")) / ps
    bins = G.gcn_graph_bins(g, 0)
    rows = sum(b["rows"] for b in bins)
    ents = sum(b["entries"] for b in bins)
    # forward + transposed per layer, each gathering the narrower of the layer's
    # input and output (the class layer aggregates Y W_neigh, 47 wide)
    agg_bytes = 2 * sum(model_bytes(rows, ents, 0, fo if fo < f else f) for f, fo in dims)
    out_json = {
        "metric": "3-layer GraphSAGE training step (fwd + bwd, LayerNorm, masked label "
                  "propagation), product-shaped graph",
        "value": round(step_ms, 3), "unit": "ms", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(step_ms, 3), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name + "_sage3", "nodes": n, "nnz": g.nnz, "f_in": f_in,
                   "hidden": hidden, "classes": C, "lp_fraction": 0.5},
        "loss": float(out[0]),
        "aggregation_ms_per_step": round(agg_ms, 3),
        "aggregation_modeled_GBps": round(agg_bytes / (agg_ms * 1e-3) / 1e9, 1),
        "gemm_ms_per_step": round(gemm_ms, 3),
        "gemm_TFLOPs": round(flop / (gemm_ms * 1e-3) / 1e12, 2),
        "gemm_frac_of_fp32_mfma_peak": round(flop / (gemm_ms * 1e-3) / 1e12
                                             / FP32_MFMA_PEAK_TFLOPS, 4),
        "kernels_ms_per_step": {k: round(v[1] / ps, 4) for k, v in prof.items()},
        "breakdown_note": OVERLAP_NOTE,
        "roofline": {"bound": "hbm", "kernel": "aggregation (6 passes)",
                     "achieved": round(agg_bytes / (agg_ms * 1e-3) / 1e9, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(agg_bytes / (agg_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": None},
    }
    print(json.dumps(out_json), flush=True)


def run_prepost(args):
    """Hybrid pre/post-aggregation on the 14M x 20M partition: the halo nodes
    belong to --senders workers (contiguous id ranges). Per sender, the host
    split (Algorithm 1), the sender's pre-aggregation SpMM, and the receiver's
    post-aggregation SpMM plus the partial-sum combine, against the plain
    aggregation that receives every halo row with a cut edge."""
    import torch
    import synth
    import paper_2411_16025_amd as G

    dev = torch.device("cuda:0")
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    t0 = time.time()
    w = synth.partition_111m()
    F, nl, nh = w.F, w.n_rows, w.n_cols - w.n_rows
    log("generated %s: %d entries in %.1f s" % (w.name, len(w.src), time.time() - t0))
    X = synth.normal(3004, w.n_cols, F)
    g_full = G.gcn_build_csr(w.n_rows, w.n_cols, d(w.src), d(w.dst), w.flags)
    deg_d = d(w.deg)
    G.gcn_normalize(g_full, deg_d)
    cut = w.src >= nl
    local = ~cut
    s_all, d_all = w.src[cut] - nl, w.dst[cut]
    owner = (s_all.astype(np.int64) * args.senders) // nh
    split_s, vol, senders = 0.0, np.zeros(4, np.int64), []
    post_src, post_dst, col_ids, n_cols = [], [], [np.arange(nl)], nl
    for o in range(args.senders):
        lo, hi = -(-o * nh // args.senders), -(-(o + 1) * nh // args.senders)
        m = owner == o
        sl, dd = (s_all[m] - lo).astype(np.int32), d_all[m]
        ts = time.time()
        is_post, src_slot, dst_slot, v = G.gcn_prepost_split(sl, dd, hi - lo, nl)
        split_s += time.time() - ts
        vol += (len(sl), len(np.unique(dd)), len(np.unique(sl)), v)
        cov_src = np.flatnonzero(src_slot >= 0)
        cov_dst = np.flatnonzero(dst_slot >= 0).astype(np.int32)
        pre = ~is_post
        gp = G.gcn_build_csr(len(cov_dst), hi - lo, d(sl[pre]), d(dst_slot[dd[pre]]), 0)
        G.gcn_normalize_rc(gp, d(w.deg[cov_dst]), deg_d[nl + lo: nl + hi].contiguous())
        senders.append((gp, d(X[nl + lo: nl + hi]), d(cov_dst)))
        col_ids.append(nl + lo + cov_src)
        post_src.append(n_cols + src_slot[sl[is_post]])
        post_dst.append(dd[is_post])
        n_cols += len(cov_src)
        log("sender %d: %d cut edges, rows sent %d (post-only %d, pre-only %d)"
            % (o, len(sl), v, len(np.unique(sl)), len(np.unique(dd))))
    col_ids = np.concatenate(col_ids)
    g_recv = G.gcn_build_csr(nl, n_cols, d(np.concatenate([w.src[local]] + post_src).astype(np.int32)),
                             d(np.concatenate([w.dst[local]] + post_dst).astype(np.int32)),
                             synth.ADD_SELF_LOOPS)
    G.gcn_normalize_rc(g_recv, deg_d[:nl].contiguous(), d(w.deg[col_ids]))
    X_full = d(X)
    X_recv = d(X[col_ids])
    Y_full = torch.empty(nl, F, device=dev)
    Y_recv = torch.empty(nl, F, device=dev)
    partials = [torch.empty(gp.n_rows, F, device=dev) for gp, _, _ in senders]

    def full():
        G.gcn_aggregate_fwd(g_full, X_full, Y_full)

    def send():
        for (gp, xs, _), P in zip(senders, partials):
            G.gcn_aggregate_fwd(gp, xs, P)

    def recv():
        G.gcn_aggregate_fwd(g_recv, X_recv, Y_recv)
        for (_, _, idx), P in zip(senders, partials):
            G.gcn_add_rows(P, idx, Y_recv)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        t = time.time()
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        return (time.time() - t) * 1e3 / args.steps

    full_ms, send_ms = timed(full), timed(send)
    recv_ms = timed(recv)
    S = torch.abs(Y_full).max().item()
    diff = torch.abs(Y_full - Y_recv).max().item()
    row_bytes = 4 * F
    out = {
        "metric": "hybrid pre/post aggregation: rows sent to one receiver and its aggregation time",
        "value": int(vol[3]), "unit": "rows", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(recv_ms, 3), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name + "_prepost", "senders": args.senders, "F": F,
                   "cut_edges": int(vol[0])},
        "rows_sent": {"edges": int(vol[0]), "pre_only": int(vol[1]), "post_only": int(vol[2]),
                      "hybrid": int(vol[3])},
        "bytes_sent_fp32": {"post_only": int(vol[2]) * row_bytes, "hybrid": int(vol[3]) * row_bytes},
        "split_host_s": round(split_s, 3),
        "receiver_full_ms": round(full_ms, 3), "receiver_hybrid_ms": round(recv_ms, 3),
        "senders_pre_ms_total": round(send_ms, 3),
        "max_abs_diff_vs_full": diff, "max_abs_output": S,
        "nnz_full": g_full.nnz, "nnz_receiver_hybrid": g_recv.nnz,
        "nnz_senders_pre": int(sum(gp.nnz for gp, _, _ in senders)),
    }
    print(json.dumps(out), flush=True)


def run_producer(args):
    """The sender side of the quantized exchange on the RMAT-24 halo share
    (4,194,304 rows x 128 fp32, N(0, 1)): row LayerNorm fused with 2-bit
    quantization (codes packed four per byte, paired (min, scale)), plus the
    8-bit and no-LayerNorm variants. Modeled bytes per call: the rows read
    (4F B), the codes and the 8-byte parameter pair written."""
    import torch
    import synth
    import paper_2411_16025_amd as G

    dev = torch.device("cuda:0")
    n, F = 1 << 22, 128
    X = torch.from_numpy(synth.normal(3005, n, F)).to(dev)
    variants = [("layernorm+int2", True, 2), ("int2", False, 2), ("layernorm+u8", True, 8),
                ("u8", False, 8)]
    res = {}
    for name, ln, bits in variants:
        fn = lambda: G.gcn_layernorm_quantize(X, bits=bits, layernorm=ln)  # noqa: E731
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(args.steps):
            fn()
        ev[1].record()
        ev[1].synchronize()
        ms = ev[0].elapsed_time(ev[1]) / args.steps
        B = n * (4 * F + code_bytes(F, bits) + 8)
        res[name] = {"ms": round(ms, 4), "modeled_GB": round(B / 1e9, 3),
                     "GBps": round(B / (ms * 1e-3) / 1e9, 1),
                     "frac": round(B / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        log("%s: %.3f ms, %.1f GB/s" % (name, ms, res[name]["GBps"]))
    main_v = res["layernorm+int2"]
    out = {
        "metric": "fused LayerNorm + 2-bit quantize of the halo rows, GB/s",
        "value": main_v["GBps"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": main_v["ms"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "rmat24 halo rows 4194304 x 128 N(0,1)", "rows": n, "F": F},
        "variants": res,
        "roofline": {"bound": "hbm", "kernel": "ln_quantize", "achieved": main_v["GBps"],
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": main_v["frac"],
                     "traffic": None},
    }
    print(json.dumps(out), flush=True)


def run_gemm(args):
    """Each fp32 product of the training steps alone, at the product-shaped
    graph's 2,449,029 rows, in the layouts the steps use (rows padded to a
    multiple of 4 floats), timed with HIP events on the stream the library
    launches on. Per product: the algorithmic bytes (each operand and the
    result once) and flops, the roofline time max(flops / 157.3 TFLOP/s,
    bytes / 8 TB/s), and its fraction of the measured time."""
    import torch
    import synth
    import paper_2411_16025_amd as G

    dev = torch.device("cuda:0")
    n, f_in, hid, C = 2_449_029, 100, 256, 47
    K3 = 2 * hid + 4  # GraphSAGE: [Y | Z | 1 0 0 0] of a hidden layer, rows of 544 floats
    rnd = lambda seed, r, c: torch.from_numpy(synth.uniform(seed, r, c)).to(dev)  # noqa: E731
    X = rnd(3100, n, f_in)
    H1 = rnd(3101, n, hid)
    W1 = rnd(3102, f_in, hid)
    W2p = rnd(3103, hid, 48)
    dZ2p = rnd(3104, n, 48)
    dZ1 = rnd(3105, n, hid)
    Cs = rnd(3106, n, (K3 + 31) // 32 * 32)[:, :K3]
    Ws = rnd(3107, K3, hid)
    W3p = rnd(3108, K3, 48)
    out_nh = torch.empty((n, hid), device=dev)
    out_nc = torch.empty((n, 48), device=dev)
    NN, NT, TN = G.GCN_GEMM_NN, G.GCN_GEMM_NT, G.GCN_GEMM_TN
    cases = [
        ("gcn Z1 = X W1", NN, X, W1, out_nh, (n, hid, f_in)),
        ("gcn Z2 = H1 W2", NN, H1, W2p[:, :C], out_nc[:, :C], (n, C, hid)),
        ("gcn dH1 = dZ2 W2^T", NT, dZ2p[:, :C], W2p[:, :C], out_nh, (n, hid, C)),
        ("gcn dW2 = H1^T dZ2", TN, H1, dZ2p[:, :C], None, (hid, C, n)),
        ("gcn dW1 = X^T dZ1", TN, X, dZ1, None, (f_in, hid, n)),
        ("sage O2 = C2 W (K=516)", NN, Cs, Ws, out_nh, (n, hid, K3)),
        ("sage O3 = C3 W3 (K=516)", NN, Cs, W3p[:, :C], out_nc[:, :C], (n, C, K3)),
        ("sage dW2 = C2^T dO2", TN, Cs, dZ1, None, (K3, hid, n)),
    ]
    res = {}
    tot_roof = tot_ms = 0.0
    for name, op, A, B, Cout, (M, N, K) in cases:
        fn = lambda: G.gcn_gemm_f32(op, A, B, C=Cout)  # noqa: E731
        for _ in range(max(args.warmup, 1)):
            fn()
        torch.cuda.synchronize()
        times = []
        for _ in range(args.steps):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev[0].record()
            fn()
            ev[1].record()
            ev[1].synchronize()
            times.append(ev[0].elapsed_time(ev[1]))
        ms = float(np.median(times))
        flops = 2.0 * M * N * K
        nbytes = 4.0 * (M * K + K * N + M * N)
        t_roof = max(flops / (FP32_MFMA_PEAK_TFLOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9)) * 1e3
        res[name] = {"M": M, "N": N, "K": K, "ms": round(ms, 4),
                     "TFLOPs": round(flops / (ms * 1e-3) / 1e12, 1),
                     "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "bound": "mfma" if flops / (FP32_MFMA_PEAK_TFLOPS * 1e12) >= nbytes / (HBM_PEAK_GBS * 1e9) else "hbm",
                     "roofline_ms": round(t_roof, 4), "frac": round(t_roof / ms, 4)}
        tot_roof += t_roof
        tot_ms += ms
        log("%-26s %8.3f ms  roofline %.3f ms  %.0f%%" % (name, ms, t_roof, 100 * t_roof / ms))
    dom = max(res, key=lambda k: res[k]["ms"])
    d = res[dom]
    out = {
        "metric": "fp32 GEMMs of the training steps: roofline time / measured time",
        "value": round(tot_roof / tot_ms, 4), "unit": "fraction", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(tot_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "training-step products at 2,449,029 rows (F_in 100, hidden 256, "
                               "47 classes)"},
        "products": res,
        "roofline": {"bound": d["bound"], "kernel": dom,
                     "achieved": d["TFLOPs"] if d["bound"] == "mfma" else d["GBps"],
                     "peak": FP32_MFMA_PEAK_TFLOPS if d["bound"] == "mfma" else HBM_PEAK_GBS,
                     "unit": "TFLOP/s" if d["bound"] == "mfma" else "GB/s", "frac": d["frac"],
                     "traffic": None},
    }
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the aggregation path runs and is timed on a "
              "single MI355X (sharding across GPUs is designed, not implemented); "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy_mib > 0:
        import torch
        a = torch.empty(args.calibrate_copy_mib << 18, dtype=torch.float32, device="cuda:0")
        a.fill_(1.0)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        torch.mul(a, 1.0, out=b)  # one elementwise kernel: reads and writes exactly this size
        torch.cuda.synchronize()
        del a, b
        log("copy calibration: %d MiB" % args.calibrate_copy_mib)
    if args.workload == "gcn_step":
        run_gcn_step(args)
        return
    if args.workload == "prepost":
        run_prepost(args)
        return
    if args.workload == "sage_step":
        run_sage_step(args)
        return
    if args.workload == "producer":
        run_producer(args)
        return
    if args.workload == "gemm":
        run_gemm(args)
        return

    import torch
    import synth
    import paper_2411_16025_amd as G

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    G.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t0 = time.time()
    w = {"rmat24_q8": synth.rmat24_q8, "rmat24": synth.rmat24, "rmat20": synth.rmat20, "er4096": synth.er_4096,
         "product": synth.product_like, "partition": synth.partition_111m,
         "perm22": synth.perm22}[args.workload]()
    k_seed = {"rmat24_q8": 5, "rmat24": 5, "rmat20": 2, "er4096": 1, "product": 3, "partition": 4,
              "perm22": 6}[args.workload]
    log("generated %s: %d edges in %.1f s" % (w.name, len(w.src), time.time() - t0))
    F = w.F
    q8 = w.n_local_cols is not None

    # ---- build (once per graph; not part of a step) ----
    src_d = torch.from_numpy(w.src).to(dev)
    dst_d = torch.from_numpy(w.dst).to(dev)
    torch.cuda.synchronize()
    tb = time.time()
    g = G.gcn_build_csr(w.n_rows, w.n_cols, src_d, dst_d, w.flags)
    torch.cuda.synchronize()
    build_ms = (time.time() - tb) * 1e3
    del src_d, dst_d
    deg_d = torch.from_numpy(w.deg).to(dev) if w.deg is not None else None
    torch.cuda.synchronize()
    tn = time.time()
    G.gcn_normalize(g, deg_d)
    torch.cuda.synchronize()
    norm_ms = (time.time() - tn) * 1e3
    log("built graph: nnz=%d build %.1f ms normalize %.1f ms" % (g.nnz, build_ms, norm_ms))

    # ---- inputs (host generation, then HBM resident) ----
    tx = time.time()
    gen = synth.normal if q8 else synth.uniform
    X_h = gen(3000 + k_seed, w.n_cols, F)
    X = torch.from_numpy(X_h).to(dev)
    G_h = gen(4000 + k_seed, w.n_rows, F)
    Gd = torch.from_numpy(G_h).to(dev)
    if args.no_cpu_baseline:
        X_h = G_h = None
    nlc = w.n_local_cols
    bits = args.halo_bits if q8 else 8
    if q8 and bits == 8:
        QX, ZX, SX = G.gcn_quantize_rows_u8(X[nlc:], paired=True)
        QG, ZG, SG = G.gcn_quantize_rows_u8(Gd[nlc:], paired=True)
    elif q8:
        QX, ZX, SX = G.gcn_layernorm_quantize(X[nlc:], bits=bits, layernorm=False)
        QG, ZG, SG = G.gcn_layernorm_quantize(Gd[nlc:], bits=bits, layernorm=False)
    if q8:
        X_loc, G_loc = X[:nlc], Gd[:nlc]
    Y = torch.empty((w.n_rows, F), dtype=torch.float32, device=dev)
    dX = torch.empty((w.n_cols, F), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    log("inputs ready in %.1f s" % (time.time() - tx))

    if q8:
        def fwd():
            G.gcn_aggregate_fwd_q8halo(g, nlc, X_loc, QX, ZX, SX, Y=Y, F=F, bits=bits)

        def bwd():
            G.gcn_aggregate_fwd_q8halo(g, nlc, G_loc, QG, ZG, SG, Y=dX, use_csc=True, F=F,
                                       bits=bits)
    else:
        def fwd():
            G.gcn_aggregate_fwd(g, X, Y=Y)

        def bwd():
            G.gcn_aggregate_bwd(g, Gd, dX=dX)

    def step():
        fwd()
        bwd()

    # ---- timed region ----
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ts = time.time()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    step_ms = (time.time() - ts) * 1e3 / args.steps
    log("timed %d steps: %.3f ms/step" % (args.steps, step_ms))

    # fwd / bwd split, HIP events on the stream the library launches on
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    fwd_ms = bwd_ms = 0.0
    per_step = []
    for _ in range(args.steps):
        ev[0].record()
        fwd()
        ev[1].record()
        bwd()
        ev[2].record()
        ev[2].synchronize()
        fwd_ms += ev[0].elapsed_time(ev[1]) / args.steps
        bwd_ms += ev[1].elapsed_time(ev[2]) / args.steps
        per_step.append(ev[0].elapsed_time(ev[2]))

    # Launch-bound graphs: the forward captured once as a HIP graph (the
    # no-allocation entry, whose partial rows live in the library's fixed
    # array) and replayed back to back, against the same number of eager
    # forwards back to back (HIP events around each series).
    graph_fwd = None
    if not q8 and w.n_rows <= (1 << 16):
        def series(fn):
            for _ in range(max(args.warmup, 1)):
                fn()
            torch.cuda.synchronize()
            e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            e[0].record()
            for _ in range(args.steps):
                fn()
            e[1].record()
            e[1].synchronize()
            return e[0].elapsed_time(e[1]) / args.steps

        try:
            G.gcn_aggregate_fwd_noalloc(g, X, Y)
            torch.cuda.synchronize()
            side = torch.cuda.Stream()  # default priority
            side.wait_stream(torch.cuda.current_stream())
            cg = torch.cuda.CUDAGraph()
            with torch.cuda.graph(cg, stream=side):
                G.gcn_aggregate_fwd_noalloc(g, X, Y)
            torch.cuda.synchronize()
            graph_fwd = {"eager_ms": round(series(fwd), 4), "graph_replay_ms": round(series(cg.replay), 4),
                         "note": "forward only, back to back; the graph replays the no-allocation "
                                 "entry captured once"}
            del cg
        except G.GcnError as e:  # a plan beyond the fixed array: no graph figure
            log("no graph replay: %s" % e)

    # per-kernel durations (events around every launch, separate from the timed region)
    G.gcn_profile_enable(True)
    for _ in range(args.profile_steps):
        step()
    torch.cuda.synchronize()
    prof = G.gcn_profile_read()
    G.gcn_profile_enable(False)

    # ---- traffic model ----
    bins_f = G.gcn_graph_bins(g, 0, halo_from=nlc if q8 else -1)
    bins_b = G.gcn_graph_bins(g, 1, halo_from=nlc if q8 else -1)

    def pass_bytes(bins):
        rows = sum(b["rows"] for b in bins)
        ents = sum(b["entries"] for b in bins)
        halo = sum(b["halo_entries"] for b in bins)
        return model_bytes(rows, ents, halo, F, bits) + 8, ents, halo

    Bf, nnz_f, halo_f = pass_bytes(bins_f)
    Bb, nnz_b, _ = pass_bytes(bins_b)
    # compulsory traffic of the step: CSR/CSC, each input row once, the outputs
    def read_once(n_in):  # input rows [0, n_in) of one pass, halo rows quantized
        n_loc = min(nlc, n_in) if q8 else n_in
        return 4 * F * n_loc + (code_bytes(F, bits) + 8) * (n_in - n_loc)
    compulsory = sum(8 * (r + 1) + 8 * e + 4 * F * r + read_once(n_in)
                     for r, e, n_in in ((w.n_rows, nnz_f, w.n_cols), (w.n_cols, nnz_b, w.n_rows)))
    value = (Bf + Bb) / (step_ms * 1e-3) / 1e9
    ef_per_s = (nnz_f + nnz_b) * F / (step_ms * 1e-3)

    # counted fabric bytes of every aggregation kernel (committed summary of
    # this workload, taken on the current sources), per pass
    counted = read_counters(counters_path(args.workload, bits))
    counted_step = None
    if counted is not None:
        counted_step = sum(f + wr for f, wr, _ in counted["rows"].values())

    # dominant kernel and its roofline figures
    agg = {k: v for k, v in prof.items() if k in KERNEL_CLASSES}
    roofline = None
    if agg:
        dom = max(agg, key=lambda k: agg[k][1])
        launches, tot_ms = agg[dom]
        per_launch_bytes = 0.5 * sum(
            model_bytes(b["rows"], b["entries"], b["halo_entries"], F, bits)
            for bins in (bins_f, bins_b) for c, b in enumerate(bins) if c in KERNEL_CLASSES[dom])
        avg_ms = tot_ms / launches
        achieved = per_launch_bytes / (avg_ms * 1e-3) / 1e9
        traffic = l2_hit = None
        if counted is not None:
            per_op = [counted["rows"].get((dom, op)) for op in ("fwd", "bwd")]
            if all(per_op):  # one launch per pass: the average of the two passes
                traffic = 0.5 * sum(f + wr for f, wr, _ in per_op)
                l2_hit = round(0.5 * sum(h for _, _, h in per_op), 4)
        roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": traffic, "model": MODEL_NOTE,
                    "bytes_per_launch": int(per_launch_bytes), "avg_launch_ms": round(avg_ms, 4)}
        if traffic is not None:
            # the counted bytes over the same launch time: the rate the memory system delivered
            tr = traffic / (avg_ms * 1e-3) / 1e9
            roofline.update({"traffic_GBps": round(tr, 1),
                             "traffic_frac": round(tr / HBM_PEAK_GBS, 4), "l2_hit": l2_hit})

    # every aggregation kernel against the same model, per pass (one forward
    # and one transposed pass per profiled step; k_tiny is two launches a pass)
    kernel_rooflines = {}
    n_pass = 2 * max(args.profile_steps, 1)
    for k, (launches, tot_ms) in agg.items():
        if not KERNEL_CLASSES.get(k) or launches == 0:
            continue
        kb = 0.5 * sum(model_bytes(b["rows"], b["entries"], b["halo_entries"], F, bits)
                       for bins in (bins_f, bins_b) for c, b in enumerate(bins)
                       if c in KERNEL_CLASSES[k])
        ms = tot_ms / n_pass
        kernel_rooflines[k] = {"ms_per_pass": round(ms, 4), "modeled_GB": round(kb / 1e9, 2),
                               "GBps": round(kb / (ms * 1e-3) / 1e9, 1),
                               "frac": round(kb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "n_rows": w.n_rows, "n_cols": w.n_cols, "nnz": g.nnz,
                   "F": F, "halo_rows": (w.n_cols - nlc) if q8 else 0,
                   "halo_storage": ("%s codes + fp32 (min, scale) pair per row"
                                    % ("u8" if bits == 8 else "2-bit packed")) if q8 else None,
                   "step": "fwd A_hat x + bwd A_hat^T g"
                           + (" with fused %d-bit halo dequant" % bits if q8 else "")},
        "modeled_frac": round(value / HBM_PEAK_GBS, 4), "model": MODEL_NOTE,
        "edge_features_per_s": float("%.4g" % ef_per_s),
        "fwd_ms": round(fwd_ms, 4), "bwd_ms": round(bwd_ms, 4),
        "fwd_graph": graph_fwd,
        # per pass: modeled and counted rates over the event-timed pass
        "per_op": {op: {
            "ms": round(ms, 4), "modeled_GBps": round(B / (ms * 1e-3) / 1e9, 1),
            "modeled_frac": round(B / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "edge_features_per_s": float("%.4g" % (nz * F / (ms * 1e-3))),
            "counted_GBps": None if counted is None else round(
                sum(f + wr for (k, o), (f, wr, _) in counted["rows"].items() if o == op)
                / (ms * 1e-3) / 1e9, 1)}
            for op, ms, B, nz in (("fwd", fwd_ms, Bf, nnz_f), ("bwd", bwd_ms, Bb, nnz_b))},
        "step_ms_median": round(float(np.median(per_step)), 4),
        "step_ms_min": round(float(np.min(per_step)), 4),
        # the L2-to-fabric bytes the kernels moved (counters; Infinity Cache
        # hits included, so an upper bound on HBM bytes) over the step time
        "counted": None if counted_step is None else {
            "GBps": round(counted_step / (step_ms * 1e-3) / 1e9, 1),
            "frac": round(counted_step / (step_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "bytes_per_step": int(counted_step), "source": counted["path"],
            "fetch_scale": counted["fetch_scale"]},
        # every input row read once (a gather of repeated rows cannot reach it)
        "compulsory_GBps": round(compulsory / (step_ms * 1e-3) / 1e9, 1),
        "compulsory_frac": round(compulsory / (step_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "modeled_bytes_per_step": int(Bf + Bb),
        "build_ms": round(build_ms, 1), "normalize_ms": round(norm_ms, 1),
        "kernels_ms_per_step": {k: round(v[1] / max(args.profile_steps, 1), 4)
                                for k, v in prof.items()},
        "row_classes": [[b["first_len"], b["last_len"], b["rows"], b["entries"]] for b in bins_f],
        "roofline": roofline,
        "kernel_rooflines": kernel_rooflines,
    }

    # ---- CPU baseline: the oracle on a bounded sample of the same workload ----
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, X_h, nlc, F, args.cpu_target_s / 2, bits,
                                           args.cpu_threads, G_h=G_h)
    print(json.dumps(out), flush=True)


def cpu_baseline(w, X_h, nlc, F, target_s, bits=8, threads=0, G_h=None):
    """The oracle (fp64 accumulation, OpenMP over rows) on a bounded sample of
    the workload: the forward pass over rows of A and, with G_h, the
    transposed pass over rows of A^T, about target_s seconds each. Small
    graphs run whole, repeatedly (median of three batches)."""
    import oracle
    import synth

    if threads > 0:
        oracle.set_num_threads(threads)
    q8 = nlc is not None

    def quant(M):
        if not q8:
            return None
        return oracle.quantize_rows(M[nlc:]) if bits == 8 else oracle.quantize_rows_bits(M[nlc:], bits)

    def one_pass(M, transpose):
        n_major = w.n_cols if transpose else w.n_rows
        order = synth.permutation(778 + int(transpose), n_major)  # rows in a seeded random order
        Q = quant(M)

        def run(n_sel, reps=1):
            sel = np.sort(order[:n_sel]).astype(np.int32)
            ptr, idx = oracle.rows_of(w.n_rows, w.n_cols, w.src, w.dst, w.flags, sel,
                                      transpose=transpose)
            val = np.ones(len(idx), np.float32)  # unit weights: the cost does not depend on them
            t = time.time()
            for _ in range(reps):
                if q8 and bits == 8:
                    oracle.spmm_q8(ptr, idx, val, nlc, M[:nlc], *Q)
                elif q8:
                    oracle.spmm_qbits(ptr, idx, val, nlc, M[:nlc], *Q, F, bits)
                else:
                    oracle.spmm(ptr, idx, val, M)
            dt = time.time() - t
            halo = int(np.sum(idx >= nlc)) if q8 else 0
            return dt, reps * len(sel), reps * len(idx), reps * halo

        n = min(n_major, max(64, n_major // 400))
        dt, rows, ents, halo = run(n)
        for _ in range(4):  # grow the sample until it is about target_s of oracle work
            if dt >= 0.6 * target_s or n >= n_major:
                break
            n = int(min(n_major, n * min(8.0, target_s / max(dt, 1e-3))))
            dt, rows, ents, halo = run(n)
        reps, batches = 1, 1
        if dt < 0.6 * target_s:  # the whole matrix is quick: repeat it, median of three batches
            reps = int(min(100000, max(2, target_s / 3 / max(dt, 1e-4))))
            batches = 3
            timed = [run(n, reps) for _ in range(batches)]
            dt, rows, ents, halo = sorted(timed)[1]
        B = model_bytes(rows, ents, halo, F, bits)
        return {"GBps": round(B / dt / 1e9, 3), "edge_features_per_s": float("%.4g" % (ents * F / dt)),
                "seconds": round(dt, 2), "bytes": B, "entries": ents,
                "sample": "%d %s (%d entries)%s" % (
                    rows // reps, "rows of A^T" if transpose else "rows of A", ents // reps,
                    ", repeated %d times (median of %d such batches)" % (reps, batches)
                    if reps > 1 else "")}

    fwd = one_pass(X_h, False)
    bwd = one_pass(G_h, True) if G_h is not None else None
    parts = [p for p in (fwd, bwd) if p is not None]
    secs = sum(p["seconds"] for p in parts)
    B = sum(p["bytes"] for p in parts)
    ents = sum(p["entries"] for p in parts)
    cpu = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    for p in parts:
        del p["bytes"], p["entries"]
    out = {"value": round(B / secs / 1e9, 3), "unit": "GB/s", "cores": oracle.num_threads(),
           "cpu_model": cpu, "host_cpus": os.cpu_count(), "kind": "oracle",
           "edge_features_per_s": float("%.4g" % (ents * F / secs)), "seconds": round(secs, 2),
           "fwd": fwd, "bwd": bwd,
           "sample": "fp64-accumulating aggregation%s of %s over uniformly sampled rows: forward %s%s;"
                     " unit weights; structure of the sampled rows built by the oracle from the edge "
                     "list beforehand (untimed)"
                     % (", %d-bit halo dequantized" % bits if q8 else "", w.name, fwd["sample"],
                        "; transposed %s" % bwd["sample"] if bwd else "")}
    return out


if __name__ == "__main__":
    main()
