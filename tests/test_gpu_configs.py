"""GPU parity on the five workloads at full size.

ER-4096 and RMAT-20 are compared in full (every entry of the structure, every
output element). The product-shaped graph, the 14M x 20M partition and the
RMAT-24 graph with uint8 halo rows are compared on a stratified sample of
output rows that the oracle computes one by one from the edge list:

  * up to 200 rows from every row-length class the kernels distinguish
    (empty, 1, 2, 3-4, 5-8, 9-16, 17-32, 33-48 entries);
  * the column-blocked rows (over 48 entries on matrices of 2^20 or more
    columns) by powers of two of their length, up to 300 per octave (their
    segment and piece counts follow the length), at least 2,000 in all, and
    every row longer than 65,536 entries;
  * the blocked rows whose columns span the narrowest range and those
    confined closest to the first and to the last column block;
  * with halo columns, up to 200 rows whose entries are all halo columns and
    200 with none.

Structure and values of the sampled rows are compared bit for bit, outputs
within 1e-5 * S; the largest err/S of each stratum is printed.
"""

import gc

import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_close, dev, host, note

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2411_16025_amd as pkg
    pkg.lib()
    return pkg


def build(G, w):
    import torch
    g = G.gcn_build_csr(w.n_rows, w.n_cols, dev(w.src), dev(w.dst), w.flags)
    G.gcn_normalize(g, dev(w.deg) if w.deg is not None else None)
    torch.cuda.synchronize()
    return g


LEN_CLASSES = [(0, 0), (1, 1), (2, 2), (3, 4), (5, 8), (9, 16), (17, 32), (33, 48)]


def stratified_rows(ptr, idx, halo_from=None, per_class=200, per_octave=300, seed=0):
    """Sampled major ids of a matrix (exported ptr/idx) and a stratum name
    for each, as described in the module docstring."""
    rng = np.random.default_rng(seed)
    lens = np.diff(ptr)
    picks = []

    def take(name, cand, k):
        cand = np.asarray(cand)
        if len(cand) > k:
            cand = rng.choice(cand, size=k, replace=False)
        picks.append((name, cand))

    for lo, hi in LEN_CLASSES:
        take("len %d-%d" % (lo, hi), np.flatnonzero((lens >= lo) & (lens <= hi)), per_class)
    lo, hi = 49, 64
    while lo <= lens.max():
        take("len %d-%d" % (lo, hi), np.flatnonzero((lens >= lo) & (lens <= hi)), per_octave)
        lo, hi = hi + 1, 2 * hi
    take("len > 65536", np.flatnonzero(lens > 65536), 10 ** 9)
    long_rows = np.flatnonzero(lens > 48)
    if len(long_rows):
        first = idx[ptr[long_rows]]
        last = idx[ptr[long_rows + 1] - 1]
        take("narrowest span", long_rows[np.argsort(last - first, kind="stable")[:10]], 10)
        take("closest to the last block", long_rows[np.argsort(-first, kind="stable")[:10]], 10)
        take("closest to the first block", long_rows[np.argsort(last, kind="stable")[:10]], 10)
    if halo_from is not None:
        nz = np.flatnonzero(lens > 0)
        first = idx[ptr[nz]]
        last = idx[ptr[nz + 1] - 1]
        take("all halo", nz[first >= halo_from], per_class)
        take("no halo", nz[last < halo_from], per_class)
    sel = np.unique(np.concatenate([c for _, c in picks])).astype(np.int32)
    strata = [(name, np.searchsorted(sel, c)) for name, c in picks if len(c)]
    n_blocked = int(np.sum(lens[sel] > 48))
    return sel, strata, n_blocked


def check_sampled(G, g, w, transpose, Xh, Yd, Q=None, nlc=None, halo_from=None, seed=0):
    """Structure, values and outputs of a stratified sample of rows against
    the oracle; returns (rows, entries, blocked rows) of the sample."""
    import torch
    gptr, gidx, gval = G.gcn_graph_export(g, 1 if transpose else 0)
    sel, strata, n_blocked = stratified_rows(gptr, gidx, halo_from=halo_from, seed=seed)
    ptr, idx, val = oracle.sampled(w.n_rows, w.n_cols, w.src, w.dst, w.flags, sel,
                                   transpose=transpose, deg=w.deg)
    for i, r in enumerate(sel):
        a, b = gptr[r], gptr[r + 1]
        assert np.array_equal(gidx[a:b], idx[ptr[i]:ptr[i + 1]]), "structure of row %d" % r
        assert np.array_equal(gval[a:b].view(np.uint32), val[ptr[i]:ptr[i + 1]].view(np.uint32)), \
            "values of row %d" % r
    del gidx, gval
    if Q is None:
        ref, S = oracle.spmm(ptr, idx, val, Xh)
    else:
        ref, S = oracle.spmm_q8(ptr, idx, val, nlc, Xh[:nlc], *Q)
    got = host(Yd[torch.from_numpy(sel.astype(np.int64)).to(Yd.device)]).astype(np.float64)
    ratio = np.abs(got - ref) / np.maximum(S, 1e-300)
    note("sampled %d rows (%d entries, %d column-blocked), transpose=%s; max err/S per stratum: %s"
         % (len(sel), int(ptr[-1]), n_blocked, transpose,
            "; ".join("%s (%d): %.1e" % (name, len(ix), ratio[ix].max()) for name, ix in strata)))
    assert_close(got, ref, S, what="sampled rows (transpose=%s)" % transpose)
    return len(sel), int(ptr[-1]), n_blocked


def test_er4096_full(G):
    note("config er4096 full")
    w = synth.er_4096()
    og = oracle.Graph(w.n_rows, w.n_cols, w.src, w.dst, w.flags)
    g = build(G, w)
    for which, (p, i, v) in ((0, (og.csr_ptr, og.csr_idx, og.csr_val)),
                             (1, (og.csc_ptr, og.csc_idx, og.csc_val))):
        ptr, idx, val = G.gcn_graph_export(g, which)
        assert np.array_equal(ptr, p) and np.array_equal(idx, i)
        assert np.array_equal(val.view(np.uint32), v.view(np.uint32))
    X = synth.uniform(3001, w.n_cols, w.F)
    Gm = synth.uniform(4001, w.n_rows, w.F)
    assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="er4096 fwd")
    assert_close(host(G.gcn_aggregate_bwd(g, dev(Gm))), *og.bwd(Gm), what="er4096 bwd")


def test_rmat20_full(G):
    note("config rmat20 full")
    w = synth.rmat20()
    og = oracle.Graph(w.n_rows, w.n_cols, w.src, w.dst, w.flags)
    g = build(G, w)
    assert g.nnz == og.nnz
    ptr, idx, val = G.gcn_graph_export(g, 0)
    assert np.array_equal(ptr, og.csr_ptr) and np.array_equal(idx, og.csr_idx)
    assert np.array_equal(val.view(np.uint32), og.csr_val.view(np.uint32))
    del ptr, idx, val
    X = synth.uniform(3002, w.n_cols, w.F)
    assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="rmat20 fwd")
    Gm = synth.uniform(4002, w.n_rows, w.F)
    assert_close(host(G.gcn_aggregate_bwd(g, dev(Gm))), *og.bwd(Gm), what="rmat20 bwd")


def test_rmat20_bf16_default_plan(G):
    # bf16 input on a matrix of 2^20 columns, so the default plan column-blocks
    # the long rows: every output element against the oracle on the
    # bf16-rounded input (1e-5 * S) and on the fp32 input (1e-2 * S)
    import torch
    from gpu_util import bf16_bits, bf16_round
    note("config rmat20 bf16 full")
    w = synth.rmat20()
    og = oracle.Graph(w.n_rows, w.n_cols, w.src, w.dst, w.flags)
    g = build(G, w)
    assert G.gcn_graph_bins(g, 0)[-1]["rows"] > 0, "no column-blocked rows"
    X = synth.uniform(3002, w.n_cols, w.F)
    Xb = torch.from_numpy(bf16_bits(X).view(np.int16)).view(torch.bfloat16).to("cuda:0")
    Xr = bf16_round(X)
    Y = host(G.gcn_aggregate_fwd(g, Xb))
    assert_close(Y, *og.fwd(Xr), what="rmat20 bf16 fwd vs rounded input")
    assert_close(Y, *og.fwd(X), rel=1e-2, what="rmat20 bf16 fwd vs fp32 input")
    del Y
    dX = host(G.gcn_aggregate_bwd(g, Xb))
    assert_close(dX, *og.bwd(Xr), what="rmat20 bf16 bwd vs rounded input")
    assert_close(dX, *og.bwd(X), rel=1e-2, what="rmat20 bf16 bwd vs fp32 input")
    g.free()


def test_product_like_sampled(G):
    import torch
    note("config product-like sampled")
    w = synth.product_like()
    g = build(G, w)
    for F in (256, 47):
        X = synth.normal(3003, w.n_cols, F)
        Y = G.gcn_aggregate_fwd(g, dev(X))
        _, _, nb = check_sampled(G, g, w, False, X, Y, seed=F)
        assert nb >= 2000
        dX = G.gcn_aggregate_bwd(g, dev(X))
        check_sampled(G, g, w, True, X, dX, seed=F + 1)
        del Y, dX
        torch.cuda.empty_cache()
    g.free()
    gc.collect()


def test_partition_sampled(G):
    import torch
    note("config partition 14M x 20M sampled")
    w = synth.partition_111m()
    g = build(G, w)
    assert g.n_rows == 14_000_000 and g.n_cols == 20_000_000
    X = synth.uniform(3004, w.n_cols, w.F)
    Y = G.gcn_aggregate_fwd(g, dev(X))
    _, _, nb = check_sampled(G, g, w, False, X, Y, halo_from=w.n_rows)
    assert nb >= 2000
    del Y, X
    Gm = synth.uniform(4004, w.n_rows, w.F)
    dX = G.gcn_aggregate_bwd(g, dev(Gm))
    # backward rows are columns of A: local and halo nodes alike
    check_sampled(G, g, w, True, Gm, dX, seed=1)
    del dX
    g.free()
    gc.collect()
    torch.cuda.empty_cache()


def test_rmat24_q8_sampled(G):
    import torch
    note("config rmat24 q8 halo sampled")
    w = synth.rmat24_q8()
    g = build(G, w)
    nlc = w.n_local_cols
    X = synth.normal(3005, w.n_cols, w.F)
    Q, Z, S = oracle.quantize_rows(X[nlc:])
    Xd = dev(X[:nlc])
    zs = dev(np.stack([Z, S], axis=1))
    Y = G.gcn_aggregate_fwd_q8halo(g, nlc, Xd, dev(Q), zs[:, 0], zs[:, 1])
    _, _, nb = check_sampled(G, g, w, False, X, Y, Q=(Q, Z, S), nlc=nlc, halo_from=nlc)
    assert nb >= 2000
    dX = G.gcn_aggregate_fwd_q8halo(g, nlc, Xd, dev(Q), zs[:, 0], zs[:, 1], use_csc=True)
    check_sampled(G, g, w, True, X, dX, Q=(Q, Z, S), nlc=nlc, halo_from=nlc, seed=1)
    del Y, dX, Xd
    g.free()
    gc.collect()
    torch.cuda.empty_cache()
