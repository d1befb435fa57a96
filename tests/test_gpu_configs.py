"""GPU parity on the five workloads at full size.

ER-4096 and RMAT-20 are compared in full (every entry of the structure, every
output element). The product-shaped graph, the 14M x 20M partition and the
RMAT-24 graph with uint8 halo rows are compared on sampled output rows that
the oracle computes one by one from the edge list: uniformly drawn rows plus
the rows with the most entries (they run through the chunked long-row path).
Structure and values of the sampled rows are compared bit for bit, outputs
within 1e-5 * S.
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


def sample_rows(w, n_major, transpose, k=48, hubs=2, seed=0):
    """k uniform rows plus the `hubs` nodes that occur most often in the edge list."""
    rng = np.random.default_rng(seed)
    sel = rng.choice(n_major, size=min(k, n_major), replace=False)
    ends = w.src if transpose else w.dst
    if w.flags & synth.SYMMETRIZE:
        cnt = np.bincount(w.src, minlength=n_major) + np.bincount(w.dst, minlength=n_major)
    else:
        cnt = np.bincount(ends, minlength=n_major)
    top = np.argsort(-cnt, kind="stable")[:hubs]
    return np.unique(np.concatenate([sel, top])).astype(np.int32)


def check_sampled(G, g, w, sel, transpose, Xh, Yd, Q=None, nlc=None):
    """Structure, values and outputs of the sampled rows against the oracle."""
    import torch
    ptr, idx, val = oracle.sampled(w.n_rows, w.n_cols, w.src, w.dst, w.flags, sel,
                                   transpose=transpose, deg=w.deg)
    gptr, gidx, gval = G.gcn_graph_export(g, 1 if transpose else 0)
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
    got = host(Yd[torch.from_numpy(sel.astype(np.int64)).to(Yd.device)])
    assert_close(got, ref, S, what="sampled rows (transpose=%s)" % transpose)
    return int(ptr[-1])


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


def test_product_like_sampled(G):
    import torch
    note("config product-like sampled")
    w = synth.product_like()
    g = build(G, w)
    for F in (256, 47):
        X = synth.normal(3003, w.n_cols, F)
        Y = G.gcn_aggregate_fwd(g, dev(X))
        sel = sample_rows(w, w.n_rows, False, seed=F)
        check_sampled(G, g, w, sel, False, X, Y)
        dX = G.gcn_aggregate_bwd(g, dev(X))
        check_sampled(G, g, w, sel, True, X, dX)
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
    check_sampled(G, g, w, sample_rows(w, w.n_rows, False), False, X, Y)
    del Y, X
    Gm = synth.uniform(4004, w.n_rows, w.F)
    dX = G.gcn_aggregate_bwd(g, dev(Gm))
    # backward rows are columns of A: local and halo nodes alike
    check_sampled(G, g, w, sample_rows(w, w.n_cols, True, seed=1), True, Gm, dX)
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
    sel = sample_rows(w, w.n_rows, False)
    check_sampled(G, g, w, sel, False, X, Y, Q=(Q, Z, S), nlc=nlc)
    dX = G.gcn_aggregate_fwd_q8halo(g, nlc, Xd, dev(Q), zs[:, 0], zs[:, 1], use_csc=True)
    check_sampled(G, g, w, sel, True, X, dX, Q=(Q, Z, S), nlc=nlc)
    del Y, dX, Xd
    g.free()
    gc.collect()
    torch.cuda.empty_cache()
