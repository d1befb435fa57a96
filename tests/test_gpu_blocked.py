"""GPU parity of the column-blocked pieces of long rows against the oracle.

Rows of at least GCN_BLOCKED_MIN entries are cut at multiples of the column
block width into pieces of at most GCN_PIECE_MAX entries, run block by
block, and summed from partial rows. By default only matrices with 2^20 or
more columns are blocked; these tests force the path on small graphs through
the plan's environment bounds (read when the graph is built) and compare with
the oracle within 1e-5 * S per element (S: the oracle's sum of |terms|).
"""

import contextlib
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_close, bf16_bits, bf16_round, dev, host, note

pytestmark = pytest.mark.gpu

SYM, LOOPS = synth.SYMMETRIZE, synth.ADD_SELF_LOOPS


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2411_16025_amd as pkg
    pkg.lib()
    return pkg


@contextlib.contextmanager
def plan_env(**kv):
    old = {k: os.environ.get(k) for k in kv}
    os.environ.update({k: str(v) for k, v in kv.items()})
    try:
        yield
    finally:
        for k, v in old.items():
            if v is None:
                del os.environ[k]
            else:
                os.environ[k] = v


def build(G, n_rows, n_cols, src, dst, flags, deg=None, **env):
    with plan_env(GCN_BLOCK_MIN_COLS=0, **env):
        g = G.gcn_build_csr(n_rows, n_cols, dev(src), dev(dst), flags)
    G.gcn_normalize(g, dev(deg) if deg is not None else None)
    return g


def rows_with_lengths(lengths, n_cols, seed, lo=0, hi=None):
    """Row i has lengths[i] distinct columns drawn from [lo, hi)."""
    hi = n_cols if hi is None else hi
    src, dst = [], []
    for i, L in enumerate(lengths):
        cols = lo + synth.permutation(seed + i, hi - lo)[:L]
        src.append(cols.astype(np.int32))
        dst.append(np.full(L, i, np.int32))
    return np.concatenate(src), np.concatenate(dst)


def check_bins(G, g, which=0):
    bins = G.gcn_graph_bins(g, which)
    assert len(bins) == 10
    return bins


@pytest.mark.parametrize("blocks,piece,seg", [(7, 16, 0), (64, 256, 0), (256, 31, 0), (2, 511, 0),
                                              (64, 32, 40), (7, 64, 100), (128, 256, 7)])
def test_rmat_blocked_fwd_bwd(G, blocks, piece, seg):
    note("blocked rmat blocks=%d piece=%d segment=%d" % (blocks, piece, seg))
    n = 1 << 14
    src, dst = synth.rmat_edges(301, n, 24 * n, perm_seed=302)
    og = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    # chunk-table rows (41 .. 299 entries, several 64-entry chunks) next to
    # the blocked ones
    g = build(G, n, n, src, dst, SYM | LOOPS, GCN_COL_BLOCKS=blocks, GCN_PIECE_MAX=piece,
              GCN_BLOCKED_MIN=300, GCN_MEDIUM_MAX=40, GCN_CHUNK_LEN=64, GCN_SEGMENT_MIN=seg)
    bins = check_bins(G, g)
    assert bins[9]["rows"] > 20 and bins[9]["first_len"] == 300
    assert bins[8]["rows"] > 20 and (bins[8]["first_len"], bins[8]["last_len"]) == (41, 299)
    for F in (4, 47, 128, 256, 1030):
        X = synth.uniform(303 + F, n, F)
        assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="fwd F=%d" % F)
    Gm = synth.uniform(310, n, 100)
    assert_close(host(G.gcn_aggregate_bwd(g, dev(Gm))), *og.bwd(Gm), what="bwd")


def test_blocked_rows_at_length_and_block_edges(G):
    # lengths around blocked_min and piece multiples; one row confined to a
    # single column block (one segment, several pieces), one to the last block
    note("blocked edges")
    n_cols = 40000
    lengths = [0, 1, 257, 299, 300, 301, 320, 321, 640, 4096, 12345, 39999]
    src, dst = rows_with_lengths(lengths, n_cols, 320)
    s1, d1 = rows_with_lengths([600], n_cols, 340, lo=0, hi=625)
    s2, d2 = rows_with_lengths([620], n_cols, 341, lo=n_cols - 625, hi=n_cols)
    src = np.concatenate([src, s1, s2])
    dst = np.concatenate([dst, d1 + len(lengths), d2 + len(lengths) + 1])
    n_rows = len(lengths) + 2
    deg = (synth.splitmix64(342, 0, n_cols) % 50).astype(np.int32)
    og = oracle.Graph(n_rows, n_cols, src, dst, 0, deg=deg)
    g = build(G, n_rows, n_cols, src, dst, 0, deg=deg, GCN_COL_BLOCKS=64, GCN_PIECE_MAX=32,
              GCN_BLOCKED_MIN=300)
    bins = check_bins(G, g)
    assert bins[9]["rows"] == 10 and bins[8]["rows"] == 2
    for F in (1, 64, 128, 300):
        X = synth.uniform(343 + F, n_cols, F)
        assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="fwd F=%d" % F)
    Gm = synth.uniform(350, n_rows, 128)
    assert_close(host(G.gcn_aggregate_bwd(g, dev(Gm))), *og.bwd(Gm), what="bwd")


def test_blocked_star_and_determinism(G):
    import torch
    note("blocked star")
    k = 1 << 16
    src = np.arange(1, k + 1, dtype=np.int32)
    dst = np.zeros(k, np.int32)
    og = oracle.Graph(k + 1, k + 1, src, dst, SYM | LOOPS)
    g = build(G, k + 1, k + 1, src, dst, SYM | LOOPS, GCN_COL_BLOCKS=64)
    assert check_bins(G, g)[9]["rows"] == 1
    X = synth.uniform(360, k + 1, 128)
    Xd = dev(X)
    outs = [G.gcn_aggregate_fwd(g, Xd).clone() for _ in range(3)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int32), outs[0].view(torch.int32))
    assert_close(host(outs[0]), *og.fwd(X), what="star")


def test_blocked_q8_halo_fwd_and_bwd(G):
    note("blocked q8 halo")
    n = 1 << 14
    src, dst = synth.rmat_edges(370, n, 24 * n, perm_seed=371)
    og = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    g = build(G, n, n, src, dst, SYM | LOOPS, GCN_COL_BLOCKS=16, GCN_BLOCKED_MIN=400)
    assert check_bins(G, g)[9]["rows"] > 0
    nlc = n - n // 4
    X = synth.normal(372, n, 128)
    for bits in (8, 2):
        Q, Z, S = oracle.quantize_rows_bits(X[nlc:], bits)
        zs = dev(np.stack([Z, S], axis=1))
        for use_csc in (False, True):
            Y = G.gcn_aggregate_fwd_q8halo(g, nlc, dev(X[:nlc]), dev(Q), zs[:, 0], zs[:, 1],
                                           use_csc=use_csc, bits=bits)
            ptr, idx, val = ((og.csc_ptr, og.csc_idx, og.csc_val) if use_csc
                             else (og.csr_ptr, og.csr_idx, og.csr_val))
            ref = oracle.spmm_qbits(ptr, idx, val, nlc, X[:nlc], Q, Z, S, 128, bits)
            assert_close(host(Y), *ref, what="%d-bit halo csc=%s" % (bits, use_csc))


def test_blocking_off_by_default_on_small_matrices(G):
    note("blocking default")
    n = 1 << 14
    src, dst = synth.rmat_edges(380, n, 24 * n, perm_seed=381)
    g = G.gcn_build_csr(n, n, dev(src), dev(dst), SYM | LOOPS)
    bins = G.gcn_graph_bins(g, 0)
    assert len(bins) == 10 and bins[9]["rows"] == 0 and bins[8]["last_len"] == -1
    with plan_env(GCN_BLOCK_MIN_COLS=0, GCN_COL_BLOCKS=1):
        g1 = G.gcn_build_csr(n, n, dev(src), dev(dst), SYM | LOOPS)
    assert G.gcn_graph_bins(g1, 0)[9]["rows"] == 0


def test_blocked_bf16_and_relu_paths(G):
    # bf16 inputs (the other gather policy) and an odd F (the guarded tail
    # policy) through the pieces
    import torch
    note("blocked bf16 / odd F")
    n = 1 << 14
    src, dst = synth.rmat_edges(390, n, 24 * n, perm_seed=391)
    og = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    g = build(G, n, n, src, dst, SYM | LOOPS, GCN_COL_BLOCKS=32, GCN_SEGMENT_MIN=8)
    assert check_bins(G, g)[9]["rows"] > 0
    X = synth.uniform(392, n, 128)
    Xb = torch.from_numpy(bf16_bits(X).view(np.int16)).view(torch.bfloat16).to("cuda:0")
    assert_close(host(G.gcn_aggregate_fwd(g, Xb)), *og.fwd(bf16_round(X)), what="bf16 fwd")
    assert_close(host(G.gcn_aggregate_bwd(g, Xb)), *og.bwd(bf16_round(X)), what="bf16 bwd")
    for F in (47, 130):
        X = synth.uniform(393 + F, n, F)
        assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="F=%d" % F)


@pytest.mark.parametrize("f_in,hidden,C", [(100, 256, 47), (300, 64, 10)])
def test_blocked_gcn_step(G, f_in, hidden, C):
    # the 2-layer GCN step on a column-blocked graph, in both associations of
    # layer 1: the inputs aggregated first (f_in <= hidden), and X W1
    # aggregated with the ReLU fused into the partial-row reduction
    from test_gpu_dense import _step_check
    note("blocked gcn step f_in=%d hidden=%d" % (f_in, hidden))
    n = 3000
    src, dst = synth.rmat_edges(395, n, 12 * n, perm_seed=396)
    w = synth.Workload("rmat3000", n, n, src, dst, SYM | LOOPS, f_in)
    with plan_env(GCN_BLOCK_MIN_COLS=0, GCN_COL_BLOCKS=16, GCN_SEGMENT_MIN=8):
        _step_check(G, w, f_in, hidden, C, 13)


@pytest.mark.parametrize("lp", [False, True])
def test_blocked_sage_step(G, lp):
    # the GraphSAGE step (mean values, strided Z blocks, F = 100 and 64) on a
    # column-blocked graph
    from test_gpu_sage import check_step
    note("blocked sage step lp=%s" % lp)
    with plan_env(GCN_BLOCK_MIN_COLS=0, GCN_COL_BLOCKS=16, GCN_SEGMENT_MIN=8):
        check_step(G, 3000, 36000, 100, 64, 10, 397, lp)
