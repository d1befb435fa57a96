"""Hybrid pre/post-aggregation (Algorithm 1, Sections 5.2 and 5.3).

Host tests: the library's split (Hopcroft-Karp per component plus Koenig)
against the oracle's (augmenting paths plus Koenig): the cover size is unique
and must agree; which minimum cover is chosen may differ, so the library's is
checked for validity (every edge covered, post flags = source in the cover,
slots in id order).

GPU tests: a graph is split over workers by node id. The receiver (worker 0)
gets, from each sender, the covered source rows and the sender's partial sums
for the covered destinations (its pre-aggregation SpMM over the pre edges);
it aggregates its local edges plus the post edges, then adds the partial sums.
The result must equal the oracle's full aggregation of the receiver's rows,
and every stored value of the split operators must equal the corresponding
entry of the full A_hat bit for bit.
"""

import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module")
def G():
    import paper_2411_16025_amd as pkg
    pkg.lib()
    return pkg


def check_split(src, dst, n_src, n_dst, res, want_volume):
    is_post, src_slot, dst_slot, vol = res
    assert vol == want_volume
    cs, cd = src_slot >= 0, dst_slot >= 0
    assert cs.sum() + cd.sum() == vol
    assert np.array_equal(is_post, cs[src])
    assert np.all(cs[src] | cd[dst]), "an edge is not covered"
    for slot, c in ((src_slot, cs), (dst_slot, cd)):
        assert np.array_equal(slot[c], np.arange(c.sum()))


def golden_fig4():
    edges = []
    for line in open(os.path.join(GOLDEN, "prepost_fig4.txt")):
        t = line.split("#", 1)[0].split()
        if t and t[0].isdigit():
            edges.append((int(t[0]), int(t[1])))
    return np.array([e[0] for e in edges]), np.array([e[1] for e in edges])


def test_split_fig4_example(G):
    src, dst = golden_fig4()
    is_post, src_slot, dst_slot, vol = G.gcn_prepost_split(src, dst)
    assert vol == 2
    assert np.flatnonzero(src_slot >= 0).tolist() == [4]
    assert np.flatnonzero(dst_slot >= 0).tolist() == [2]
    assert is_post.tolist() == [True, True, True, False, False]


@pytest.mark.parametrize("seed", range(20))
def test_split_matches_oracle_small(G, seed):
    rng = np.random.default_rng(100 + seed)
    n_src, n_dst = int(rng.integers(1, 40)), int(rng.integers(1, 40))
    m = int(rng.integers(0, 120))
    src = rng.integers(0, n_src, m).astype(np.int32)
    dst = rng.integers(0, n_dst, m).astype(np.int32)
    res = G.gcn_prepost_split(src, dst, n_src, n_dst)
    want = oracle.bipartite_cover(src, dst, n_src, n_dst)[0] if m else 0
    check_split(src, dst, n_src, n_dst, res, want)


@pytest.mark.parametrize("n,m", [(2000, 6000), (20000, 160000)])
def test_split_matches_oracle_rmat(G, n, m):
    src, dst = synth.rmat_edges(7 + n, n, m, perm_seed=8 + n)
    res = G.gcn_prepost_split(src, dst, n, n)
    check_split(src, dst, n, n, res, oracle.bipartite_cover(src, dst, n, n)[0])


def test_split_special_graphs(G):
    # complete bipartite K_{3,5}: cover = the smaller side
    a, b = np.meshgrid(np.arange(3), np.arange(5), indexing="ij")
    res = G.gcn_prepost_split(a.ravel(), b.ravel(), 3, 5)
    assert res[3] == 3 and res[0].all()
    # a perfect matching of 7 disjoint edges: every component needs one row
    res = G.gcn_prepost_split(np.arange(7), np.arange(7)[::-1], 7, 7)
    assert res[3] == 7
    # a long path u0-v0-u1-v1-...: matching of size n
    n = 50000
    src = np.concatenate([np.arange(n), np.arange(1, n)])
    dst = np.concatenate([np.arange(n), np.arange(n - 1)])
    res = G.gcn_prepost_split(src, dst, n, n)
    check_split(src, dst, n, n, res, n)
    # repeated pairs count once; no edges at all
    res = G.gcn_prepost_split(np.array([1, 1, 1]), np.array([0, 0, 0]), 4, 2)
    assert res[3] == 1 and res[0].tolist() in ([True] * 3, [False] * 3)
    res = G.gcn_prepost_split(np.zeros(0, np.int32), np.zeros(0, np.int32), 3, 3)
    assert res[3] == 0 and (res[1] < 0).all() and (res[2] < 0).all()


def test_split_rejects_bad_arguments(G):
    import ctypes
    L = G.lib()
    assert L.gcn_prepost_split(-1, 2, 0, None, None, None, None, None, None) == 1
    assert L.gcn_prepost_split(2, 2, 3, None, None, None, None, None, None) == 1
    src = (ctypes.c_int32 * 2)(0, 2)
    dst = (ctypes.c_int32 * 2)(0, 0)
    assert L.gcn_prepost_split(2, 2, 2, src, dst, None, None, None, None) == 2
    assert "outside" in L.gcn_last_error().decode()
    with pytest.raises(G.GcnError):
        G.gcn_prepost_split(np.array([0, 5]), np.array([0, 0]), 3, 1)


# ---------------------------------------------------------------------------
# GPU: hybrid aggregation over workers equals the full aggregation.
# ---------------------------------------------------------------------------

def global_graph(seed, n, m):
    """Entries (row, col) of the symmetrized RMAT graph without self-loops, and
    each node's degree."""
    s, d = synth.rmat_edges(seed, n, m, perm_seed=seed + 1)
    keys = np.unique(np.concatenate([d.astype(np.int64) * n + s, s.astype(np.int64) * n + d]))
    rows, cols = keys // n, keys % n
    keep = rows != cols
    rows, cols = rows[keep], cols[keep]
    return rows, cols, np.bincount(rows, minlength=n).astype(np.int32)


def hybrid_receiver(G, bounds, rows, cols, deg, X, check_values=None):
    """Worker 0 = nodes [0, bounds[1]); worker w = [bounds[w], bounds[w+1]).
    Returns the receiver's output and, per sender, (cut edges, distinct
    destinations, distinct sources, rows sent)."""
    import torch
    from gpu_util import dev
    n0 = bounds[1]
    degd = dev(deg)
    local = (rows < n0) & (cols < n0)
    post_src, post_dst, partials, volumes = [], [], [], []
    recv_X, col_ids = [dev(X[:n0])], [np.arange(n0)]
    n_cols = n0
    for w in range(1, len(bounds) - 1):
        lo, hi = bounds[w], bounds[w + 1]
        cut = (rows < n0) & (cols >= lo) & (cols < hi)
        s_loc = (cols[cut] - lo).astype(np.int32)
        d_rec = rows[cut].astype(np.int32)
        is_post, src_slot, dst_slot, vol = G.gcn_prepost_split(s_loc, d_rec, hi - lo, n0)
        volumes.append((len(s_loc), len(np.unique(d_rec)), len(np.unique(s_loc)), vol))
        cov_src = np.flatnonzero(src_slot >= 0)
        cov_dst = np.flatnonzero(dst_slot >= 0).astype(np.int32)
        # sender: partial sums of the covered destinations over the pre edges
        if len(cov_dst):
            pre = ~is_post
            gp = G.gcn_build_csr(len(cov_dst), hi - lo, dev(s_loc[pre]),
                                 dev(dst_slot[d_rec[pre]]), 0)
            G.gcn_normalize_rc(gp, dev(deg[cov_dst]), degd[lo:hi].contiguous())
            if check_values is not None:
                check_values(gp, cov_dst, lo + np.arange(hi - lo))
            partials.append((G.gcn_aggregate_fwd(gp, dev(X[lo:hi])), dev(cov_dst)))
        # sent: the covered source rows and the partial sums
        recv_X.append(dev(X[lo + cov_src]))
        col_ids.append(lo + cov_src)
        post_src.append(n_cols + src_slot[s_loc[is_post]])
        post_dst.append(d_rec[is_post])
        n_cols += len(cov_src)
    col_ids = np.concatenate(col_ids)
    src_all = np.concatenate([cols[local]] + post_src).astype(np.int32)
    dst_all = np.concatenate([rows[local]] + post_dst).astype(np.int32)
    gr = G.gcn_build_csr(n0, n_cols, dev(src_all), dev(dst_all), synth.ADD_SELF_LOOPS)
    G.gcn_normalize_rc(gr, degd[:n0].contiguous(), dev(deg[col_ids]))
    if check_values is not None:
        check_values(gr, np.arange(n0), col_ids)
    Y = G.gcn_aggregate_fwd(gr, torch.cat(recv_X))
    for P, idx in partials:
        G.gcn_add_rows(P, idx, Y)
    torch.cuda.synchronize()
    return Y, volumes


def value_checker(G, og, n):
    """Every stored value of a split operator equals the entry of the full
    A_hat at the same (global row, global column), bit for bit."""
    full_rows = np.repeat(np.arange(n, dtype=np.int64), np.diff(og.csr_ptr))
    full_keys = full_rows * n + og.csr_idx

    def check(g, row_ids, col_ids):
        ptr, idx, val = G.gcn_graph_export(g, 0)
        r = np.asarray(row_ids, np.int64)[np.repeat(np.arange(len(ptr) - 1), np.diff(ptr))]
        keys = r * n + np.asarray(col_ids, np.int64)[idx]
        pos = np.searchsorted(full_keys, keys)
        assert np.array_equal(full_keys[np.minimum(pos, len(full_keys) - 1)], keys), \
            "an entry of the split operator is not an entry of A"
        assert np.array_equal(val.view(np.uint32), og.csr_val[pos].view(np.uint32))
    return check


@pytest.mark.gpu
@pytest.mark.parametrize("n,m,bounds,F", [
    (3000, 12000, (0, 1500, 3000), 32),
    (5000, 30000, (0, 1000, 2500, 5000), 47),
    (4096, 40000, (0, 4000, 4096), 64),
])
def test_hybrid_equals_full_aggregation(G, n, m, bounds, F):
    from gpu_util import assert_close, host, note
    note("prepost n=%d m=%d bounds=%s F=%d" % (n, m, bounds, F))
    rows, cols, deg = global_graph(11 + n, n, m)
    X = synth.normal(12 + n, n, F)
    og = oracle.Graph(n, n, cols.astype(np.int32), rows.astype(np.int32), synth.ADD_SELF_LOOPS)
    Y, volumes = hybrid_receiver(G, bounds, rows, cols, deg, X,
                                 check_values=value_checker(G, og, n))
    ref, S = og.fwd(X)
    n0 = bounds[1]
    assert_close(host(Y), ref[:n0], S[:n0], what="hybrid receiver rows")
    for n_edges, n_pre, n_post, vol in volumes:
        assert vol <= min(n_pre, n_post) <= n_edges


@pytest.mark.gpu
def test_hybrid_rmat20_two_workers(G):
    from gpu_util import assert_close, host, note
    n = 1 << 20
    note("prepost rmat20 two workers F=64")
    rows, cols, deg = global_graph(21, n, 16 * n)
    X = synth.uniform(22, n, 64)
    Y, volumes = hybrid_receiver(G, (0, n // 2, n), rows, cols, deg, X)
    og = oracle.Graph(n, n, cols.astype(np.int32), rows.astype(np.int32), synth.ADD_SELF_LOOPS)
    ref, S = og.fwd(X)
    assert_close(host(Y), ref[: n // 2], S[: n // 2], what="rmat20 hybrid receiver rows")
    n_edges, n_pre, n_post, vol = volumes[0]
    assert vol < min(n_pre, n_post)


@pytest.mark.gpu
def test_add_rows_exact(G):
    import torch
    from gpu_util import dev, host
    for F, ld in ((64, 64), (47, 50), (5, 5)):
        Y0 = synth.normal(31, 300, ld)
        P = synth.normal(32, 40, F)
        idx = np.random.default_rng(F).choice(300, 40, replace=False).astype(np.int32)
        Yd = dev(Y0)
        G.gcn_add_rows(dev(P), dev(idx), Yd[:, :F])
        torch.cuda.synchronize()
        want = Y0.copy()
        want[idx, :F] = (want[idx, :F] + P).astype(np.float32)
        assert np.array_equal(host(Yd).view(np.uint32), want.view(np.uint32))


@pytest.mark.gpu
def test_hybrid_partition_sampled(G):
    """The 14M x 20M partition with its halo nodes owned by 7 senders
    (contiguous id ranges): sampled receiver rows against the oracle."""
    import gc
    import torch
    from gpu_util import assert_close, host, note
    note("prepost partition 14M x 20M, 7 senders, sampled")
    w = synth.partition_111m()
    nl, nh = w.n_rows, w.n_cols - w.n_rows
    bounds = [0, nl] + [nl - (-(o * nh) // 7) for o in range(1, 8)]
    assert bounds[-1] == w.n_cols
    X = synth.normal(3014, w.n_cols, w.F)
    Y, volumes = hybrid_receiver(G, bounds, w.dst, w.src, w.deg, X)
    assert sum(v[3] for v in volumes) < sum(v[2] for v in volumes)
    rng = np.random.default_rng(7)
    cnt = np.bincount(w.dst, minlength=nl)
    sel = np.unique(np.concatenate([rng.choice(nl, 48, replace=False),
                                    np.argsort(-cnt, kind="stable")[:2]])).astype(np.int32)
    ptr, idx, val = oracle.sampled(nl, w.n_cols, w.src, w.dst, w.flags, sel, deg=w.deg)
    ref, S = oracle.spmm(ptr, idx, val, X)
    got = host(Y[torch.from_numpy(sel.astype(np.int64)).to(Y.device)])
    assert_close(got, ref, S, what="partition hybrid sampled rows")
    del Y
    gc.collect()
    torch.cuda.empty_cache()
