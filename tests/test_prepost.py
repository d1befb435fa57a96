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


def hybrid_receiver(G, bounds, rows, cols, deg, X, check_values=None, bits=None):
    """Worker 0 = nodes [0, bounds[1]); worker w = [bounds[w], bounds[w+1]).
    Returns the receiver's output and, per sender, (cut edges, distinct
    destinations, distinct sources, rows sent), and a dict of what was sent.

    bits (8 or 2): the senders quantize what they send, the covered source
    rows and their partial sums, per row with gcn_layernorm_quantize (no
    LayerNorm); the receiver aggregates the source rows through the fused
    dequantizing kernel (columns >= its own nodes are the received rows) and
    adds the partial sums with gcn_add_rows_q."""
    import torch
    from gpu_util import dev, host
    n0 = bounds[1]
    F = X.shape[1]
    degd = dev(deg)
    local = (rows < n0) & (cols < n0)
    post_src, post_dst, partials, volumes = [], [], [], []
    recv_X, col_ids = [dev(X[:n0])], [np.arange(n0)]
    recv_q = []
    sent = dict(pre=[], P=[], Pq=[])
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
            P = G.gcn_aggregate_fwd(gp, dev(X[lo:hi]))
            if bits is None:
                partials.append((P, dev(cov_dst)))
            else:
                q = G.gcn_layernorm_quantize(P, bits=bits, layernorm=False)
                partials.append((q, dev(cov_dst)))
                sent["pre"].append((lo, hi, s_loc[pre], dst_slot[d_rec[pre]], cov_dst))
                sent["P"].append(host(P))
                sent["Pq"].append(tuple(host(t) for t in q))
        # sent: the covered source rows and the partial sums
        if bits is None:
            recv_X.append(dev(X[lo + cov_src]))
        elif len(cov_src):
            recv_q.append(G.gcn_layernorm_quantize(dev(X[lo + cov_src]), bits=bits,
                                                   layernorm=False))
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
    if bits is None:
        Y = G.gcn_aggregate_fwd(gr, torch.cat(recv_X))
        for P, idx in partials:
            G.gcn_add_rows(P, idx, Y)
    else:
        Qh = torch.cat([q[0] for q in recv_q])
        Zh = torch.cat([q[1] for q in recv_q]).contiguous()
        Sh = torch.cat([q[2] for q in recv_q]).contiguous()
        Y = G.gcn_aggregate_fwd_q8halo(gr, n0, recv_X[0], Qh, Zh, Sh, F=F, bits=bits)
        for (Q, Z, S), idx in partials:
            G.gcn_add_rows_q(Q, Z, S, idx, Y, bits=bits, F=F)
        sent.update(Qh=host(Qh), Zh=host(Zh), Sh=host(Sh), src_all=src_all, dst_all=dst_all,
                    col_ids=col_ids, n_cols=n_cols)
    torch.cuda.synchronize()
    return Y, volumes, sent


def quantized_receiver_reference(n0, X, deg, bits, sent, sel=None):
    """The oracle's output for the receiver rows sel (default: all) of a
    quantized hybrid exchange: its own operator over [own rows | received
    source rows dequantized], plus the dequantized partial sums. The codes
    are checked first: the source rows' against the oracle's quantizer on
    the same inputs, the partial sums' against the oracle's quantizer on the
    GPU's fp32 partial sums (themselves checked against the oracle's
    pre-aggregation within 1e-5 * S), both bit for bit. Returns (Y, S, B):
    B[r] bounds the quantization error of row r against the exchange in fp32
    (half a code step of every dequantized term it receives, times its
    weight, plus 4 units of fp32 rounding of the row's largest value)."""
    from gpu_util import assert_close
    F = X.shape[1]
    col_ids = sent["col_ids"]
    Qr, Zr, Sr = oracle.quantize_rows_bits(X[col_ids[n0:]], bits)
    assert np.array_equal(sent["Qh"], Qr), "source-row codes"
    assert np.array_equal(sent["Zh"].view(np.uint32), Zr.view(np.uint32))
    assert np.array_equal(sent["Sh"].view(np.uint32), Sr.view(np.uint32))
    if sel is None:
        sel = np.arange(n0, dtype=np.int32)
    ptr, idx = oracle.rows_of(n0, sent["n_cols"], sent["src_all"], sent["dst_all"],
                              synth.ADD_SELF_LOOPS, sel)
    val = oracle.normalize_listed(ptr, deg[sel], deg[col_ids][idx])
    Y, S = oracle.spmm_qbits(ptr, idx, val, n0, X[:n0], Qr, Zr, Sr, F, bits)
    half = np.zeros((sent["n_cols"], 1), np.float32)
    # the quantizer picks the nearest code in fp32 arithmetic: within half a
    # step, plus a few units of fp32 rounding of the row's largest value
    half[n0:, 0] = Sr / 2 + np.abs(oracle.dequant_rows_bits(Qr, Zr, Sr, F, bits)).max(axis=1) * 2.0 ** -21
    B, _ = oracle.spmm(ptr, idx, val, half)
    B = B[:, 0].copy()
    pos = {int(r): i for i, r in enumerate(sel)}
    for (lo, hi, s_pre, d_pre, cov_dst), P, (Q, Z, Sc) in zip(sent["pre"], sent["P"], sent["Pq"]):
        gp_ptr, gp_idx = oracle.structure(len(cov_dst), hi - lo, s_pre, d_pre, 0)
        gp_val = oracle.normalize_listed(gp_ptr, deg[cov_dst], deg[lo + gp_idx])
        assert_close(P, *oracle.spmm(gp_ptr, gp_idx, gp_val, X[lo:hi]), what="partial sums")
        Qo, Zo, So = oracle.quantize_rows_bits(P, bits)
        assert np.array_equal(Q, Qo), "partial-sum codes"
        assert np.array_equal(Z.view(np.uint32), Zo.view(np.uint32))
        assert np.array_equal(Sc.view(np.uint32), So.view(np.uint32))
        D = oracle.dequant_rows_bits(Qo, Zo, So, F, bits).astype(np.float64)
        for j, r in enumerate(cov_dst):
            i = pos.get(int(r))
            if i is not None:
                Y[i] += D[j]
                S[i] += np.abs(D[j])
                B[i] += So[j] / 2 + np.abs(D[j]).max() * 2.0 ** -21
    return Y, S, B


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
    Y, volumes, _ = hybrid_receiver(G, bounds, rows, cols, deg, X,
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
    Y, volumes, _ = hybrid_receiver(G, (0, n // 2, n), rows, cols, deg, X)
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
@pytest.mark.parametrize("bits", [8, 2])
def test_add_rows_q_exact(G, bits):
    # Y[idx] += fmaf(q, S, Z) in fp32: the oracle's dequantized value (one
    # rounding) added in fp32, bit for bit; paired and separate (Z, S)
    import torch
    from gpu_util import dev, host, note
    for F, ld, paired in ((64, 64, True), (47, 50, False), (5, 5, True), (256, 256, False)):
        note("add_rows_q bits=%d F=%d" % (bits, F))
        Y0 = synth.normal(33, 300, ld)
        P = synth.normal(34, 40, F) * 3
        P[7] = 1.25  # a constant row: S = 0, every code 0, dequantized value Z
        Q, Z, S = oracle.quantize_rows_bits(P, bits)
        idx = np.random.default_rng(F + bits).choice(300, 40, replace=False).astype(np.int32)
        Yd = dev(Y0)
        if paired:
            zs = dev(np.stack([Z, S], axis=1))
            z, sc = zs[:, 0], zs[:, 1]
        else:
            z, sc = dev(Z), dev(S)
        G.gcn_add_rows_q(dev(Q), z, sc, dev(idx), Yd[:, :F], bits=bits, F=F)
        torch.cuda.synchronize()
        want = Y0.copy()
        want[idx, :F] = (want[idx, :F] + oracle.dequant_rows_bits(Q, Z, S, F, bits)).astype(np.float32)
        assert np.array_equal(host(Yd).view(np.uint32), want.view(np.uint32))


@pytest.mark.gpu
@pytest.mark.parametrize("bits", [8, 2])
@pytest.mark.parametrize("n,m,bounds,F", [
    (3000, 12000, (0, 1500, 3000), 32),
    (5000, 30000, (0, 1000, 2500, 5000), 47),
])
def test_hybrid_quantized_exchange(G, bits, n, m, bounds, F):
    # Sections 5.2 and 6.1 together on one GPU: the senders quantize the
    # covered source rows and their partial sums; the receiver dequantizes
    # the source rows inside the aggregation and the partial sums in the
    # combine. Every receiver row against the oracle on the same codes
    # (1e-5 * S), and against the full fp32 aggregation within the
    # quantization error of what it received.
    from gpu_util import assert_close, host, note
    note("prepost quantized bits=%d n=%d bounds=%s F=%d" % (bits, n, bounds, F))
    rows, cols, deg = global_graph(11 + n, n, m)
    X = synth.normal(12 + n, n, F)
    Y, volumes, sent = hybrid_receiver(G, bounds, rows, cols, deg, X, bits=bits)
    n0 = bounds[1]
    ref, S, B = quantized_receiver_reference(n0, X, deg, bits, sent)
    Yh = host(Y)
    assert_close(Yh, ref, S, what="quantized hybrid receiver vs oracle")
    og = oracle.Graph(n, n, cols.astype(np.int32), rows.astype(np.int32), synth.ADD_SELF_LOOPS)
    full, Sf = og.fwd(X)
    err = np.abs(Yh - full[:n0])
    assert np.all(err <= B[:, None] + 1e-5 * Sf[:n0] + 1e-30), "beyond the quantization error"
    note("largest deviation from fp32 exchange: %.3e of its bound"
         % float((err / (B[:, None] + 1e-5 * Sf[:n0] + 1e-30)).max()))


@pytest.mark.gpu
def test_hybrid_partition_quantized_sampled(G):
    """The 14M x 20M partition, 7 senders, 8-bit exchange: stratified rows of
    the receiver (every length class, the longest rows, rows with and
    without received columns) against the oracle on the same codes."""
    import gc
    import torch
    from gpu_util import assert_close, host, note
    note("prepost partition 14M x 20M, 7 senders, 8-bit exchange, sampled")
    w = synth.partition_111m()
    nl, nh = w.n_rows, w.n_cols - w.n_rows
    bounds = [0, nl] + [nl - (-(o * nh) // 7) for o in range(1, 8)]
    X = synth.normal(3014, w.n_cols, w.F)
    Y, volumes, sent = hybrid_receiver(G, bounds, w.dst, w.src, w.deg, X, bits=8)
    from test_gpu_configs import stratified_rows
    ptr_r, idx_r = oracle.rows_of(nl, sent["n_cols"], sent["src_all"], sent["dst_all"],
                                  synth.ADD_SELF_LOOPS, np.arange(nl, dtype=np.int32))
    sel, strata, _ = stratified_rows(ptr_r, idx_r, halo_from=nl, per_class=100, per_octave=100)
    del ptr_r, idx_r
    ref, S, _ = quantized_receiver_reference(nl, X, w.deg, 8, sent, sel=sel)
    got = host(Y[torch.from_numpy(sel.astype(np.int64)).to(Y.device)])
    note("sampled %d receiver rows: %s" % (len(sel), ", ".join("%s %d" % (k, len(v)) for k, v in strata)))
    assert_close(got, ref, S, what="partition quantized hybrid sampled rows")
    del Y
    gc.collect()
    torch.cuda.empty_cache()


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
    Y, volumes, _ = hybrid_receiver(G, bounds, w.dst, w.src, w.deg, X)
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
