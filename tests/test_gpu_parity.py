"""GPU parity: the HIP path against the CPU oracle on seeded inputs.

Structure, values and integer work are compared bit for bit; fp32
aggregations within 1e-5 * S per element, where S is the oracle's sum of
|terms| (fp32 accumulation in any order is correct); bf16 inputs within
1e-5 * S against the oracle on the same bf16-rounded input and 1e-2 * S
against the fp32 input.
"""

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


def gpu_graph(G, n_rows, n_cols, src, dst, flags, deg=None, normalize=True):
    g = G.gcn_build_csr(n_rows, n_cols, dev(src), dev(dst), flags)
    if normalize:
        G.gcn_normalize(g, dev(deg) if deg is not None else None)
    return g


def check_structure(G, g, og, normalized=True):
    for which, (p, i, v) in ((0, (og.csr_ptr, og.csr_idx, og.csr_val)),
                             (1, (og.csc_ptr, og.csc_idx, og.csc_val))):
        ptr, idx, val = G.gcn_graph_export(g, which)
        assert np.array_equal(ptr, p), "ptr differs (which=%d)" % which
        assert np.array_equal(idx, i), "idx differs (which=%d)" % which
        if normalized:
            assert np.array_equal(val.view(np.uint32), v.view(np.uint32)), \
                "val differs (which=%d)" % which
        else:
            assert np.all(val == 1.0)


# ---------------------------------------------------------------------------
# Structure and normalization, bit-exact.
# ---------------------------------------------------------------------------

CASES = [
    ("er_sym_loops", 3000, 3000, "er", SYM | LOOPS),
    ("er_directed_loops", 3000, 3000, "er", LOOPS),
    ("rmat_directed_noloops", 4096, 4096, "rmat", 0),
    ("rmat_sym_noloops", 5000, 5000, "rmat", SYM),
    ("rect_loops", 2000, 3500, "rect", LOOPS),
    ("rect_tall", 3500, 2000, "rect", 0),
]


def case_edges(kind, n_rows, n_cols, seed):
    if kind == "er":
        return synth.er_edges(seed, n_rows, 8 * n_rows)
    if kind == "rmat":
        return synth.rmat_edges(seed, n_rows, 10 * n_rows, perm_seed=seed + 1)
    src, dst = synth.er_edges(seed, max(n_rows, n_cols), 6 * max(n_rows, n_cols))
    return (src % n_cols).astype(np.int32), (dst % n_rows).astype(np.int32)


@pytest.mark.parametrize("name,n_rows,n_cols,kind,flags", CASES)
def test_structure_and_values_bit_exact(G, name, n_rows, n_cols, kind, flags):
    note("structure " + name)
    src, dst = case_edges(kind, n_rows, n_cols, 100 + len(name))
    deg = None
    if n_rows != n_cols:
        deg = (synth.splitmix64(7, 0, max(n_rows, n_cols)) % 1000).astype(np.int32)
    og = oracle.Graph(n_rows, n_cols, src, dst, flags, deg=deg)
    g = gpu_graph(G, n_rows, n_cols, src, dst, flags, normalize=False)
    assert g.nnz == og.nnz
    check_structure(G, g, og, normalized=False)
    G.gcn_normalize(g, dev(deg) if deg is not None else None)
    check_structure(G, g, og, normalized=True)


def test_normalization_bit_exact_over_wide_degrees(G):
    # rectangular graph, supplied degrees spread over [0, 2^30): every entry's
    # value exercises the double sqrt and division rounding
    note("normalize wide degrees")
    n_rows, n_cols = 4000, 60000
    src, dst = synth.er_edges(11, n_cols, 200000)
    dst = (dst % n_rows).astype(np.int32)
    h = synth.splitmix64(12, 0, n_cols)
    deg = ((h >> np.uint64(34)) >> (h & np.uint64(31))).astype(np.int32)  # log-uniform-ish
    deg[:10] = [0, 1, 2, 3, 2**30 - 1, 2**30, 2**31 - 2, 12345678, 99999, 7]
    og = oracle.Graph(n_rows, n_cols, src, dst, LOOPS, deg=deg)
    g = gpu_graph(G, n_rows, n_cols, src, dst, LOOPS, deg=deg)
    check_structure(G, g, og)


@pytest.mark.parametrize("flags", [SYM | LOOPS, SYM])
def test_normalize_rc_symmetric_graph_unequal_degrees(G, flags):
    # A symmetric graph stores A once for both directions. Row and column
    # degrees that differ make A_hat non-symmetric: entry (r, c) of A is
    # f(dr[r], dc[c]) and entry (c, r) of A^T must carry the same value, so
    # the transpose needs values of its own; the backward then computes
    # A_hat^T G, not A_hat G.
    note("normalize_rc symmetric flags=%d" % flags)
    n = 3000
    src, dst = synth.rmat_edges(141, n, 10 * n, perm_seed=142)
    og = oracle.Graph(n, n, src, dst, flags, normalized=False)
    dr = (synth.splitmix64(143, 0, n) % 500).astype(np.int32)
    dc = (synth.splitmix64(144, 0, n) % 70).astype(np.int32)
    csr_val = oracle.normalize_listed(og.csr_ptr, dr, dc[og.csr_idx])
    csc_val = oracle.normalize_listed(og.csc_ptr, dc, dr[og.csc_idx])
    assert not np.array_equal(csr_val, csc_val)
    g = gpu_graph(G, n, n, src, dst, flags, normalize=False)
    G.gcn_normalize_rc(g, dev(dr), dev(dc))
    for which, (p, i, v) in ((0, (og.csr_ptr, og.csr_idx, csr_val)),
                             (1, (og.csc_ptr, og.csc_idx, csc_val))):
        ptr, idx, val = G.gcn_graph_export(g, which)
        assert np.array_equal(ptr, p) and np.array_equal(idx, i)
        assert np.array_equal(val.view(np.uint32), v.view(np.uint32)), "values of %d" % which
    X = synth.uniform(145, n, 64)
    assert_close(host(G.gcn_aggregate_fwd(g, dev(X))),
                 *oracle.spmm(og.csr_ptr, og.csr_idx, csr_val, X), what="fwd")
    assert_close(host(G.gcn_aggregate_bwd(g, dev(X))),
                 *oracle.spmm(og.csc_ptr, og.csc_idx, csc_val, X), what="bwd")
    # the same degree array for both: the symmetric normalization again
    G.gcn_normalize(g)
    og2 = oracle.Graph(n, n, src, dst, flags)
    for which, v in ((0, og2.csr_val), (1, og2.csc_val)):
        _, _, val = G.gcn_graph_export(g, which)
        assert np.array_equal(val.view(np.uint32), v.view(np.uint32))


# ---------------------------------------------------------------------------
# Aggregation, fp32 and bf16.
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def rmat14(G):
    n = 1 << 14
    src, dst = synth.rmat_edges(21, n, 12 * n, perm_seed=22)
    og = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    g = gpu_graph(G, n, n, src, dst, SYM | LOOPS)
    return n, og, g


@pytest.mark.parametrize("F", [1, 3, 4, 47, 64, 100, 128, 256, 300, 1030, 2049])
def test_fwd_bwd_fp32_feature_sweep(G, rmat14, F):
    n, og, g = rmat14
    note("fwd/bwd fp32 rmat14 F=%d" % F)
    X = synth.uniform(31, n, F)
    Yref, S = og.fwd(X)
    Y = host(G.gcn_aggregate_fwd(g, dev(X)))
    assert_close(Y, Yref, S, what="fwd F=%d" % F)
    Gm = synth.uniform(32, n, F)
    dref, S2 = og.bwd(Gm)
    dX = host(G.gcn_aggregate_bwd(g, dev(Gm)))
    assert_close(dX, dref, S2, what="bwd F=%d" % F)


@pytest.mark.parametrize("pad", [4, 5])
def test_leading_dimension_padding(G, rmat14, pad):
    import torch
    n, og, g = rmat14
    F = 47
    note("ld padding F=47 pad=%d" % pad)
    X = synth.uniform(33, n, F, ld=F + pad)
    Yref, S = og.fwd(X[:, :F])
    Xd = dev(X)[:, :F]
    Yfull = torch.full((n, F + pad), 7.0, device="cuda:0")
    G.gcn_aggregate_fwd(g, Xd, Y=Yfull[:, :F])
    Yh = host(Yfull)
    assert_close(Yh[:, :F], Yref, S, what="fwd ld pad")
    assert np.all(Yh[:, F:] == 7.0), "padding columns were overwritten"


def test_bf16_inputs(G, rmat14):
    import torch
    n, og, g = rmat14
    F = 128
    note("bf16 fwd/bwd")
    X = synth.uniform(34, n, F)
    Xb = torch.from_numpy(bf16_bits(X).view(np.int16)).view(torch.bfloat16).to("cuda:0")
    Y = host(G.gcn_aggregate_fwd(g, Xb))
    Yr, Sr = og.fwd(bf16_round(X))
    assert_close(Y, Yr, Sr, what="bf16 vs oracle on rounded input")
    Yf, Sf = og.fwd(X)
    assert_close(Y, Yf, Sf, rel=1e-2, what="bf16 vs fp32 oracle")
    dX = host(G.gcn_aggregate_bwd(g, Xb))
    assert_close(dX, *og.bwd(bf16_round(X)), what="bf16 bwd")


def test_adjoint_identity_on_gpu_outputs(G):
    # <A_hat x, g> = <x, A_hat^T g>, independent of the oracle
    n = 6000
    note("adjoint identity")
    src, dst = synth.rmat_edges(41, n, 60000, perm_seed=42)
    g = gpu_graph(G, n, n, src, dst, LOOPS)
    F = 16
    x = synth.uniform(43, n, F).astype(np.float64)
    gg = synth.uniform(44, n, F).astype(np.float64)
    Y = host(G.gcn_aggregate_fwd(g, dev(x.astype(np.float32)))).astype(np.float64)
    dX = host(G.gcn_aggregate_bwd(g, dev(gg.astype(np.float32)))).astype(np.float64)
    lhs = np.sum(Y * gg)
    rhs = np.sum(x * dX)
    mag = np.sum(np.abs(Y) * np.abs(gg)) + np.sum(np.abs(x) * np.abs(dX))
    assert abs(lhs - rhs) <= 1e-5 * mag


def test_determinism_bitwise(G):
    import torch
    note("determinism")
    n = 1 << 15
    src, dst = synth.rmat_edges(51, n, 40 * n, perm_seed=52)
    g = gpu_graph(G, n, n, src, dst, SYM | LOOPS)
    bins = G.gcn_graph_bins(g, 0)
    # rows summed from partial rows: the chunk table by default, column-blocked
    # pieces when blocking is forced on small matrices (GCN_BLOCK_MIN_COLS=0)
    assert bins[8]["rows"] + bins[9]["rows"] > 0, "expected rows summed from partial rows"
    X = dev(synth.uniform(53, n, 128))
    outs = [G.gcn_aggregate_fwd(g, X).clone() for _ in range(3)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int32), outs[0].view(torch.int32))


# ---------------------------------------------------------------------------
# Shapes at the edges of the binning.
# ---------------------------------------------------------------------------

def rows_with_lengths(lengths, n_cols, seed):
    """Rectangular graph whose row i has exactly lengths[i] distinct columns."""
    src, dst = [], []
    for i, L in enumerate(lengths):
        cols = (synth.permutation(seed + i, n_cols)[:L]).astype(np.int32)
        src.append(cols)
        dst.append(np.full(L, i, np.int32))
    return np.concatenate(src), np.concatenate(dst)


@pytest.mark.parametrize("F", [64, 128, 256])
def test_row_lengths_at_class_boundaries(G, F):
    note("class boundaries F=%d" % F)
    lengths = [0, 1, 2, 3, 4, 5, 8, 9, 16, 17, 32, 33, 255, 256, 257, 1000, 2047, 2048, 2049,
               4095, 4096, 4097, 6000, 0, 1, 12345, 40000]
    n_cols = 50000
    src, dst = rows_with_lengths(lengths, n_cols, 61)
    n_rows = len(lengths)
    deg = (synth.splitmix64(62, 0, n_cols) % 100).astype(np.int32)
    og = oracle.Graph(n_rows, n_cols, src, dst, 0, deg=deg)
    g = gpu_graph(G, n_rows, n_cols, src, dst, 0, deg=deg)
    X = synth.uniform(63, n_cols, F)
    assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="fwd")
    Gm = synth.uniform(64, n_rows, F)
    assert_close(host(G.gcn_aggregate_bwd(g, dev(Gm))), *og.bwd(Gm), what="bwd")


def test_small_chunks_many_partials(G):
    # a short chunk length forces multi-chunk rows on a small graph
    note("chunk_len 64")
    os.environ["GCN_CHUNK_LEN"] = "64"
    os.environ["GCN_MEDIUM_MAX"] = "40"
    try:
        n = 3000
        src, dst = synth.rmat_edges(65, n, 30 * n, perm_seed=66)
        og = oracle.Graph(n, n, src, dst, SYM | LOOPS)
        g = gpu_graph(G, n, n, src, dst, SYM | LOOPS)
    finally:
        del os.environ["GCN_CHUNK_LEN"]
        del os.environ["GCN_MEDIUM_MAX"]
    bins = G.gcn_graph_bins(g, 0)
    assert bins[8]["first_len"] == 41 and bins[8]["rows"] > 10
    for F in (4, 100, 128):
        X = synth.uniform(67, n, F)
        assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="fwd F=%d" % F)


def test_empty_graph_is_identity_bitwise(G):
    note("empty graph")
    n = 1000
    e = np.zeros(0, np.int32)
    g = gpu_graph(G, n, n, e, e, SYM | LOOPS)
    X = synth.uniform(71, n, 128)
    assert np.array_equal(host(G.gcn_aggregate_fwd(g, dev(X))), X)
    assert np.array_equal(host(G.gcn_aggregate_bwd(g, dev(X))), X)


def test_no_entries_at_all_gives_zeros(G):
    note("no entries")
    n = 777
    e = np.zeros(0, np.int32)
    g = gpu_graph(G, n, n + 5, e, e, 0, normalize=False)
    assert g.nnz == 0
    X = synth.uniform(72, n + 5, 33)
    assert np.all(host(G.gcn_aggregate_fwd(g, dev(X))) == 0)
    assert np.all(host(G.gcn_aggregate_bwd(g, dev(synth.uniform(73, n, 33)))) == 0)


def test_star_giant_row(G):
    note("star giant row")
    k = 1 << 17
    src = np.arange(1, k + 1, dtype=np.int32)
    dst = np.zeros(k, np.int32)
    og = oracle.Graph(k + 1, k + 1, src, dst, SYM | LOOPS)
    g = gpu_graph(G, k + 1, k + 1, src, dst, SYM | LOOPS)
    X = synth.uniform(74, k + 1, 128)
    assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="star")


def test_star_2p20_leaves_default_plan(G):
    # the single giant row of a power-law extreme: a star with 2^20 leaves,
    # 2^20 + 1 columns, so the default plan cuts the hub row at column blocks
    # (its 2^20 + 1 entries make the most segments and pieces a row gets);
    # forward and transposed, against the oracle and the closed form
    note("star 2^20 leaves, default plan")
    k = 1 << 20
    src = np.arange(1, k + 1, dtype=np.int32)
    dst = np.zeros(k, np.int32)
    og = oracle.Graph(k + 1, k + 1, src, dst, SYM | LOOPS)
    g = gpu_graph(G, k + 1, k + 1, src, dst, SYM | LOOPS)
    bins = G.gcn_graph_bins(g, 0)
    assert bins[-1]["rows"] == 1 and bins[-1]["entries"] == k + 1, bins[-1]
    X = synth.uniform(75, k + 1, 128)
    Y = host(G.gcn_aggregate_fwd(g, dev(X)))
    ref, S = og.fwd(X)
    assert_close(Y, ref, S, what="star 2^20 fwd")
    # the hub row in closed form: x_0 / (k + 1) + (sum of the leaves' rows) /
    # sqrt(2 (k + 1)), up to the fp32 rounding of the two stored values
    hub = (X[0].astype(np.float64) / (k + 1)
           + X[1:].astype(np.float64).sum(axis=0) / np.sqrt(2.0 * (k + 1)))
    assert np.allclose(Y[0], hub, rtol=0, atol=1e-5 * S[0].max())
    Gm = synth.uniform(76, k + 1, 128)
    assert_close(host(G.gcn_aggregate_bwd(g, dev(Gm))), *og.bwd(Gm), what="star 2^20 bwd")
    g.free()


def test_unnormalized_index_add(G):
    # val = 1: Index_add semantics, rows of src summed into dst
    note("index_add")
    n = 5000
    src, dst = synth.rmat_edges(75, n, 50000, perm_seed=76)
    og = oracle.Graph(n, n, src, dst, 0, deg=np.zeros(n, np.int32), normalized=False)
    g = gpu_graph(G, n, n, src, dst, 0, normalize=False)
    X = synth.uniform(77, n, 64)
    assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="index_add")


# ---------------------------------------------------------------------------
# Quantization and the fused halo path.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("F", [128, 47, 3])
def test_quantize_kernel_bit_exact(G, F):
    note("quantize F=%d" % F)
    X = synth.normal(81, 3000, F)
    X[5] = 1.5
    Q, Z, S = oracle.quantize_rows(X)
    q, z, s = (host(t) for t in G.gcn_quantize_rows_u8(dev(X)))
    assert np.array_equal(q, Q)
    assert np.array_equal(z.view(np.uint32), Z.view(np.uint32))
    assert np.array_equal(s.view(np.uint32), S.view(np.uint32))


@pytest.mark.parametrize("F", [128, 48, 47])
def test_q8_permutation_graph_dequant_bit_exact(G, F):
    # one entry per row into a distinct halo column, value 1: Y is the
    # dequantized halo row itself, fmaf(q, S, Z), bit for bit
    note("q8 permutation F=%d" % F)
    n_local, n_halo = 500, 4096
    perm = synth.permutation(82, n_halo)
    src = (n_local + perm).astype(np.int32)
    dst = np.arange(n_halo, dtype=np.int32)
    g = gpu_graph(G, n_halo, n_local + n_halo, src, dst, 0, normalize=False)
    Xl = synth.uniform(83, n_local, F)
    Qh = synth.random_bytes(84, n_halo, F)
    Z = synth.normal(85, n_halo, 1)[:, 0]
    S = np.abs(synth.normal(86, n_halo, 1)[:, 0]) * 0.01
    S[:3] = 0.0
    Y = host(G.gcn_aggregate_fwd_q8halo(g, n_local, dev(Xl), dev(Qh), dev(Z), dev(S)))
    D = oracle.dequant_rows(Qh, Z, S)
    assert np.array_equal(Y.view(np.uint32), D[perm].view(np.uint32))


@pytest.mark.parametrize("F", [128, 64, 47])
def test_q8_halo_fwd_and_bwd(G, F):
    note("q8 halo fwd/bwd F=%d" % F)
    n = 1 << 14
    src, dst = synth.rmat_edges(91, n, 16 * n, perm_seed=92)
    og = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    g = gpu_graph(G, n, n, src, dst, SYM | LOOPS)
    nlc = n - n // 4
    X = synth.normal(93, n, F)
    Q, Z, S = oracle.quantize_rows(X[nlc:])
    Y = host(G.gcn_aggregate_fwd_q8halo(g, nlc, dev(X[:nlc]), dev(Q), dev(Z), dev(S)))
    assert_close(Y, *oracle.spmm_q8(og.csr_ptr, og.csr_idx, og.csr_val, nlc, X[:nlc], Q, Z, S),
                 what="q8 fwd")
    Gm = synth.normal(94, n, F)
    QG, ZG, SG = oracle.quantize_rows(Gm[nlc:])
    dX = host(G.gcn_aggregate_fwd_q8halo(g, nlc, dev(Gm[:nlc]), dev(QG), dev(ZG), dev(SG),
                                         use_csc=True))
    assert_close(dX, *oracle.spmm_q8(og.csc_ptr, og.csc_idx, og.csc_val, nlc, Gm[:nlc], QG, ZG,
                                     SG), what="q8 bwd")


def test_q8_paired_params_and_quantizer(G):
    # (Z, S) side by side (ldp = 2), written by the GPU quantizer and read by
    # the fused kernel; codes and params must equal the oracle's bit for bit
    import torch
    note("q8 paired params")
    n = 1 << 13
    src, dst = synth.rmat_edges(98, n, 12 * n, perm_seed=99)
    og = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    g = gpu_graph(G, n, n, src, dst, SYM | LOOPS)
    nlc, F = n - n // 4, 128
    X = synth.normal(100, n, F)
    Q, Z, S = oracle.quantize_rows(X[nlc:])
    Xd = dev(X)
    q, z, s = G.gcn_quantize_rows_u8(Xd[nlc:], paired=True)
    assert z.stride(0) == 2 and s.data_ptr() == z.data_ptr() + 4
    assert np.array_equal(host(q), Q)
    assert np.array_equal(host(z).view(np.uint32), Z.view(np.uint32))
    assert np.array_equal(host(s).view(np.uint32), S.view(np.uint32))
    Y = host(G.gcn_aggregate_fwd_q8halo(g, nlc, Xd[:nlc], q, z, s))
    assert_close(Y, *oracle.spmm_q8(og.csr_ptr, og.csr_idx, og.csr_val, nlc, X[:nlc], Q, Z, S),
                 what="q8 paired")
    # a general stride (ldp = 3) reads the same values
    zs3 = torch.zeros((n - nlc, 3), dtype=torch.float32, device="cuda:0")
    zs3[:, 0] = dev(Z)
    zs3[:, 1] = dev(S)
    Y3 = host(G.gcn_aggregate_fwd_q8halo(g, nlc, Xd[:nlc], q, zs3[:, 0], zs3[:, 1]))
    assert np.array_equal(Y3.view(np.uint32), Y.view(np.uint32))


def test_q8_rectangular_csc(G):
    # non-symmetric rectangular graph: the CSC path with halo rows of G
    note("q8 rectangular csc")
    n_rows, n_cols = 3000, 5000
    src, dst = case_edges("rect", n_rows, n_cols, 95)
    deg = (synth.splitmix64(96, 0, max(n_rows, n_cols)) % 300).astype(np.int32)
    og = oracle.Graph(n_rows, n_cols, src, dst, LOOPS, deg=deg)
    g = gpu_graph(G, n_rows, n_cols, src, dst, LOOPS, deg=deg)
    F = 64
    nl = 2000  # input rows of A^T are the n_rows destinations
    Gm = synth.normal(97, n_rows, F)
    QG, ZG, SG = oracle.quantize_rows(Gm[nl:])
    dX = host(G.gcn_aggregate_fwd_q8halo(g, nl, dev(Gm[:nl]), dev(QG), dev(ZG), dev(SG),
                                         use_csc=True))
    assert dX.shape == (n_cols, F)
    assert_close(dX, *oracle.spmm_q8(og.csc_ptr, og.csc_idx, og.csc_val, nl, Gm[:nl], QG, ZG, SG),
                 what="q8 csc rect")
    # all-halo and no-halo extremes
    Q0, Z0, S0 = oracle.quantize_rows(Gm)
    dX0 = host(G.gcn_aggregate_fwd_q8halo(g, 0, None, dev(Q0), dev(Z0), dev(S0), use_csc=True))
    assert_close(dX0, *oracle.spmm_q8(og.csc_ptr, og.csc_idx, og.csc_val, 0, Gm[:0], Q0, Z0, S0),
                 what="all halo")
    dX1 = host(G.gcn_aggregate_fwd_q8halo(g, n_rows, dev(Gm), None, None, None, use_csc=True))
    assert_close(dX1, *og.bwd(Gm), what="no halo")


# ---------------------------------------------------------------------------
# Errors detected on the device.
# ---------------------------------------------------------------------------

def test_device_detected_errors(G):
    note("device errors")
    src = np.array([0, 1, 9], np.int32)
    dst = np.array([1, 2, 3], np.int32)
    with pytest.raises(G.GcnError) as ei:
        G.gcn_build_csr(5, 5, dev(src), dev(dst), 0)
    assert ei.value.status == 2
    g = gpu_graph(G, 5, 6, src[:2], dst[:2], 0, normalize=False)
    with pytest.raises(G.GcnError) as ei:
        G.gcn_normalize(g, dev(np.array([1, 1, 0, 0, 0, -1], np.int32)))
    assert ei.value.status == 1
    with pytest.raises(G.GcnError) as ei:
        G.gcn_normalize(g)  # rectangular without degrees
    assert ei.value.status == 1
    X = dev(np.zeros((6, 4), np.float32))
    with pytest.raises(G.GcnError) as ei:
        G.gcn_aggregate_fwd_q8halo(g, 7, dev(np.zeros((8, 4), np.float32)), None, None, None)
    assert ei.value.status == 2
    g.free()
    with pytest.raises(G.GcnError):
        G.gcn_aggregate_fwd(g, X)
