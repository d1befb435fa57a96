"""Pins of the CPU oracle against facts that do not come from the oracle.

Each test ties an oracle routine to something fixed independently of it:
dense brute force built straight from the edge list, the eigenvector of the
GCN propagation matrix, the adjoint identity, closed forms of small graphs,
hand-derived golden matrices, nearest-code optimality of the quantizer, and
finite differences of the training loss.
"""

import math
import os

import numpy as np
import pytest

import oracle
import synth

SYM, LOOPS = oracle.SYMMETRIZE, oracle.ADD_SELF_LOOPS
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# Dense brute force: A~ straight from the edge list, no sorting involved.
# ---------------------------------------------------------------------------

def dense_adjacency(n_rows, n_cols, src, dst, flags):
    A = np.zeros((n_rows, n_cols), np.float64)
    A[dst, src] = 1.0
    if flags & SYM:
        A[src, dst] = 1.0
    if flags & LOOPS:
        m = min(n_rows, n_cols)
        A[np.arange(m), np.arange(m)] = 1.0
    return A


def dense_ahat(A, deg):
    d = np.asarray(deg, np.float64) + 1.0
    n_rows = A.shape[0]
    return A / np.sqrt(d[:n_rows, None] * d[None, : A.shape[1]])


def csr_to_dense(ptr, idx, val, n_major, n_minor):
    M = np.zeros((n_major, n_minor), np.float64)
    rows = np.repeat(np.arange(n_major), np.diff(ptr))
    M[rows, idx] = val
    return M


@pytest.mark.parametrize("seed", range(8))
def test_dense_brute_force_symmetric(seed):
    n = [7, 33, 64, 129, 200, 257, 400, 512][seed]
    m = 3 * n + seed
    src, dst = synth.er_edges(9000 + seed, n, m)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    A = dense_adjacency(n, n, src, dst, SYM | LOOPS)
    # structure: nonzero pattern of A~ equals the CSR and the CSC
    pat = csr_to_dense(g.csr_ptr, g.csr_idx, np.ones(g.nnz), n, n)
    assert np.array_equal(pat, A)
    patc = csr_to_dense(g.csc_ptr, g.csc_idx, np.ones(len(g.csc_idx)), n, n)
    assert np.array_equal(patc, A.T)
    deg = A.sum(axis=1) - 1.0
    assert np.array_equal(g.deg, deg.astype(np.int32))
    Ah = dense_ahat(A, deg)
    X = synth.uniform(3000 + seed, n, 5)
    Y, S = g.fwd(X)
    ref = Ah @ X.astype(np.float64)
    # the oracle's only rounding beyond double is the fp32 val (<= 2^-24 rel)
    assert np.all(np.abs(Y - ref) <= 2.0**-23 * S + 1e-300)
    # val itself equals the dense normalized entry to fp32 rounding
    dense_val = Ah[np.repeat(np.arange(n), np.diff(g.csr_ptr)), g.csr_idx]
    assert np.array_equal(g.csr_val, dense_val.astype(np.float32))


@pytest.mark.parametrize("seed", range(4))
def test_dense_brute_force_rectangular(seed):
    # one worker's share: rows 0..n_r-1 are local, columns n_r.. are halo,
    # normalization by a supplied global degree
    n_r, n_c = [(10, 17), (64, 100), (130, 260), (300, 301)][seed]
    m = 4 * n_r
    src, dst = synth.er_edges(9100 + seed, n_c, m)
    dst = dst % n_r
    deg = (synth.splitmix64(9200 + seed, 0, n_c) % 50).astype(np.int32) + 3
    g = oracle.Graph(n_r, n_c, src, dst, LOOPS, deg=deg)
    A = dense_adjacency(n_r, n_c, src, dst, LOOPS)
    assert np.array_equal(csr_to_dense(g.csr_ptr, g.csr_idx, np.ones(g.nnz), n_r, n_c), A)
    assert np.array_equal(csr_to_dense(g.csc_ptr, g.csc_idx, np.ones(g.nnz), n_c, n_r), A.T)
    Ah = dense_ahat(A, deg)
    X = synth.uniform(3100 + seed, n_c, 9)
    Y, S = g.fwd(X)
    assert np.all(np.abs(Y - Ah @ X.astype(np.float64)) <= 2.0**-23 * S + 1e-300)
    G = synth.uniform(4100 + seed, n_r, 9)
    dX, S2 = g.bwd(G)
    assert np.all(np.abs(dX - Ah.T @ G.astype(np.float64)) <= 2.0**-23 * S2 + 1e-300)


def test_duplicates_and_drawn_self_loops_are_dropped():
    src = np.array([0, 0, 1, 2, 2, 3, 3], np.int32)
    dst = np.array([1, 1, 0, 2, 3, 2, 0], np.int32)
    g = oracle.Graph(4, 4, src, dst, SYM | LOOPS)
    # undirected edges {0,1}, {2,3}, {0,3} plus four self-loops
    assert g.nnz == 3 * 2 + 4
    assert list(g.deg) == [2, 1, 1, 2]


def test_unnormalized_graph_is_index_add():
    # Index_add (Section 4): rows of src added into dst, value 1 per entry
    n = 50
    src, dst = synth.er_edges(77, n, 300)
    g = oracle.Graph(n, n, src, dst, 0, deg=np.zeros(n, np.int32), normalized=False)
    X = synth.uniform(78, n, 3)
    Y, _ = g.fwd(X)
    ref = np.zeros((n, 3))
    seen = set()
    for s, d in zip(src, dst):
        if (s, d) not in seen:
            seen.add((s, d))
            ref[d] += X[s]
    assert np.array_equal(Y, ref)


# ---------------------------------------------------------------------------
# Invariants.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("scale", [8, 11])
def test_eigenvector_invariant(scale):
    # A_hat sqrt(d~) = sqrt(d~) for symmetric binary A with one self-loop
    n = 1 << scale
    src, dst = synth.rmat_edges(500 + scale, n, 8 * n, perm_seed=600 + scale)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    v = np.sqrt(g.deg.astype(np.float64) + 1.0)
    x = v.astype(np.float32)[:, None]
    Y, S = g.fwd(x)
    # positive terms: error <= rounding of val (2^-24) and of x (2^-24)
    assert np.all(np.abs(Y[:, 0] - v) <= 2.0**-22 * S[:, 0])


def test_partition_row_sum_invariant():
    # For any row set under degrees d~: (A_hat sqrt(d~))_i = nnz_i / sqrt(d~_i)
    n_r, n_c = 300, 500
    src, dst = synth.er_edges(31, n_c, 2000)
    dst = dst % n_r
    deg = (synth.splitmix64(32, 0, n_c) % 40).astype(np.int32) + 5
    g = oracle.Graph(n_r, n_c, src, dst, LOOPS, deg=deg)
    d = deg.astype(np.float64) + 1.0
    Y, S = g.fwd(np.sqrt(d).astype(np.float32)[:, None])
    expect = np.diff(g.csr_ptr) / np.sqrt(d[:n_r])
    assert np.all(np.abs(Y[:, 0] - expect) <= 2.0**-22 * S[:, 0])


@pytest.mark.parametrize("seed", range(3))
def test_adjoint_identity(seed):
    # <A x, g> = <x, A^T g>: ties the CSC path to the CSR path
    n = 700
    src, dst = synth.rmat_edges(40 + seed, n, 5000)  # directed, not symmetrized
    g = oracle.Graph(n, n, src, dst, LOOPS)
    assert not np.array_equal(g.csr_idx, g.csc_idx)
    x = synth.uniform(50 + seed, n, 4)
    gg = synth.uniform(60 + seed, n, 4)
    Y, S = g.fwd(x)
    dX, S2 = g.bwd(gg)
    lhs = np.sum(Y * gg.astype(np.float64))
    rhs = np.sum(x.astype(np.float64) * dX)
    mag = np.sum(S * np.abs(gg)) + np.sum(np.abs(x) * S2)
    assert abs(lhs - rhs) <= 1e-12 * mag


# ---------------------------------------------------------------------------
# Closed forms and hand-derived matrices.
# ---------------------------------------------------------------------------

def test_empty_graph_is_identity_bitwise():
    n = 37
    g = oracle.Graph(n, n, np.zeros(0, np.int32), np.zeros(0, np.int32), SYM | LOOPS)
    assert np.all(g.csr_val == 1.0)
    X = synth.uniform(5, n, 11)
    Y, _ = g.fwd(X)
    assert np.array_equal(Y.astype(np.float32), X)


def test_cycle_closed_form():
    n = 41
    src = np.arange(n, dtype=np.int32)
    dst = ((src + 1) % n).astype(np.int32)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    X = synth.uniform(6, n, 3).astype(np.float64)
    Y, S = g.fwd(X.astype(np.float32))
    ref = (np.roll(X, 1, 0) + X + np.roll(X, -1, 0)) / 3.0
    assert np.all(np.abs(Y - ref) <= 2.0**-23 * S)


def test_complete_graph_closed_form():
    n = 23
    ii, jj = np.meshgrid(np.arange(n), np.arange(n))
    g = oracle.Graph(n, n, ii.ravel().astype(np.int32), jj.ravel().astype(np.int32), SYM | LOOPS)
    X = synth.uniform(7, n, 4).astype(np.float64)
    Y, S = g.fwd(X.astype(np.float32))
    assert np.all(np.abs(Y - X.mean(axis=0)[None, :]) <= 2.0**-23 * S)


def test_star_closed_form():
    k = 1000
    src = np.arange(1, k + 1, dtype=np.int32)
    dst = np.zeros(k, np.int32)
    g = oracle.Graph(k + 1, k + 1, src, dst, SYM | LOOPS)
    val = dict(zip(zip(np.repeat(np.arange(k + 1), np.diff(g.csr_ptr)), g.csr_idx), g.csr_val))
    assert val[(0, 0)] == np.float32(1.0 / (k + 1))
    assert val[(0, 5)] == np.float32(1.0 / math.sqrt(2 * (k + 1)))
    assert val[(5, 0)] == val[(0, 5)]
    assert val[(5, 5)] == np.float32(0.5)


def _read_golden(name):
    edges, entries = [], []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            parts = line.split()
            if parts[0] == "edges":
                edges.append((int(parts[1]), int(parts[2])))
            else:
                entries.append((int(parts[0]), int(parts[1]), float(parts[2])))
    return edges, entries


@pytest.mark.parametrize("name", ["path3_ahat.txt", "star3_ahat.txt"])
def test_golden_hand_derived(name):
    edges, entries = _read_golden(name)
    n = 1 + max(max(e) for e in edges)
    src = np.array([e[0] for e in edges], np.int32)
    dst = np.array([e[1] for e in edges], np.int32)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    got = csr_to_dense(g.csr_ptr, g.csr_idx, g.csr_val.astype(np.float64), n, n)
    want = np.zeros((n, n))
    for r, c, v in entries:
        want[r, c] = v
    assert np.array_equal(got != 0, want != 0)
    assert np.array_equal(got.astype(np.float32), want.astype(np.float32))


@pytest.mark.parametrize("name", ["path3_ahat.txt", "star3_ahat.txt"])
def test_golden_degrees_and_listed_normalization(name):
    # row_degrees counts the neighbours of the hand-derived graphs (the self-
    # loop left out), and normalize_listed, given each entry's row degree and
    # column degree, reproduces their hand-derived A_hat entries
    edges, entries = _read_golden(name)
    n = 1 + max(max(e) for e in edges)
    want_deg = np.zeros(n, np.int32)
    for a, b in edges:
        want_deg[a] += 1
        want_deg[b] += 1
    src = np.array([e[0] for e in edges], np.int32)
    dst = np.array([e[1] for e in edges], np.int32)
    ptr, idx = oracle.structure(n, n, src, dst, SYM | LOOPS)
    deg = oracle.row_degrees(ptr, idx)
    assert np.array_equal(deg, want_deg)
    rows = np.repeat(np.arange(n), np.diff(ptr))
    val = oracle.normalize_listed(ptr, deg, deg[idx])
    want = {(r, c): np.float32(v) for r, c, v in entries}
    assert len(want) == len(idx)
    for r, c, v in zip(rows, idx, val):
        assert v == want[(int(r), int(c))], (r, c, v)


def test_degrees_closed_forms():
    # star: the centre has k neighbours, every leaf one; complete graph on m
    # nodes: m - 1 each; drawn self-loops and duplicates count no neighbour
    k, m = 300, 40
    ptr, idx = oracle.structure(k + 1, k + 1, np.arange(1, k + 1, dtype=np.int32),
                                np.zeros(k, np.int32), SYM | LOOPS)
    deg = oracle.row_degrees(ptr, idx)
    assert deg[0] == k and np.all(deg[1:] == 1)
    u, v = np.triu_indices(m, 1)
    src = np.concatenate([u, u, np.arange(m)]).astype(np.int32)
    dst = np.concatenate([v, v, np.arange(m)]).astype(np.int32)
    ptr, idx = oracle.structure(m, m, src, dst, SYM | LOOPS)
    assert np.all(oracle.row_degrees(ptr, idx) == m - 1)


# ---------------------------------------------------------------------------
# Sampled rows agree with the whole-matrix route.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("transpose", [False, True])
def test_rows_of_matches_structure(transpose):
    n = 3000
    src, dst = synth.rmat_edges(90, n, 20000, perm_seed=91)
    for flags in (SYM | LOOPS, LOOPS, 0):
        ptr, idx = oracle.structure(n, n, src, dst, flags, transpose)
        sel = np.unique(synth.splitmix64(92, 0, 300) % n).astype(np.int32)[::-1].copy()
        sp, si = oracle.rows_of(n, n, src, dst, flags, sel, transpose)
        for i, r in enumerate(sel):
            assert np.array_equal(si[sp[i]:sp[i + 1]], idx[ptr[r]:ptr[r + 1]])


def test_sampled_normalization_matches_graph():
    n = 2048
    src, dst = synth.rmat_edges(93, n, 16 * n, perm_seed=94)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    sel = np.array([0, 5, 77, 1000, 2047], np.int32)
    for transpose in (False, True):
        ptr, idx, val = oracle.sampled(n, n, src, dst, SYM | LOOPS, sel, transpose)
        gp = g.csc_ptr if transpose else g.csr_ptr
        gi = g.csc_idx if transpose else g.csr_idx
        gv = g.csc_val if transpose else g.csr_val
        for i, r in enumerate(sel):
            assert np.array_equal(idx[ptr[i]:ptr[i + 1]], gi[gp[r]:gp[r + 1]])
            assert np.array_equal(val[ptr[i]:ptr[i + 1]], gv[gp[r]:gp[r + 1]])


# ---------------------------------------------------------------------------
# Quantization (Section 2.4) and the fused dequantize path.
# ---------------------------------------------------------------------------

def test_quantizer_nearest_code_and_roundtrip():
    X = synth.normal(11, 400, 128)
    X[3, :] = 0.25          # constant row: S = 0, every code 0, dequant = Z
    X[4, :7] = [-3.0, 5.0, 1.0, 1.0, 2.0, -3.0, 5.0]
    Q, Z, S = oracle.quantize_rows(X)
    assert S[3] == 0 and np.all(Q[3] == 0)
    D = oracle.dequant_rows(Q, Z, S)
    assert np.all(D[3] == np.float32(0.25))
    assert np.array_equal(Z, X.min(axis=1))
    for i in range(X.shape[0]):
        if S[i] == 0:
            continue
        assert Q[i, np.argmin(X[i])] == 0
        assert Q[i, np.argmax(X[i])] == 255
        # round trip within half a step (plus float rounding)
        err = np.abs(X[i].astype(np.float64) - D[i])
        assert np.all(err <= 0.5 * S[i] * (1 + 1e-5) + 4 * np.spacing(np.abs(X[i]).max()))
        # the chosen code is the nearest of all 256 (brute force)
        codes = np.arange(256, dtype=np.float64)
        grid = codes[None, :] * np.float64(S[i]) + np.float64(Z[i])
        best = np.abs(X[i].astype(np.float64)[:, None] - grid).min(axis=1)
        chosen = np.abs(X[i].astype(np.float64) - (Q[i] * np.float64(S[i]) + Z[i]))
        assert np.all(chosen <= best + 1e-6 * S[i])


def test_dequant_single_rounding():
    # dequant is fmaf(q, S, Z): q = 0 gives Z exactly; compare to exact double
    assert oracle.dequant(0, 0.123, -7.5) == np.float32(-7.5)
    rng = np.random.default_rng(0)
    for _ in range(2000):
        q = int(rng.integers(0, 256))
        s = np.float32(rng.standard_normal() * 0.01)
        z = np.float32(rng.standard_normal())
        exact = q * np.float64(s) + np.float64(z)  # exact: 8-bit x 24-bit + 24-bit fits in 53
        assert oracle.dequant(q, s, z) == np.float32(exact)


def test_q8_permutation_graph_is_exact_dequant():
    # one entry per row into a distinct halo column, value 1, no self-loops:
    # Y = fmaf(1, deq, 0) = deq exactly
    n_local, n_halo, F = 50, 64, 40
    perm = synth.permutation(12, n_halo)
    src = (n_local + perm).astype(np.int32)
    dst = np.arange(n_halo, dtype=np.int32)
    ptr, idx = oracle.structure(n_halo, n_local + n_halo, src, dst, 0)
    val = np.ones(len(idx), np.float32)
    Xl = synth.uniform(13, n_local, F)
    Q = synth.random_bytes(14, n_halo, F)
    Z = synth.uniform(15, n_halo, 1)[:, 0]
    S = np.abs(synth.uniform(16, n_halo, 1)[:, 0]) * 0.01
    Y, _ = oracle.spmm_q8(ptr, idx, val, n_local, Xl, Q, Z, S)
    D = oracle.dequant_rows(Q, Z, S)
    assert np.array_equal(Y.astype(np.float32), D[perm])


def test_q8_matches_dequantized_then_plain():
    n = 900
    src, dst = synth.rmat_edges(17, n, 9000, perm_seed=18)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    n_lc = 675
    X = synth.normal(19, n, 24)
    Q, Z, S = oracle.quantize_rows(X[n_lc:])
    Xd = X.copy()
    Xd[n_lc:] = oracle.dequant_rows(Q, Z, S)
    Y1, S1 = oracle.spmm_q8(g.csr_ptr, g.csr_idx, g.csr_val, n_lc, X[:n_lc], Q, Z, S)
    Y2, S2 = g.fwd(Xd)
    assert np.array_equal(Y1, Y2) and np.array_equal(S1, S2)


# ---------------------------------------------------------------------------
# Two-layer GCN step: analytic gradients against finite differences.
# ---------------------------------------------------------------------------

def test_gcn_step_gradients_finite_difference():
    n, fin, hid, ncls = 60, 7, 6, 5
    src, dst = synth.rmat_edges(20, n, 240, perm_seed=21)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    X = synth.normal(22, n, fin).astype(np.float64)
    W1 = synth.glorot(23, fin, hid).astype(np.float64)
    W2 = synth.glorot(24, hid, ncls).astype(np.float64)
    y = synth.labels(25, n, ncls)
    out = oracle.gcn_step(g, X, W1, W2, y)
    eps = 1e-6
    for W, dW, which in ((W1, out["dW1"], 0), (W2, out["dW2"], 1)):
        for (i, j) in [(0, 0), (1, 2), (W.shape[0] - 1, W.shape[1] - 1), (3, 1)]:
            Wp, Wm = W.copy(), W.copy()
            Wp[i, j] += eps
            Wm[i, j] -= eps
            args_p = (Wp, W2) if which == 0 else (W1, Wp)
            args_m = (Wm, W2) if which == 0 else (W1, Wm)
            lp = oracle.gcn_step(g, X, *args_p, y)["loss"]
            lm = oracle.gcn_step(g, X, *args_m, y)["loss"]
            fd = (lp - lm) / (2 * eps)
            assert abs(fd - dW[i, j]) <= 1e-6 * max(1.0, abs(fd))


def test_gcn_step_initial_loss_near_log_classes():
    n, ncls = 400, 47
    src, dst = synth.rmat_edges(26, n, 3200, perm_seed=27)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    X = synth.normal(28, n, 100)
    out = oracle.gcn_step(g, X, synth.glorot(29, 100, 256), synth.glorot(30, 256, ncls),
                          synth.labels(31, n, ncls))
    assert abs(out["loss"] - math.log(ncls)) < 0.5


def test_gcn_forward_brute_force_loops():
    # The forward of the two-layer step written out with explicit loops from
    # the edge list (Section 2.1: each layer aggregates the neighbours' rows
    # of X W, then the activation; GCN's propagation matrix): neighbour sets
    # of the symmetrized edge list without drawn self pairs, d~ = |N(i)| + 1,
    # A_hat[i][j] = 1 / sqrt(d~_i d~_j) over N(i) and i itself;
    # H1 = relu(A_hat (X W1)), logits = A_hat (H1 W2), loss = mean of
    # log sum exp(logits) - logit of the label. A ReLU placed before the
    # aggregation, a dropped self term or a transposed weight fails here.
    n, fin, hid, ncls = 12, 3, 4, 3
    src, dst = synth.rmat_edges(34, n, 30, perm_seed=35)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    rng = np.random.default_rng(36)
    X = rng.normal(size=(n, fin))
    W1 = rng.normal(size=(fin, hid))
    W2 = rng.normal(size=(hid, ncls))
    y = rng.integers(0, ncls, n)
    nbr = [set() for _ in range(n)]
    for s, d in zip(src, dst):
        if s != d:
            nbr[d].add(int(s))
            nbr[s].add(int(d))
    dt = [len(nb) + 1 for nb in nbr]

    def agg(H):
        out = []
        for i in range(n):
            row = [H[i][f] / dt[i] for f in range(len(H[0]))]  # self term 1/sqrt(d~_i d~_i)
            for j in nbr[i]:
                w = 1.0 / math.sqrt(dt[i] * dt[j])
                row = [row[f] + w * H[j][f] for f in range(len(H[0]))]
            out.append(row)
        return out

    def matmul(H, W):
        return [[sum(H[i][k] * W[k][c] for k in range(len(W))) for c in range(len(W[0]))]
                for i in range(len(H))]

    H1 = [[max(v, 0.0) for v in row] for row in agg(matmul(X.tolist(), W1.tolist()))]
    logits = agg(matmul(H1, W2.tolist()))
    loss = 0.0
    for i in range(n):
        m = max(logits[i])
        loss += m + math.log(sum(math.exp(v - m) for v in logits[i])) - logits[i][y[i]]
    loss /= n
    out = oracle.gcn_step(g, X, W1, W2, y)
    # the oracle aggregates with fp32-rounded A_hat values: within 2^-24 relative per entry
    assert np.allclose(out["H1"], np.array(H1), rtol=1e-6, atol=1e-7)
    assert np.allclose(out["logits"], np.array(logits), rtol=1e-6, atol=1e-7)
    assert abs(out["loss"] - loss) <= 1e-6 * abs(loss)


def test_double_input_aggregation_matches_dense():
    # the float64-input aggregation of the training step against dense A_hat H
    n = 150
    src, dst = synth.er_edges(33, n, 600)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    A = dense_adjacency(n, n, src, dst, SYM | LOOPS)
    Ah = csr_to_dense(g.csr_ptr, g.csr_idx, g.csr_val.astype(np.float64), n, n)
    assert np.array_equal(Ah != 0, A != 0)
    H = np.random.default_rng(3).standard_normal((n, 7))
    got = oracle._agg64(g.csr_ptr, g.csr_idx, g.csr_val, H)
    assert np.allclose(got, Ah @ H, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------------------
# Producer side: LayerNorm (Section 6.1 step 2) and b-bit quantization.
# ---------------------------------------------------------------------------

def test_layernorm_moments_and_affine():
    X = synth.normal(40, 300, 100) * 7 + 3
    Y = oracle.layernorm_rows(X, eps=0.0).astype(np.float64)
    assert np.allclose(Y.mean(axis=1), 0, atol=1e-6)
    assert np.allclose(Y.var(axis=1), 1, rtol=1e-5)
    g = synth.uniform(41, 1, 100)[0]
    b = synth.uniform(42, 1, 100)[0]
    Y2 = oracle.layernorm_rows(X, g, b, eps=0.0).astype(np.float64)
    assert np.allclose(Y2, Y * g + b, rtol=1e-5, atol=1e-5)
    # a hand case: row (1, 2, 3, 4): mean 2.5, var 1.25
    Y3 = oracle.layernorm_rows(np.array([[1, 2, 3, 4]], np.float32), eps=0.0)
    assert np.allclose(Y3[0], (np.array([1, 2, 3, 4]) - 2.5) / np.sqrt(1.25), rtol=1e-6)
    # a constant row normalizes to beta (here 0) for eps > 0
    assert np.all(oracle.layernorm_rows(np.full((1, 9), 5.0, np.float32)) == 0)


@pytest.mark.parametrize("bits", [8, 2])
def test_bit_quantizer_nearest_code(bits):
    X = synth.normal(43, 200, 37)
    X[7] = -2.0
    Q, Z, S = oracle.quantize_rows_bits(X, bits)
    levels = (1 << bits) - 1
    D = oracle.dequant_rows_bits(Q, Z, S, 37, bits).astype(np.float64)
    assert S[7] == 0 and np.all(D[7] == -2.0)
    assert np.allclose(S[S > 0], (X.max(1) - X.min(1))[S > 0] / levels, rtol=1e-6)
    grid = np.arange(levels + 1, dtype=np.float64)
    F = X.shape[1]
    codes = Q[:, :F] if bits == 8 else (Q[:, np.arange(F) // 4] >> (2 * (np.arange(F) % 4))) & 3
    assert codes.max() <= levels
    for i in range(X.shape[0]):
        if S[i] == 0:
            continue
        cand = grid[None, :] * np.float64(S[i]) + np.float64(Z[i])
        best = np.abs(X[i].astype(np.float64)[:, None] - cand).min(axis=1)
        chosen = np.abs(X[i].astype(np.float64) - (codes[i] * np.float64(S[i]) + np.float64(Z[i])))
        assert np.all(chosen <= best + 1e-6 * S[i])
        # the dequantized fp32 value is that code's grid point, rounded once
        assert np.all(D[i] == (codes[i] * np.float64(S[i]) + np.float64(Z[i])).astype(np.float32))
    if bits == 8:
        Q8, Z8, S8 = oracle.quantize_rows(X)
        assert np.array_equal(Q, Q8) and np.array_equal(Z, Z8) and np.array_equal(S, S8)


def test_int2_packing_layout():
    # feature f of a row sits in bits [2(f % 4), 2(f % 4) + 2) of byte f / 4
    X = np.array([[0.0, 1.0, 2.0, 3.0, 3.0, 0.0]], np.float32)
    Q, Z, S = oracle.quantize_rows_bits(X, 2)
    assert Z[0] == 0 and S[0] == 1
    assert Q.shape == (1, 2)
    assert Q[0, 0] == 0 | (1 << 2) | (2 << 4) | (3 << 6)
    assert Q[0, 1] == 3  # features 4, 5 = (3, 0); padding codes are 0


def test_int2_halo_aggregation_matches_dequantized_plain():
    n = 500
    src, dst = synth.rmat_edges(44, n, 5000, perm_seed=45)
    g = oracle.Graph(n, n, src, dst, SYM | LOOPS)
    nlc, F = 375, 19
    X = synth.normal(46, n, F)
    Q, Z, S = oracle.quantize_rows_bits(X[nlc:], 2)
    Xd = X.copy()
    Xd[nlc:] = oracle.dequant_rows_bits(Q, Z, S, F, 2)
    Y1, S1 = oracle.spmm_qbits(g.csr_ptr, g.csr_idx, g.csr_val, nlc, X[:nlc], Q, Z, S, F, 2)
    Y2, S2 = g.fwd(Xd)
    assert np.array_equal(Y1, Y2) and np.array_equal(S1, S2)


# ---------------------------------------------------------------------------
# Algorithm 1 (Section 5.2): minimum vertex cover and the pre/post split.
# ---------------------------------------------------------------------------

def _brute_force_cover(eu, ev, n_u, n_v):
    import itertools
    verts = [("u", i) for i in range(n_u)] + [("v", j) for j in range(n_v)]
    for k in range(len(verts) + 1):
        for comb in itertools.combinations(verts, k):
            c = set(comb)
            if all(("u", a) in c or ("v", b) in c for a, b in zip(eu, ev)):
                return k
    return len(verts)


def test_golden_prepost_fig4():
    edges, expect = [], {}
    for line in open(os.path.join(GOLDEN, "prepost_fig4.txt")):
        line = line.split("#", 1)[0].split()
        if not line:
            continue
        if line[0].isdigit():
            edges.append((int(line[0]), int(line[1])))
        else:
            expect.setdefault(line[0], []).append([int(t) for t in line[1:]])
    src = np.array([e[0] for e in edges])
    dst = np.array([e[1] for e in edges])
    is_post, vol, cov_src, cov_dst = oracle.prepost_split(src, dst)
    assert len(edges) == expect["volume_edges"][0][0]
    assert len(np.unique(dst)) == expect["volume_pre"][0][0]
    assert len(np.unique(src)) == expect["volume_post"][0][0]
    assert vol == expect["volume_hybrid"][0][0]
    assert sorted(list(cov_src) + list(cov_dst)) == expect["cover"][0]
    got = {("post" if p else "pre", int(s), int(d)) for p, s, d in zip(is_post, src, dst)}
    want = {(k, a, b) for k in ("post", "pre") for a, b in expect.get(k, [])}
    assert got == want


@pytest.mark.parametrize("seed", range(12))
def test_cover_is_minimum_brute_force(seed):
    # Koenig: cover size = maximum matching = the brute-force minimum cover
    rng = np.random.default_rng(seed)
    n_u, n_v = int(rng.integers(1, 7)), int(rng.integers(1, 7))
    m = int(rng.integers(1, 14))
    eu = rng.integers(0, n_u, m).astype(np.int32)
    ev = rng.integers(0, n_v, m).astype(np.int32)
    size, cu, cv = oracle.bipartite_cover(eu, ev, n_u, n_v)
    assert np.all(cu[eu] | cv[ev])
    assert cu.sum() + cv.sum() == size
    assert size == _brute_force_cover(eu, ev, n_u, n_v)


def test_split_covers_every_edge_on_random_remote_graph():
    src, dst = synth.rmat_edges(47, 5000, 20000, perm_seed=48)
    dst = dst + 10000  # the two workers' node ids are disjoint
    is_post, vol, cs, cd = oracle.prepost_split(src, dst)
    cover_s, cover_d = set(cs.tolist()), set(cd.tolist())
    assert all((s in cover_s) == p for s, p in zip(src, is_post))
    assert all(d in cover_d for d, p in zip(dst, is_post) if not p)
    assert vol == len(cover_s) + len(cover_d)
    assert vol <= min(len(np.unique(src)), len(np.unique(dst)))


# ---------------------------------------------------------------------------
# GraphSAGE-mean (Section 2.1 with AGGREGATE = mean; the evaluation model of
# Table 2) and masked label propagation (Section 6.1 step 1, Lemma 2).
# ---------------------------------------------------------------------------

def _dense_binary(n, src, dst, flags):
    A = np.zeros((n, n))
    for s, d in zip(src, dst):
        if s == d and flags & LOOPS:
            continue
        A[d, s] = 1
        if flags & SYM:
            A[s, d] = 1
    if flags & LOOPS:
        A[np.arange(n), np.arange(n)] = 1
    return A


@pytest.mark.parametrize("flags", [SYM, 0, SYM | LOOPS])
def test_mean_values_match_dense(flags):
    n = 40
    src, dst = synth.er_edges(50 + flags, n, 90)
    g = oracle.Graph(n, n, src, dst, flags, mean=True)
    A = _dense_binary(n, src, dst, flags)
    lens = A.sum(axis=1)
    M = np.divide(A, lens[:, None], out=np.zeros_like(A), where=lens[:, None] > 0)
    D = np.zeros((n, n))
    rows = np.repeat(np.arange(n), np.diff(g.csr_ptr))
    D[rows, g.csr_idx] = g.csr_val
    assert np.array_equal(D != 0, A != 0)
    assert np.array_equal(D, M.astype(np.float32).astype(np.float64))
    T = np.zeros((n, n))
    cols = np.repeat(np.arange(n), np.diff(g.csc_ptr))
    T[cols, g.csc_idx] = g.csc_val
    assert np.array_equal(T, D.T)
    # D^-1 A 1 = 1 on rows with entries
    ones, _ = g.fwd(np.ones((n, 1), np.float32))
    assert np.allclose(ones[lens > 0, 0], 1.0, atol=1e-6) and np.all(ones[lens == 0] == 0)


def test_mean_values_star_closed_form():
    k = 7
    src = np.arange(1, k + 1, dtype=np.int32)
    dst = np.zeros(k, np.int32)
    g = oracle.Graph(k + 1, k + 1, src, dst, SYM, mean=True)
    assert np.all(g.csr_val[g.csr_ptr[0]:g.csr_ptr[1]] == np.float32(1.0 / k))
    assert np.all(g.csr_val[g.csr_ptr[1]:] == 1.0)


def _sage_case(seed, n=50, f_in=6, hidden=5, C=4, lp=False):
    src, dst = synth.er_edges(seed, n, 3 * n)
    g = oracle.Graph(n, n, src, dst, SYM, mean=True)
    rng = np.random.default_rng(seed)
    X = rng.normal(size=(n, f_in))
    dims = [(f_in, hidden), (hidden, hidden), (hidden, C)]
    params = []
    for a, b in dims:
        params += [rng.normal(size=(a, b)) * 0.5, rng.normal(size=(a, b)) * 0.5, rng.normal(size=b) * 0.1]
    y = rng.integers(0, C, n)
    mask = (rng.random(n) < 0.4).astype(np.uint8) if lp else None
    E = rng.normal(size=(C, f_in)) if lp else None
    return g, X, params, y, mask, E, src, dst


@pytest.mark.parametrize("lp", [False, True])
def test_sage_step_gradients_finite_difference(lp):
    g, X, params, y, mask, E, _, _ = _sage_case(60, lp=lp)
    out = oracle.sage_step(g, X, params, y, mask, E)
    rng = np.random.default_rng(61)
    h = 1e-6
    targets = [(k, params) for k in range(9)] + ([("E", None)] if lp else [])
    for k, _ in targets:
        P = E if k == "E" else params[k]
        G = out["dE"] if k == "E" else out["grads"][k]
        assert G.shape == P.shape
        for _ in range(4):
            i = tuple(rng.integers(0, s) for s in P.shape)
            old = P[i]
            P[i] = old + h
            lp_ = oracle.sage_step(g, X, params, y, mask, E)["loss"]
            P[i] = old - h
            lm = oracle.sage_step(g, X, params, y, mask, E)["loss"]
            P[i] = old
            fd = (lp_ - lm) / (2 * h)
            assert abs(fd - G[i]) <= 1e-6 * max(1.0, abs(fd)) + 1e-8, (k, i, fd, G[i])


def test_sage_forward_brute_force_loops():
    g, X, params, y, _, _, src, dst = _sage_case(62, n=12, f_in=3, hidden=4, C=3)
    n = X.shape[0]
    # neighbours: the deduplicated, symmetrized edge list; a drawn self pair
    # counts as an edge (no self-loop is added, the root term is separate)
    nbr = [set() for _ in range(n)]
    for s, d in zip(src, dst):
        nbr[d].add(int(s))
        nbr[s].add(int(d))
    H = [list(map(float, row)) for row in X]
    for l in range(3):
        Ws, Wn, b = params[3 * l], params[3 * l + 1], params[3 * l + 2]
        Y = []
        for row in H:
            mu = sum(row) / len(row)
            var = sum((v - mu) ** 2 for v in row) / len(row)
            Y.append([(v - mu) / math.sqrt(var + 1e-5) for v in row])
        Z = []
        for i in range(n):
            nb = sorted(nbr[i])
            Z.append([sum(Y[j][f] for j in nb) / len(nb) if nb else 0.0 for f in range(len(Y[0]))])
        out = []
        for i in range(n):
            o = [b[c] + sum(Y[i][f] * Ws[f][c] + Z[i][f] * Wn[f][c] for f in range(len(Y[0])))
                 for c in range(len(b))]
            out.append([max(v, 0.0) for v in o] if l < 2 else o)
        H = out
    logits = oracle.sage_step(g, X, params, y)["logits"]
    # the oracle aggregates with fp32-rounded 1/len values: within 2^-24 relative
    assert np.allclose(logits, np.array(H), rtol=1e-6, atol=1e-6)


def test_sage_label_propagation_reduces_to_plain_step():
    g, X, params, y, _, _, _, _ = _sage_case(63)
    base = oracle.sage_step(g, X, params, y)
    zero = oracle.sage_step(g, X, params, y, np.zeros(len(y), np.uint8), np.ones((4, 6)))
    assert zero["loss"] == base["loss"]
    assert all(np.array_equal(a, b) for a, b in zip(zero["grads"], base["grads"]))
    assert np.all(zero["dE"] == 0)
    # an embedded row's input is X + E[label]: the same as adding it to X directly
    mask = np.zeros(len(y), np.uint8)
    mask[5] = 1
    E = np.arange(24, dtype=np.float64).reshape(4, 6)
    a = oracle.sage_step(g, X, params, y, mask, E)
    X2 = X.copy()
    X2[5] += E[y[5]]
    keep = np.ones(len(y), np.uint8)
    keep[5] = 0
    b = oracle.sage_step(g, X2, params, y, np.where(keep == 1, 0, 1).astype(np.uint8),
                         np.zeros((4, 6)))
    assert abs(a["loss"] - b["loss"]) < 1e-12


def test_sage_initial_loss_near_log_classes():
    g, X, params, y, _, _, _, _ = _sage_case(64, n=200, C=10)
    small = [p * 1e-3 for p in params]
    assert abs(oracle.sage_step(g, X, small, y)["loss"] - math.log(10)) < 1e-3
