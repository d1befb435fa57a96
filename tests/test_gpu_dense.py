"""GPU parity of the dense side of a layer and of the 2-layer GCN step.

GEMMs are compared with float64 products of the same fp32 inputs, within
1e-5 of the sum of |terms| per element (fp32 accumulation); the TN product is
also checked for identical bits across runs. Softmax cross-entropy against
its float64 definition. The whole step against the oracle's float64 step on a small graph and on the
product-shaped graph: the loss within 1e-5 relative, dW1 and dW2 within
1e-5 of the sum of |products| of their last GEMM.
"""

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


# (narrow outputs, N <= 64, take the register-streaming kernel: 1 to 4
# column tiles, K tails within a 16-deep chunk, partial last wavefronts)
SHAPES = [(1, 1, 1), (64, 64, 32), (1000, 47, 256), (777, 256, 100), (130, 100, 5),
          (4099, 33, 47), (517, 20, 516), (3001, 48, 1030), (95, 16, 17)]


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_gemm_nn_nt(G, M, N, K):
    note("gemm nn/nt %dx%dx%d" % (M, N, K))
    A = synth.uniform(201, M, K)
    B = synth.uniform(202, K, N)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    S = np.abs(A).astype(np.float64) @ np.abs(B).astype(np.float64)
    C = host(G.gcn_gemm_f32(G.GCN_GEMM_NN, dev(A), dev(B)))
    assert_close(C, ref, S, what="NN")
    Bt = np.ascontiguousarray(B.T)
    C2 = host(G.gcn_gemm_f32(G.GCN_GEMM_NT, dev(A), dev(Bt)))
    assert_close(C2, ref, S, what="NT")


# Tall products (M >= 65536) whose B fits in LDS take the resident-B kernel:
# 48-column slices (N <= 48) and 256-column slices (N > 128), K tails of 0
# to 15 past the last 16-deep chunk, every ring shape (chunk counts
# divisible by 8, 4, 2 and odd; for 256 columns by 4, 3, 2 and odd), several
# tiles per wavefront (M up to 10^6), a partial last column slice (N = 300),
# 16-byte aligned C rows (ldc a multiple of 4) and C rows of odd stride
# (element stores); a repeated call gives identical bits. K < 16 and
# 48 < N <= 128 check the staged tile.
RESIDENT = [(1000003, 47, 47), (65573, 48, 516), (65536, 1, 4), (70001, 16, 17),
            (65573, 33, 15), (65573, 40, 68), (65573, 48, 48), (65573, 48, 640),
            (131101, 47, 256), (500003, 256, 100), (65573, 300, 47), (65573, 512, 48),
            (65573, 129, 112), (65573, 200, 16), (65573, 256, 64), (65573, 100, 100)]


def _ld4(n):
    return (n + 3) // 4 * 4


@pytest.mark.parametrize("M,N,K", RESIDENT)
def test_gemm_resident_b(G, M, N, K):
    import torch
    note("gemm resident-B %dx%dx%d" % (M, N, K))
    A = synth.uniform(211, M, K, ld=_ld4(K))
    B = synth.uniform(212, K, N, ld=_ld4(N))
    A64 = A[:, :K].astype(np.float64)
    B64 = B[:, :N].astype(np.float64)
    ref = A64 @ B64
    S = np.abs(A64) @ np.abs(B64)
    del A64, B64
    Ad = dev(A)[:, :K]
    for aligned in (True, False):
        ldc = _ld4(N) if aligned else (N | 1) + 2 * (N % 2)
        Cfull = torch.full((M, ldc), 7.0, device="cuda:0")
        C = G.gcn_gemm_f32(G.GCN_GEMM_NN, Ad, dev(B)[:, :N], C=Cfull[:, :N])
        Ch = host(Cfull)
        assert_close(Ch[:, :N], ref, S, what="NN ldc %d" % ldc)
        assert np.all(Ch[:, N:] == 7.0)
        del C, Cfull, Ch
    Bt = np.zeros((N, _ld4(K)), np.float32)
    Bt[:, :K] = B[:, :N].T
    C2 = G.gcn_gemm_f32(G.GCN_GEMM_NT, Ad, dev(Bt)[:, :K],
                        C=torch.empty((M, _ld4(N)), device="cuda:0")[:, :N])
    assert_close(host(C2), ref, S, what="NT")
    C3 = G.gcn_gemm_f32(G.GCN_GEMM_NT, Ad, dev(Bt)[:, :K],
                        C=torch.empty((M, _ld4(N)), device="cuda:0")[:, :N])
    assert torch.equal(C2.view(torch.int32), C3.view(torch.int32)), "NT not bit-identical"


# The staged A^T B tile takes ceil(M / 16 / ceil(M / 128)) wavefronts: 1, 2,
# 3, 7 (M = 100, 200, 516) and 8 (M = 256) are covered below.
@pytest.mark.parametrize("K,M,N", [(5, 3, 2), (8192, 100, 256), (20000, 256, 47),
                                   (100003, 64, 64), (33, 1, 300), (20000, 200, 256),
                                   (20000, 48, 100), (20011, 516, 128), (8192, 20, 96),
                                   (8192, 16, 68)])
def test_gemm_tn_split_k(G, K, M, N):
    import torch
    note("gemm tn %dx%dx%d" % (K, M, N))
    A = synth.uniform(203, K, M)
    B = synth.uniform(204, K, N)
    ref = A.T.astype(np.float64) @ B.astype(np.float64)
    S = np.abs(A).T.astype(np.float64) @ np.abs(B).astype(np.float64)
    Ad, Bd = dev(A), dev(B)
    C = G.gcn_gemm_f32(G.GCN_GEMM_TN, Ad, Bd)
    assert_close(host(C), ref, S, what="TN")
    C2 = G.gcn_gemm_f32(G.GCN_GEMM_TN, Ad, Bd)
    assert torch.equal(C.view(torch.int32), C2.view(torch.int32))


# Weight-gradient shapes (K = nodes >= 65536, N <= 64, at most 16 output
# tiles of 64 x 64) take the streaming A^T B kernel: dW2 (256 x 47), a
# GraphSAGE class layer (516 x 47, two workgroups of tiles), one-column and
# ragged tiles, K not a multiple of 4 (a partial last step), 16-byte aligned
# rows (leading dimensions padded to a multiple of 4); dW1 (100 x 256) checks
# the staged tile at the same depth. Also checked: identical bits on a
# second run.
TN_STREAM = [(1000003, 256, 47), (300007, 100, 256), (65536, 516, 47), (70001, 33, 5),
             (65539, 1, 1), (131072, 64, 64)]


@pytest.mark.parametrize("K,M,N", TN_STREAM)
def test_gemm_tn_stream(G, K, M, N):
    import torch
    note("gemm tn stream %dx%dx%d" % (K, M, N))
    A = synth.uniform(213, K, M, ld=_ld4(M))
    B = synth.uniform(214, K, N, ld=_ld4(N))
    A64 = A[:, :M].astype(np.float64)
    B64 = B[:, :N].astype(np.float64)
    ref = A64.T @ B64
    S = np.abs(A64).T @ np.abs(B64)
    del A64, B64
    Ad, Bd = dev(A)[:, :M], dev(B)[:, :N]
    C = G.gcn_gemm_f32(G.GCN_GEMM_TN, Ad, Bd)
    assert_close(host(C), ref, S, what="TN stream")
    C2 = G.gcn_gemm_f32(G.GCN_GEMM_TN, Ad, Bd)
    assert torch.equal(C.view(torch.int32), C2.view(torch.int32))


def test_gemm_strided_operands(G):
    import torch
    note("gemm strided")
    A = synth.uniform(205, 300, 40, ld=44)
    B = synth.uniform(206, 40, 20, ld=23)
    Cfull = torch.full((300, 25), 3.0, device="cuda:0")
    G.gcn_gemm_f32(G.GCN_GEMM_NN, dev(A)[:, :40], dev(B)[:, :20], C=Cfull[:, :20])
    ref = A[:, :40].astype(np.float64) @ B[:, :20].astype(np.float64)
    S = np.abs(A[:, :40]).astype(np.float64) @ np.abs(B[:, :20]).astype(np.float64)
    Ch = host(Cfull)
    assert_close(Ch[:, :20], ref, S, what="strided")
    assert np.all(Ch[:, 20:] == 3.0)


def test_relu_and_backward(G):
    note("relu")
    H = synth.uniform(207, 1000, 70)
    dH = synth.uniform(208, 1000, 70)
    Hd = dev(H)
    G.gcn_relu(Hd)
    assert np.array_equal(host(Hd), np.maximum(H, 0))
    dHd = dev(dH)
    G.gcn_relu_bwd(Hd, dHd)
    assert np.array_equal(host(dHd), np.where(H > 0, dH, 0).astype(np.float32))


# class counts on both sides of each 16-class step of the kernel's lane
# layout (16 lanes per row, C / 16 rounded up classes per lane), row counts
# that leave a wavefront's 16 rows and a workgroup's 64 rows ragged
@pytest.mark.parametrize("n,C", [(1, 1), (5000, 47), (333, 64), (100, 2), (1000, 16), (64, 17),
                                 (777, 32), (129, 33), (2047, 48), (70, 49)])
def test_softmax_xent(G, n, C):
    note("softmax xent n=%d C=%d" % (n, C))
    z = synth.normal(209, n, C) * 3
    y = synth.labels(210, n, C)
    loss, d = G.gcn_softmax_xent(dev(z), dev(y))
    z64 = z.astype(np.float64)
    m = z64.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(z64 - m).sum(axis=1))
    ref = np.mean(lse - z64[np.arange(n), y])
    assert abs(float(loss) - ref) <= 1e-6 * max(1.0, abs(ref))
    P = np.exp(z64 - lse[:, None])
    P[np.arange(n), y] -= 1.0
    P /= n
    assert np.allclose(host(d), P, rtol=1e-5, atol=1e-7 / n)


def _step_check(G, w, f_in, hidden, n_classes, seed):
    import torch
    g = G.gcn_build_csr(w.n_rows, w.n_cols, dev(w.src), dev(w.dst), w.flags)
    G.gcn_normalize(g)
    X = synth.normal(3000 + seed, w.n_rows, f_in)
    W1 = synth.glorot(5000 + seed, f_in, hidden)
    W2 = synth.glorot(5100 + seed, hidden, n_classes)
    y = synth.labels(5200 + seed, w.n_rows, n_classes)
    loss, dW1, dW2 = G.gcn_gcn2_step(g, dev(X), dev(W1), dev(W2), dev(y))
    torch.cuda.synchronize()
    og = oracle.Graph(w.n_rows, w.n_cols, w.src, w.dst, w.flags)
    ref = oracle.gcn_step(og, X, W1, W2, y)
    assert abs(float(loss) - ref["loss"]) <= 1e-5 * abs(ref["loss"]), (float(loss), ref["loss"])
    # Each weight-gradient element sums n products of mixed sign; its fp32
    # error scales with the magnitude of every product that can enter it:
    # |X|^T (A_hat^T |dH1|) with dH1 before the ReLU mask (an activation within
    # rounding of 0 may fall on either side), and |H1|^T (A_hat^T |dlogits|).
    S_dz1 = oracle._agg64(og.csc_ptr, og.csc_idx, og.csc_val, np.abs(ref["dH1"]))
    S_dz2 = oracle._agg64(og.csc_ptr, og.csc_idx, og.csc_val, np.abs(ref["dlogits"]))
    S1 = np.abs(X).astype(np.float64).T @ S_dz1
    S2 = np.abs(ref["H1"]).T @ S_dz2
    assert_close(host(dW1), ref["dW1"], S1, what="dW1")
    assert_close(host(dW2), ref["dW2"], S2, what="dW2")
    # repeated steps give identical bits
    loss2, dW1b, dW2b = G.gcn_gcn2_step(g, dev(X), dev(W1), dev(W2), dev(y))
    assert float(loss2) == float(loss)
    assert torch.equal(dW1b.view(torch.int32), dW1.view(torch.int32))
    assert torch.equal(dW2b.view(torch.int32), dW2.view(torch.int32))
    return float(loss)


def test_gcn_step_small(G):
    note("gcn step small")
    n = 3000
    src, dst = synth.rmat_edges(211, n, 12 * n, perm_seed=212)
    w = synth.Workload("rmat3000", n, n, src, dst, synth.SYMMETRIZE | synth.ADD_SELF_LOOPS, 100)
    _step_check(G, w, 100, 256, 47, 11)


def test_gcn_step_transform_first(G):
    # f_in > hidden: layer 1 multiplies X W1 before aggregating, and its
    # backward aggregates the gradient (the other association of the step)
    note("gcn step transform first")
    n = 2000
    src, dst = synth.rmat_edges(213, n, 10 * n, perm_seed=214)
    w = synth.Workload("rmat2000", n, n, src, dst, synth.SYMMETRIZE | synth.ADD_SELF_LOOPS, 300)
    _step_check(G, w, 300, 64, 10, 12)


def test_gcn_step_unaligned_inputs(G):
    # f_in = 101: X rows are not 16-byte aligned, so layer 1 aggregates them
    # on the scalar path before its product (P is stored padded to 104)
    note("gcn step unaligned inputs")
    n = 2000
    src, dst = synth.rmat_edges(215, n, 10 * n, perm_seed=216)
    w = synth.Workload("rmat2000", n, n, src, dst, synth.SYMMETRIZE | synth.ADD_SELF_LOOPS, 101)
    _step_check(G, w, 101, 128, 10, 14)


@pytest.mark.parametrize("n,f_in,hidden,C", [(1203, 20, 200, 33), (777, 60, 300, 16),
                                             (2000, 112, 128, 48), (35, 100, 256, 47),
                                             (500, 112, 256, 48), (16, 100, 256, 47),
                                             (17, 4, 32, 2)])
def test_gcn_step_fused_backward_shapes(G, n, f_in, hidden, C):
    # f_in <= 112 and C <= 48: layer 1's backward runs as one fused pass
    # (dZ1 in registers); f_in of 2, 4 and 7 16-column blocks, 1-3 class
    # blocks, hidden slices of 128 columns with partial ones, partial row
    # groups, and chunks of one group. With hidden <= 256 the forward is
    # fused too: step counts 8, 16, 25 and 28, a hidden width of 300 that
    # keeps the separate products, (112, 256, 48) whose weight tables take
    # the whole 160 KB of LDS, exactly one row group, and a one-step input
    # with two classes
    note("gcn step fused backward n=%d f_in=%d hidden=%d C=%d" % (n, f_in, hidden, C))
    src, dst = synth.rmat_edges(217 + n, n, 8 * n, perm_seed=218)
    w = synth.Workload("rmat%d" % n, n, n, src, dst, synth.SYMMETRIZE | synth.ADD_SELF_LOOPS, f_in)
    _step_check(G, w, f_in, hidden, C, 15)


def test_gcn_step_product_like(G):
    import gc
    import torch
    note("gcn step product-like full size")
    w = synth.product_like()
    loss = _step_check(G, w, 100, 256, 47, 3)
    assert abs(loss - np.log(47)) < 0.5
    gc.collect()
    torch.cuda.empty_cache()

