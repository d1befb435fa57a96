"""GPU parity of the producer side (LayerNorm + b-bit quantization, Section
6.1 steps 2-3 and Section 7.3) and of the 2-bit halo aggregation.

Without LayerNorm the codes and parameters are bit-exact. With it, both
sides compute the row statistics in double, whose summation order differs,
then round once to fp32: the normalized values must agree to the last bit
on at least 99.9% of rows and within one ulp everywhere. The codes and
parameters are then checked on every row, bit for bit: against the oracle's
quantizer applied to the kernel's own normalized rows (the same fp32
computation on the same numbers), and, on the rows whose normalized values
agree exactly, against the oracle's whole LayerNorm + quantize chain.
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


def check_codes_every_row(q, z, s, y, bits):
    """Codes and (Z, S) of every row equal the oracle's quantizer applied to
    the kernel's own normalized rows y, bit for bit."""
    Qy, Zy, Sy = oracle.quantize_rows_bits(y, bits)
    assert np.array_equal(q, Qy), "codes differ on %d rows" % np.any(q != Qy, axis=1).sum()
    assert np.array_equal(z.view(np.uint32), Zy.view(np.uint32))
    assert np.array_equal(s.view(np.uint32), Sy.view(np.uint32))


@pytest.mark.parametrize("bits", [8, 2])
@pytest.mark.parametrize("F", [128, 47, 3])
def test_quantize_without_layernorm_bit_exact(G, bits, F):
    note("quantize bits=%d F=%d" % (bits, F))
    X = synth.normal(301, 2000, F)
    X[9] = 0.5
    Q, Z, S = oracle.quantize_rows_bits(X, bits)
    q, z, s = G.gcn_layernorm_quantize(dev(X), bits=bits, layernorm=False)
    assert np.array_equal(host(q), Q)
    assert np.array_equal(host(z).view(np.uint32), Z.view(np.uint32))
    assert np.array_equal(host(s).view(np.uint32), S.view(np.uint32))


@pytest.mark.parametrize("bits", [8, 2])
@pytest.mark.parametrize("F", [128, 100])
def test_layernorm_quantize(G, bits, F):
    note("layernorm quantize bits=%d F=%d" % (bits, F))
    n = 20000
    X = synth.normal(302, n, F) * 5 + 2
    gamma = 1 + 0.1 * synth.uniform(303, 1, F)[0]
    beta = 0.1 * synth.uniform(304, 1, F)[0]
    Yr = oracle.layernorm_rows(X, gamma, beta, eps=1e-5)
    Qr, Zr, Sr = oracle.quantize_rows_bits(Yr, bits)
    q, z, s, y = G.gcn_layernorm_quantize(dev(X), bits=bits, gamma=dev(gamma), beta=dev(beta),
                                          eps=1e-5, with_y=True)
    y, q, z, s = host(y), host(q), host(z), host(s)
    ulp = np.abs(y.view(np.int32).astype(np.int64) - Yr.view(np.int32).astype(np.int64))
    assert ulp.max() <= 1
    same = np.all(ulp == 0, axis=1)
    assert same.mean() >= 0.999
    check_codes_every_row(q, z, s, y, bits)
    assert np.array_equal(q[same], Qr[same])
    assert np.array_equal(z[same].view(np.uint32), Zr[same].view(np.uint32))
    assert np.array_equal(s[same].view(np.uint32), Sr[same].view(np.uint32))


@pytest.mark.parametrize("bits", [8, 2])
@pytest.mark.parametrize("F", [128, 100])
def test_quantize_special_values_bit_exact(G, bits, F):
    # NaN features get code 0 on both sides (a NaN never wins the min or max
    # of the row, and clamping maps it to 0); a row holding an infinite
    # feature has an infinite scale, which the kernel quantizes by division;
    # a constant row with NaNs has S = 0. NaNs stay off the first feature,
    # where the oracle's running min and max would start from them.
    note("quantize special values bits=%d F=%d" % (bits, F))
    n = 600
    X = synth.normal(310, n, F)
    rng = np.random.default_rng(311)
    for i in range(0, n, 3):
        X[i, rng.integers(1, F, 3)] = np.nan
    X[1, 5] = np.inf
    X[4, 7] = -np.inf
    X[7, 2], X[7, 9] = np.inf, -np.inf
    X[10, 1:] = np.nan
    X[13] = 0.25
    X[13, 3] = np.nan
    X[16, 1:] = 3.0e38  # the range overflows to +inf
    X[16, 0] = -3.0e38
    Q, Z, S = oracle.quantize_rows_bits(X, bits)
    assert np.isinf(S[[1, 4, 7, 16]]).all() and S[10] == 0 and S[13] == 0
    q, z, s = G.gcn_layernorm_quantize(dev(X), bits=bits, layernorm=False)
    assert np.array_equal(host(z).view(np.uint32), Z.view(np.uint32))
    assert np.array_equal(host(s).view(np.uint32), S.view(np.uint32))
    assert np.array_equal(host(q), Q), "codes differ on %d rows" % np.any(host(q) != Q, axis=1).sum()


def near_half_step_rows(seed, n, F, bits, scale_exp):
    """Rows whose values sit on and around the midpoints between codes: the
    row's minimum is 0 and its maximum (2^bits - 1) * S0, the others are
    (k + 1/2) * S nudged by -2 .. +2 ulps, where S is the scale the quantizer
    will compute from the row; S0 is drawn around 2^scale_exp."""
    rng = np.random.default_rng(seed)
    levels = (1 << bits) - 1
    X = np.zeros((n, F), np.float32)
    for i in range(n):
        s0 = np.float32(np.ldexp(1.0 + rng.random(), scale_exp))
        mx = np.float32(levels * s0)
        s = np.float32(mx / np.float32(levels))  # the quantizer's S, in fp32
        k = rng.integers(0, levels, F).astype(np.float64)
        v = ((k + 0.5) * np.float64(s)).astype(np.float32)
        nudge = rng.integers(-2, 3, F).astype(np.int32)
        v = (v.view(np.int32) + nudge).view(np.float32)
        v = np.clip(v, np.float32(0), mx)
        v[0], v[1] = 0.0, mx
        X[i] = v
    return X


@pytest.mark.parametrize("bits", [8, 2])
@pytest.mark.parametrize("scale_exp", [0, -20, 30, -99, 99, -110, 110])
def test_quantize_codes_near_half_steps(G, bits, scale_exp):
    # codes where rounding the quotient (x - Z) / S decides between two codes:
    # bit-exact with the oracle's IEEE division, at scales inside and outside
    # the range where the kernel divides by multiplying with 1 / S
    note("quantize near half steps bits=%d 2^%d" % (bits, scale_exp))
    for F in (128, 100):
        X = near_half_step_rows(500 + scale_exp + bits, 600, F, bits, scale_exp)
        Q, Z, S = oracle.quantize_rows_bits(X, bits)
        q, z, s = G.gcn_layernorm_quantize(dev(X), bits=bits, layernorm=False)
        assert np.array_equal(host(s).view(np.uint32), S.view(np.uint32))
        assert np.array_equal(host(z).view(np.uint32), Z.view(np.uint32))
        assert np.array_equal(host(q), Q), "codes differ on %d rows" % np.any(host(q) != Q, axis=1).sum()


@pytest.mark.parametrize("F", [128, 64, 47])
def test_int2_halo_fwd_and_bwd(G, F):
    note("int2 halo F=%d" % F)
    n = 1 << 14
    src, dst = synth.rmat_edges(305, n, 16 * n, perm_seed=306)
    og = oracle.Graph(n, n, src, dst, synth.SYMMETRIZE | synth.ADD_SELF_LOOPS)
    g = G.gcn_build_csr(n, n, dev(src), dev(dst), synth.SYMMETRIZE | synth.ADD_SELF_LOOPS)
    G.gcn_normalize(g)
    nlc = n - n // 4
    X = synth.normal(307, n, F)
    Q, Z, S = oracle.quantize_rows_bits(X[nlc:], 2)
    zs = dev(np.stack([Z, S], axis=1))
    Y = host(G.gcn_aggregate_fwd_q8halo(g, nlc, dev(X[:nlc]), dev(Q), zs[:, 0], zs[:, 1], bits=2))
    assert_close(Y, *oracle.spmm_qbits(og.csr_ptr, og.csr_idx, og.csr_val, nlc, X[:nlc], Q, Z, S,
                                       F, 2), what="int2 fwd")
    dX = host(G.gcn_aggregate_fwd_q8halo(g, nlc, dev(X[:nlc]), dev(Q), zs[:, 0], zs[:, 1],
                                         use_csc=True, bits=2))
    assert_close(dX, *oracle.spmm_qbits(og.csc_ptr, og.csc_idx, og.csc_val, nlc, X[:nlc], Q, Z, S,
                                        F, 2), what="int2 bwd")


@pytest.mark.parametrize("F", [128, 47, 5])
def test_int2_permutation_dequant_bit_exact(G, F):
    note("int2 permutation F=%d" % F)
    n_local, n_halo = 300, 2048
    perm = synth.permutation(308, n_halo)
    src = (n_local + perm).astype(np.int32)
    dst = np.arange(n_halo, dtype=np.int32)
    g = G.gcn_build_csr(n_halo, n_local + n_halo, dev(src), dev(dst), 0)
    Q = synth.random_bytes(309, n_halo, (F + 3) // 4)
    if F % 4:  # padding codes of the last byte are 0, as the producer writes them
        Q[:, -1] &= (1 << (2 * (F % 4))) - 1
    Z = synth.normal(310, n_halo, 1)[:, 0]
    S = np.abs(synth.normal(311, n_halo, 1)[:, 0])
    Y = host(G.gcn_aggregate_fwd_q8halo(g, n_local, dev(synth.uniform(312, n_local, F)), dev(Q),
                                        dev(Z), dev(S), bits=2))
    D = oracle.dequant_rows_bits(Q, Z, S, F, 2)
    assert np.array_equal(Y.view(np.uint32), D[perm].view(np.uint32))


@pytest.mark.parametrize("bits", [8, 2])
@pytest.mark.parametrize("F,ld", [(64, 64), (256, 256), (512, 512), (1000, 1000), (47, 48),
                                  (1025, 1028), (6, 8)])
def test_quantize_register_kernel_shapes(G, bits, F, ld):
    # every row-width class of the register-resident kernel, ragged tails on a
    # padded leading dimension, and the row-per-wavefront kernel beyond 1024
    import torch
    note("quantize shapes bits=%d F=%d ld=%d" % (bits, F, ld))
    n = 1531  # not a multiple of any rows-per-block figure
    Xp = synth.normal(320 + F, n, ld)
    X = Xp[:, :F]
    Q, Z, S = oracle.quantize_rows_bits(X, bits)
    q, z, s = G.gcn_layernorm_quantize(dev(Xp)[:, :F], bits=bits, layernorm=False)
    assert np.array_equal(host(q), Q)
    assert np.array_equal(host(z).view(np.uint32), Z.view(np.uint32))
    assert np.array_equal(host(s).view(np.uint32), S.view(np.uint32))
    Yr = oracle.layernorm_rows(X)
    Qr, Zr, Sr = oracle.quantize_rows_bits(Yr, bits)
    q, z, s, y = G.gcn_layernorm_quantize(dev(Xp)[:, :F], bits=bits, with_y=True)
    y, q, z, s = host(y), host(q), host(z), host(s)
    ulp = np.abs(y.view(np.int32).astype(np.int64) - Yr.view(np.int32).astype(np.int64))
    assert ulp.max() <= 1
    same = np.all(ulp == 0, axis=1)
    assert same.mean() >= 0.99
    check_codes_every_row(q, z, s, y, bits)
    assert np.array_equal(q[same], Qr[same])
    assert np.array_equal(z[same].view(np.uint32), Zr[same].view(np.uint32))
    assert np.array_equal(s[same].view(np.uint32), Sr[same].view(np.uint32))
    if bits == 8:  # the plain u8 entry point shares the kernels
        qu, zu, su = G.gcn_quantize_rows_u8(dev(Xp)[:, :F])
        assert np.array_equal(host(qu), Q)
        assert np.array_equal(host(su).view(np.uint32), S.view(np.uint32))
    torch.cuda.synchronize()
