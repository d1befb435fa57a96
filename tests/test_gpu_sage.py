"""GPU parity of the GraphSAGE row: the mean operator D^-1 A, the LayerNorm
forward and backward kernels, and the 3-layer GraphSAGE training step with
and without masked label propagation, against the float64 oracle.

Tolerances. Mean values and structure are bit-exact. Aggregations with them
are within 1e-5 * S as every fp32 aggregation. LayerNorm values agree to the
last bit on at least 99.9% of rows and within one ulp everywhere (statistics
in double on both sides, summation order differs). The LayerNorm backward is
compared against the float64 formula applied to the kernel's own forward
output, per element within 1e-5 times the sum of the magnitudes of the
formula's terms. The training step runs in fp32 against float64 with the
GPU's own ReLU patterns (a unit whose pre-activation lies within fp32
rounding of 0 can fall either way, and a switched unit moves whole gradient
terms): the oracle reports every unit where the GPU's pattern differs from
float64's, and each must lie within 1e-5 of 0 relative to the magnitude of
its terms. Then the hidden outputs, the logits, every gradient and dE are
compared element by element within 1e-5 times the magnitude of their terms
(tests/step_bounds.py), and the loss within 1e-5 relative.
"""

import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_close, dev, host, note
from step_bounds import check_elementwise, sage_step_scales

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2411_16025_amd as pkg
    pkg.lib()
    return pkg


@pytest.mark.parametrize("flags,n,m", [(synth.SYMMETRIZE, 3000, 20000), (0, 2500, 30000),
                                       (synth.SYMMETRIZE | synth.ADD_SELF_LOOPS, 4096, 10000)])
def test_mean_values_bit_exact(G, flags, n, m):
    note("mean values flags=%d n=%d" % (flags, n))
    src, dst = synth.rmat_edges(400 + flags, n, m, perm_seed=401)
    og = oracle.Graph(n, n, src, dst, flags, mean=True)
    g = G.gcn_build_csr(n, n, dev(src), dev(dst), flags)
    G.gcn_normalize_mean(g)
    for which, (p, i, v) in ((0, (og.csr_ptr, og.csr_idx, og.csr_val)),
                             (1, (og.csc_ptr, og.csc_idx, og.csc_val))):
        ptr, idx, val = G.gcn_graph_export(g, which)
        assert np.array_equal(ptr, p) and np.array_equal(idx, i)
        assert np.array_equal(val.view(np.uint32), v.view(np.uint32)), "values of %d" % which
    X = synth.normal(402, n, 64)
    assert_close(host(G.gcn_aggregate_fwd(g, dev(X))), *og.fwd(X), what="mean fwd")
    assert_close(host(G.gcn_aggregate_bwd(g, dev(X))), *og.bwd(X), what="mean bwd")


def test_symmetric_normalization_after_mean(G):
    # a symmetric graph whose transpose got its own entries for the mean values
    # takes the symmetric normalization in both copies
    note("sym after mean")
    n = 2000
    src, dst = synth.er_edges(403, n, 8000)
    flags = synth.SYMMETRIZE | synth.ADD_SELF_LOOPS
    g = G.gcn_build_csr(n, n, dev(src), dev(dst), flags)
    G.gcn_normalize_mean(g)
    G.gcn_normalize(g)
    og = oracle.Graph(n, n, src, dst, flags)
    for which, v in ((0, og.csr_val), (1, og.csc_val)):
        _, _, val = G.gcn_graph_export(g, which)
        assert np.array_equal(val.view(np.uint32), v.view(np.uint32))


@pytest.mark.parametrize("F,ld", [(100, 100), (256, 256), (47, 48), (1100, 1100), (5, 7)])
def test_layernorm_fwd(G, F, ld):
    note("layernorm fwd F=%d" % F)
    n = 3001
    Xp = synth.normal(404 + F, n, ld) * 3 + 1
    X = Xp[:, :F]
    Y, rstd = G.gcn_layernorm_fwd(dev(Xp)[:, :F], eps=1e-5)
    Y, rstd = host(Y), host(rstd)
    ref = oracle.layernorm_rows(X, eps=1e-5)
    ulp = np.abs(Y.view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64))
    assert ulp.max() <= 1 and np.all(ulp == 0, axis=1).mean() >= 0.999
    _, r64 = oracle.layernorm64(X.astype(np.float64), 1e-5)
    assert np.allclose(rstd, r64, rtol=1e-6, atol=0)


@pytest.mark.parametrize("F,ld", [(100, 100), (256, 256), (47, 48), (1100, 1100), (32, 32),
                                  (64, 68), (512, 512), (100, 104)])
def test_layernorm_bwd(G, F, ld):
    note("layernorm bwd F=%d" % F)
    n = 2003
    X = synth.normal(410 + F, n, ld)[:, :F] * 2
    Yd, rd = G.gcn_layernorm_fwd(dev(X), eps=1e-5)
    # the gradients and the mask are passed as row views of ld-wide storage
    g1p = synth.normal(411 + F, n, ld)
    g2p = synth.normal(412 + F, n, ld)
    maskp = np.maximum(synth.normal(413 + F, n, ld), 0).astype(np.float32)
    g1, g2, mask = g1p[:, :F], g2p[:, :F], maskp[:, :F]
    Y, r = host(Yd).astype(np.float64), host(rd).astype(np.float64)
    g = (g1 + g2).astype(np.float64)  # the kernel adds the two in fp32
    for use2, usem in ((False, False), (True, True), (True, False), (False, True)):
        gg = g if use2 else g1.astype(np.float64)
        ref = oracle.layernorm64_bwd(Y, r, gg)
        S = r[:, None] * (np.abs(gg) + np.abs(gg).mean(1, keepdims=True)
                          + np.abs(Y) * np.abs(gg * Y).mean(1, keepdims=True))
        if usem:
            ref = ref * (mask > 0)
        out = host(G.gcn_layernorm_bwd(Yd, rd, dev(g1p)[:, :F], dev(g2p)[:, :F] if use2 else None,
                                       dev(maskp)[:, :F] if usem else None))
        assert np.all(np.abs(out - ref) <= 1e-5 * S + 1e-30), (use2, usem)


def test_layernorm_bwd_in_place_mask(G):
    # the step overwrites the ReLU output of the layer below with its gradient
    import torch
    n, F = 1000, 256
    X = synth.normal(420, n, F)
    Yd, rd = G.gcn_layernorm_fwd(dev(X))
    g1 = dev(synth.normal(421, n, F))
    H = dev(np.maximum(synth.normal(422, n, F), 0))
    want = host(G.gcn_layernorm_bwd(Yd, rd, g1, None, H.clone()))
    G.gcn_layernorm_bwd(Yd, rd, g1, None, H, dX=H)
    torch.cuda.synchronize()
    assert np.array_equal(host(H).view(np.uint32), want.view(np.uint32))


def sage_case(n, m, f_in, hidden, C, seed, lp):
    src, dst = synth.rmat_edges(seed, n, m, perm_seed=seed + 1)
    X = synth.normal(seed + 2, n, f_in)
    params = []
    for k, (a, b) in enumerate([(f_in, hidden), (hidden, hidden), (hidden, C)]):
        params += [synth.glorot(seed + 10 + 3 * k, a, b), synth.glorot(seed + 11 + 3 * k, a, b),
                   0.1 * synth.uniform(seed + 12 + 3 * k, 1, b)[0]]
    y = synth.labels(seed + 30, n, C)
    mask = (synth.uniform(seed + 31, n, 1)[:, 0] < 0.0).astype(np.uint8) if lp else None
    E = 0.5 * synth.normal(seed + 32, C, f_in) if lp else None
    return src, dst, X, params, y, mask, E


NAMES = ["W_self1", "W_neigh1", "b1", "W_self2", "W_neigh2", "b2", "W_self3", "W_neigh3", "b3"]


def check_against_oracle(og, X, params, y, mask, E, masks, hidden_out, logits, loss, grads, dE):
    """Run the oracle with the GPU's ReLU patterns, check that every unit
    where they differ from float64's is marginal, then compare the hidden
    outputs, logits, loss, gradients and dE element by element; the worst
    err/scale of each is printed. Returns the oracle's result."""
    ref = oracle.sage_step(og, X, params, y, mask, E, masks=masks)
    note("oracle step done")
    for l in range(2):
        fm = ref["flip_margins"][l]
        note("layer %d: %d units differ from float64's pattern (largest margin %.1e)"
             % (l + 1, fm.size, fm.max() if fm.size else 0.0))
        assert np.all(fm < 1e-5), "layer %d: a clear ReLU decision differs" % (l + 1)
    scales, s_dE, s_logits, s_hidden = sage_step_scales(og, params, y, mask, E, ref)
    note("error scales done")
    worst = {}
    for l in range(2):
        if hidden_out[l] is not None:
            # ReLU outputs: where both are 0 the pattern agrees; elsewhere O
            Yl, _, Zl, _ = ref["saved"][l]
            Pl = [np.asarray(p, np.float64) for p in params[3 * l:3 * l + 3]]
            O = (Yl @ Pl[0] + Zl @ Pl[1] + Pl[2]) * masks[l]
            worst["H%d" % (l + 1)] = check_elementwise(hidden_out[l], O, s_hidden[l],
                                                       what="H%d" % (l + 1))
            del O
    if logits is not None:
        worst["logits"] = check_elementwise(logits, ref["logits"], s_logits, what="logits")
    if loss is not None:
        assert abs(loss - ref["loss"]) <= 1e-5 * abs(ref["loss"]), (loss, ref["loss"])
    for nm, a, b, sc in zip(NAMES, grads, ref["grads"], scales):
        worst[nm] = check_elementwise(a, b, sc, what=nm)
    if dE is not None:
        worst["dE"] = check_elementwise(dE, ref["dE"], s_dE, what="dE")
    note("max err/scale " + " ".join("%s %.1e" % kv for kv in worst.items()))
    return ref


def check_step(G, n, m, f_in, hidden, C, seed, lp, flags=synth.SYMMETRIZE):
    """The step against the oracle run with the GPU's own ReLU patterns (from
    the forward entry point, whose activations are bit-identical to the
    step's)."""
    src, dst, X, params, y, mask, E = sage_case(n, m, f_in, hidden, C, seed, lp)
    og = oracle.Graph(n, n, src, dst, flags, mean=True)
    g = G.gcn_build_csr(n, n, dev(src), dev(dst), flags)
    G.gcn_normalize_mean(g)
    pd = [dev(p) for p in params]
    args = (dev(y), dev(mask) if lp else None, dev(E) if lp else None)
    H1, H2, logits = G.gcn_sage3_forward(g, dev(X), pd, *args)
    H1, H2 = host(H1), host(H2)
    masks = [H1 > 0, H2 > 0]
    loss, grads, dE = G.gcn_sage3_step(g, dev(X), pd, *args)
    got_loss = float(host(loss))
    got = [host(t) for t in grads]
    ref = check_against_oracle(og, X, params, y, mask, E, masks, [H1, H2], host(logits),
                               got_loss, got, host(dE) if lp else None)
    # a repeated step gives identical bits (its weight gradients run on a
    # second stream, forked from and joined to the caller's)
    loss2, grads2, dE2 = G.gcn_sage3_step(g, dev(X), pd, *args)
    assert float(host(loss2)) == got_loss
    for nm, a, b in zip(NAMES, got, grads2):
        assert np.array_equal(a.view(np.uint32), host(b).view(np.uint32)), nm
    if lp:
        assert np.array_equal(host(dE).view(np.uint32), host(dE2).view(np.uint32))
    return ref


@pytest.mark.parametrize("lp", [False, True])
# hidden 64, 128 and 48 (multiples of 16) take the fused class-layer backward
# (its input gradient and LayerNorm backward in one kernel), hidden 33 the
# separate product and LayerNorm backward
@pytest.mark.parametrize("n,f_in,hidden,C", [(3000, 100, 64, 10), (2000, 47, 33, 5),
                                             (2000, 50, 128, 47), (1500, 20, 48, 16)])
def test_sage_step_small(G, lp, n, f_in, hidden, C):
    note("sage step n=%d f_in=%d hidden=%d C=%d lp=%s" % (n, f_in, hidden, C, lp))
    check_step(G, n, 12 * n, f_in, hidden, C, 430 + n + f_in, lp)


def test_sage_step_product_full(G):
    """The step at the benchmark's size: the product-shaped graph (2,449,029
    nodes, symmetrized, no self-loops, mean aggregation), F_in 100, hidden 256,
    47 classes, labels of half of the nodes embedded. Every unit where the
    GPU's ReLU pattern differs from float64's is checked for its margin, then
    the logits, loss, every gradient and dE are compared element by element,
    as in the small cases."""
    import gc
    import torch
    note("sage step product-shaped full size")
    w = synth.product_like()
    n, f_in, hidden, C = w.n_rows, 100, 256, 47
    X = synth.normal(3003, n, f_in)
    params = []
    for k, (a, b) in enumerate([(f_in, hidden), (hidden, hidden), (hidden, C)]):
        params += [synth.glorot(5003 + 3 * k, a, b), synth.glorot(5004 + 3 * k, a, b),
                   0.1 * synth.uniform(5005 + 3 * k, 1, b)[0]]
    y = synth.labels(5203, n, C)
    mask = (synth.uniform(5204, n, 1)[:, 0] < 0.0).astype(np.uint8)
    E = 0.5 * synth.normal(5205, C, f_in)
    g = G.gcn_build_csr(n, n, dev(w.src), dev(w.dst), synth.SYMMETRIZE)
    G.gcn_normalize_mean(g)
    pd = [dev(p) for p in params]
    args = (dev(y), dev(mask), dev(E))
    H1, H2, logits = G.gcn_sage3_forward(g, dev(X), pd, *args)
    masks = [host(H1) > 0, host(H2) > 0]
    logits = host(logits)
    del H1, H2
    loss, grads, dE = G.gcn_sage3_step(g, dev(X), pd, *args)
    got = [host(t) for t in grads]
    got_dE = host(dE)
    got_loss = float(host(loss))
    del loss, grads, dE
    loss2, grads2, dE2 = G.gcn_sage3_step(g, dev(X), pd, *args)  # identical bits again
    assert float(host(loss2)) == got_loss
    for a, b in zip(got + [got_dE], [host(t) for t in grads2] + [host(dE2)]):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    del loss2, grads2, dE2
    g.free()
    torch.cuda.empty_cache()
    og = oracle.Graph(n, n, w.src, w.dst, synth.SYMMETRIZE, mean=True)
    del w
    gc.collect()
    check_against_oracle(og, X, params, y, mask, E, masks, [None, None], logits, got_loss, got,
                         got_dE)
    del og
    gc.collect()


@pytest.mark.parametrize("n,f_in,hidden,C,mask_kind", [
    (1500, 30, 20, 64, "half"),     # the widest class count, narrow rows (8-lane LayerNorm)
    (1200, 1030, 40, 7, "half"),    # inputs wider than the register LayerNorm kernel
    (1000, 16, 16, 3, "all"),       # every label embedded: no row in the loss
])
def test_sage_step_edge_cases(G, n, f_in, hidden, C, mask_kind):
    note("sage edge n=%d f_in=%d hidden=%d C=%d mask=%s" % (n, f_in, hidden, C, mask_kind))
    src, dst, X, params, y, mask, E = sage_case(n, 10 * n, f_in, hidden, C, 460 + f_in, True)
    if mask_kind == "all":
        mask[:] = 1
    og = oracle.Graph(n, n, src, dst, synth.SYMMETRIZE, mean=True)
    g = G.gcn_build_csr(n, n, dev(src), dev(dst), synth.SYMMETRIZE)
    G.gcn_normalize_mean(g)
    pd = [dev(p) for p in params]
    args = (dev(y), dev(mask), dev(E))
    H1, H2, logits = G.gcn_sage3_forward(g, dev(X), pd, *args)
    H1, H2 = host(H1), host(H2)
    masks = [H1 > 0, H2 > 0]
    loss, grads, dE = G.gcn_sage3_step(g, dev(X), pd, *args)
    got_loss = float(host(loss))
    got = [host(t) for t in grads]
    if mask_kind == "all":
        ref = oracle.sage_step(og, X, params, y, mask, E, masks=masks)
        assert got_loss == 0.0 and ref["loss"] == 0.0
        assert all(np.all(t == 0) for t in got) and np.all(host(dE) == 0)
        return
    check_against_oracle(og, X, params, y, mask, E, masks, [H1, H2], host(logits), got_loss, got,
                         host(dE))
