"""Per-element error scales for the GraphSAGE training step (host side, test
infrastructure).

Every checked value v of the step is a sum of terms; its scale is the sum of
the magnitudes of those terms, taken one contraction deep from the oracle's
own float64 intermediates, as for a single fp32 aggregation (where the scale
is the oracle's sum of |val * x|). A weight gradient Y^T dO has the terms
Y[r, i] dO[r, j]; dO of a hidden layer is itself the LayerNorm backward of
dY = dO' W_self^T + A^T (dO' W_neigh^T), and its scale T carries the
magnitudes of those terms as well:

  T(dY)  = |dO'| |W_self|^T + A^T (|dO'| |W_neigh|^T)
  T(dO)  = pattern * rstd * (T(dY) + mean T(dY) + |Y| mean(T(dY) |Y|))

(row means over the features), with dO' the upstream gradient of the layer
above, so cancellation in the backward chain widens the scale of what is
built from it. The softmax gradient (p - onehot) / n_rows_in_loss has scale
(p + onehot) / n_rows_in_loss. Forward values (the hidden outputs before
their ReLU and the logits) have the scale |Y| |W_self| + |Z| |W_neigh| + |b|.

A layer whose output is narrower than its input (fo < f, the class layer)
is evaluated by the library as Y W_self + D^-1 A (Y W_neigh) + b: its middle
terms are D^-1[i, s] Y[s, k] W_neigh[k, c], so |Z| = |D^-1 A Y| gives way to
D^-1 A |Y| in the scales of its output and of dW_neigh (= Y^T (D^-1 A)^T dO).
T(dY) is the same either way (magnitudes multiply associatively).

The tests compare each element with |got - want| <= 1e-5 * scale: about 170
units of fp32 roundoff per unit of scale. Both sides use the same ReLU
patterns (the GPU's, after every unit where they differ from float64's has
been shown to lie within 1e-5 of 0 relative to its terms).
"""

import numpy as np

import oracle


def _rowmean(a):
    return a.mean(axis=1, keepdims=True)


def sage_step_scales(graph, params, labels, lp_mask, E, ref):
    """(scales of the 9 gradients, scale of dE or None, scale of the logits,
    scales of the two hidden layers' outputs before the ReLU) for the step
    the oracle ran in `ref` (oracle.sage_step)."""
    agg_t = lambda T: oracle._agg64(graph.csc_ptr, graph.csc_idx, graph.csc_val, T)
    agg = lambda T: oracle._agg64(graph.csr_ptr, graph.csr_idx, graph.csr_val, T)
    P = [np.abs(np.asarray(p, np.float64)) for p in params]
    # |Z| of the layers that aggregate Y, D^-1 A |Y| of those that aggregate Y W_neigh
    zmag = []
    for l in range(3):
        Yl, _, Zl, _ = ref["saved"][l]
        f, fo = np.shape(params[3 * l])
        zmag.append(agg(np.abs(Yl)) if fo < f else np.abs(Zl))
    y = np.asarray(labels)
    n = len(y)
    m = None if lp_mask is None else np.asarray(lp_mask).astype(bool)
    fwd_scales = []
    for l in range(3):
        Yl = ref["saved"][l][0]
        fwd_scales.append(np.abs(Yl) @ P[3 * l] + zmag[l] @ P[3 * l + 1] + P[3 * l + 2])
    logits = ref["logits"]
    mx = logits.max(axis=1, keepdims=True)
    p = np.exp(logits - mx)
    p /= p.sum(axis=1, keepdims=True)
    loss_rows = np.ones(n, bool) if m is None else ~m
    p[np.arange(n), y] += 1.0
    T = p / max(int(loss_rows.sum()), 1)
    T[~loss_rows] = 0.0
    del p
    scales = [None] * 9
    T_dE = None
    for l in (2, 1, 0):
        Yl, rstd, _, _ = ref["saved"][l]
        scales[3 * l] = np.abs(Yl).T @ T
        scales[3 * l + 1] = zmag[l].T @ T
        scales[3 * l + 2] = T.sum(axis=0)
        if l == 0 and m is None:
            break
        dO = np.abs(ref["douts"][l])
        TdY = dO @ P[3 * l].T + agg_t(dO @ P[3 * l + 1].T)
        del dO
        aY = np.abs(Yl)
        T = rstd[:, None] * (TdY + _rowmean(TdY) + aY * _rowmean(TdY * aY))
        del TdY, aY
        if l > 0:
            T *= ref["saved"][l - 1][3]
        else:
            T_dE = np.zeros(np.shape(E), np.float64)
            np.add.at(T_dE, y[m], T[m])
    return scales, T_dE, fwd_scales[2], fwd_scales[:2]


def check_elementwise(got, want, scale, rel=1e-5, what=""):
    """Assert |got - want| <= rel * scale everywhere; returns max err/scale."""
    got = np.asarray(got, np.float64)
    err = np.abs(got - want)
    ratio = err / np.maximum(scale, 1e-300)
    worst = float(ratio.max()) if ratio.size else 0.0
    bad = err > rel * scale + 1e-30
    assert not bad.any(), "%s: %d of %d elements outside %.0e * scale (max err/scale %.3e)" % (
        what, int(bad.sum()), bad.size, rel, worst)
    return worst
