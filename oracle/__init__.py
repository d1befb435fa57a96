"""CPU oracle for the GCN aggregation path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the GPU smoke check and the benchmark's CPU-baseline leg
may import this package. The GPU library neither imports nor links it; the two
share no code (only the seeded input generators in ``synth`` serve both).

Python side of ``oracle.cpp`` (structure, normalization, fp64-accumulated
aggregation, per-row uint8 quantization and fused halo dequantization; see
the header there for the paper passages each function follows) plus the
two-layer GCN training step in float64 numpy.

Paper: SuperGCN (Chen et al., arXiv 2411.16025). Sections cited:
  * 2.1  -- a GCN layer is AGGREGATE over neighbours then UPDATE (e.g. a
            linear transform); GCN is the model family cited there.
  * 2.4  -- integer quantization Z = min, S = (max - min)/(2^b - 1).
  * 4    -- Index_add / SpMM aggregation, clustering and sorting of idx.
  * 6.1  -- quantize, communicate, dequantize the boundary features.
  * 6.3, Lemma 2 -- the layer written as A H W.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

SYMMETRIZE = 1
ADD_SELF_LOOPS = 2


def build(force: bool = True) -> str:
    """Compile liboracle.so with g++ (OpenMP, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["g++", "-O2", "-std=c++17", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
             _SRC, "-o", tmp])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i64, u32 = ctypes.c_int64, ctypes.c_uint32
        lib.orc_structure.argtypes = [i64, i64, i64, P, P, u32, ctypes.c_int, i64, P, P]
        lib.orc_structure.restype = i64
        lib.orc_rows_of.argtypes = [i64, i64, i64, P, P, u32, ctypes.c_int, i64, P, i64, P, P]
        lib.orc_rows_of.restype = i64
        lib.orc_row_degrees.argtypes = [i64, P, P, P]
        lib.orc_normalize.argtypes = [i64, P, P, P, P]
        lib.orc_normalize_listed.argtypes = [i64, P, P, P, P]
        lib.orc_spmm.argtypes = [i64, P, P, P, P, i64, i64, P, P]
        lib.orc_spmm_f64.argtypes = [i64, P, P, P, P, i64, i64, P]
        lib.orc_dequant.argtypes = [ctypes.c_uint8, ctypes.c_float, ctypes.c_float]
        lib.orc_dequant.restype = ctypes.c_float
        lib.orc_dequant_rows.argtypes = [i64, i64, P, i64, P, P, P, i64]
        lib.orc_spmm_q8.argtypes = [i64, P, P, P, i64, P, i64, P, i64, P, P, i64, P, P]
        lib.orc_quantize_rows.argtypes = [i64, i64, P, i64, P, i64, P, P]
        lib.orc_layernorm_rows.argtypes = [i64, i64, P, i64, P, P, ctypes.c_double, P, i64]
        lib.orc_quantize_rows_bits.argtypes = [i64, i64, ctypes.c_int, P, i64, P, i64, P, P, i64]
        lib.orc_dequant_rows_bits.argtypes = [i64, i64, ctypes.c_int, P, i64, P, P, i64, P, i64]
        lib.orc_spmm_qbits.argtypes = [i64, P, P, P, i64, P, i64, ctypes.c_int, P, i64, P, P, i64,
                                       i64, P, P]
        lib.orc_bipartite_cover.argtypes = [i64, i64, i64, P, P, P, P]
        lib.orc_bipartite_cover.restype = i64
        lib.orc_num_threads.restype = ctypes.c_int
        lib.orc_set_num_threads.argtypes = [ctypes.c_int]
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def num_threads() -> int:
    return _L().orc_num_threads()


def set_num_threads(n: int) -> None:
    """Thread count of the oracle's later parallel loops (results do not depend on it)."""
    _L().orc_set_num_threads(int(n))


_ERR = {-1: "capacity", -2: "id out of range", -3: "symmetrize needs a square shape",
        -4: "repeated selection"}


def structure(n_rows, n_cols, src, dst, flags, transpose=False):
    """Sorted, deduplicated (ptr int64, idx int32) of A or (transpose) A^T."""
    src = _c(src, np.int32)
    dst = _c(dst, np.int32)
    cap = len(src) * (2 if flags & SYMMETRIZE else 1) + min(n_rows, n_cols)
    n_major = n_cols if transpose else n_rows
    ptr = np.empty(n_major + 1, np.int64)
    idx = np.empty(max(cap, 1), np.int32)
    nnz = _L().orc_structure(n_rows, n_cols, len(src), _p(src), _p(dst), flags, int(transpose),
                             cap, _p(ptr), _p(idx))
    if nnz < 0:
        raise ValueError("oracle structure: " + _ERR[nnz])
    return ptr, idx[:nnz].copy()


def rows_of(n_rows, n_cols, src, dst, flags, sel, transpose=False):
    """Structure of the listed (distinct) major ids only, from the edge list."""
    src = _c(src, np.int32)
    dst = _c(dst, np.int32)
    sel = _c(sel, np.int32)
    cap = len(src) * (2 if flags & SYMMETRIZE else 1) + len(sel)
    ptr = np.empty(len(sel) + 1, np.int64)
    idx = np.empty(max(cap, 1), np.int32)
    tot = _L().orc_rows_of(n_rows, n_cols, len(src), _p(src), _p(dst), flags, int(transpose),
                           len(sel), _p(sel), cap, _p(ptr), _p(idx))
    if tot < 0:
        raise ValueError("oracle rows_of: " + _ERR[tot])
    return ptr, idx[:tot].copy()


def row_degrees(ptr, idx):
    """Entries per row whose column differs from the row id."""
    ptr = _c(ptr, np.int64)
    idx = _c(idx, np.int32)
    deg = np.empty(len(ptr) - 1, np.int32)
    _L().orc_row_degrees(len(ptr) - 1, _p(ptr), _p(idx), _p(deg))
    return deg


def normalize(ptr, idx, deg):
    """val[k] = fp32(1 / sqrt((deg[r]+1)(deg[c]+1))) for entry k = (r, c)."""
    ptr = _c(ptr, np.int64)
    idx = _c(idx, np.int32)
    deg = _c(deg, np.int32)
    n_major = len(ptr) - 1
    if len(idx) and (len(deg) < n_major or int(idx.max()) >= len(deg)):
        raise ValueError("deg must cover every row and column id")
    val = np.empty(len(idx), np.float32)
    _L().orc_normalize(len(ptr) - 1, _p(ptr), _p(idx), _p(deg), _p(val))
    return val


def normalize_listed(ptr, deg_rows, deg_cols):
    ptr = _c(ptr, np.int64)
    deg_rows = _c(deg_rows, np.int32)
    deg_cols = _c(deg_cols, np.int32)
    val = np.empty(len(deg_cols), np.float32)
    _L().orc_normalize_listed(len(ptr) - 1, _p(ptr), _p(deg_rows), _p(deg_cols), _p(val))
    return val


def spmm(ptr, idx, val, X):
    """(Y, S): Y = A X accumulated in float64, S = sum of |terms| per element."""
    ptr = _c(ptr, np.int64)
    idx = _c(idx, np.int32)
    val = _c(val, np.float32)
    X = np.asarray(X, np.float32)
    if X.strides[1] != 4:
        X = np.ascontiguousarray(X)
    assert X.ndim == 2
    F = X.shape[1]
    ldx = X.strides[0] // 4
    n = len(ptr) - 1
    Y = np.empty((n, F), np.float64)
    S = np.empty((n, F), np.float64)
    _L().orc_spmm(n, _p(ptr), _p(idx), _p(val), X.ctypes.data, ldx, F, _p(Y), _p(S))
    return Y, S


def dequant(q, scale, zero) -> np.float32:
    return np.float32(_L().orc_dequant(int(q), float(scale), float(zero)))


def dequant_rows(Q, zmin, scale):
    Q = _c(Q, np.uint8)
    n, F = Q.shape
    out = np.empty((n, F), np.float32)
    _L().orc_dequant_rows(n, F, _p(Q), F, _p(_c(zmin, np.float32)), _p(_c(scale, np.float32)),
                          _p(out), F)
    return out


def spmm_q8(ptr, idx, val, n_local_cols, X_local, Q, zmin, scale):
    """(Y, S) with columns >= n_local_cols dequantized from uint8 codes."""
    ptr = _c(ptr, np.int64)
    idx = _c(idx, np.int32)
    val = _c(val, np.float32)
    X_local = np.asarray(X_local, np.float32)
    Q = np.asarray(Q, np.uint8)
    if X_local.strides[1] != 4:
        X_local = np.ascontiguousarray(X_local)
    if Q.strides[1] != 1:
        Q = np.ascontiguousarray(Q)
    F = X_local.shape[1]
    assert Q.shape[1] == F
    n = len(ptr) - 1
    Y = np.empty((n, F), np.float64)
    S = np.empty((n, F), np.float64)
    zmin = _c(zmin, np.float32)
    scale = _c(scale, np.float32)
    _L().orc_spmm_q8(n, _p(ptr), _p(idx), _p(val), n_local_cols, X_local.ctypes.data,
                     X_local.strides[0] // 4, Q.ctypes.data, Q.strides[0], _p(zmin), _p(scale),
                     F, _p(Y), _p(S))
    return Y, S


def quantize_rows(X):
    """Per-row uint8 codes and (zmin, scale), round-to-nearest-even."""
    X = np.asarray(X, np.float32)
    if X.strides[1] != 4:
        X = np.ascontiguousarray(X)
    n, F = X.shape
    Q = np.empty((n, F), np.uint8)
    zmin = np.empty(n, np.float32)
    scale = np.empty(n, np.float32)
    _L().orc_quantize_rows(n, F, X.ctypes.data, X.strides[0] // 4, _p(Q), F, _p(zmin), _p(scale))
    return Q, zmin, scale


def layernorm_rows(X, gamma=None, beta=None, eps=1e-5):
    """Row LayerNorm in double, rounded once to fp32 (biased variance)."""
    X = np.ascontiguousarray(X, np.float32)
    n, F = X.shape
    Y = np.empty((n, F), np.float32)
    g = None if gamma is None else _c(gamma, np.float32)
    b = None if beta is None else _c(beta, np.float32)
    _L().orc_layernorm_rows(n, F, _p(X), F, _p(g), _p(b), float(eps), _p(Y), F)
    return Y


def code_bytes(F, bits):
    return F if bits == 8 else (F + 3) // 4


def quantize_rows_bits(X, bits):
    """(Q, zmin, scale) with b-bit codes; 2-bit codes packed 4 per byte."""
    X = np.ascontiguousarray(X, np.float32)
    n, F = X.shape
    Q = np.zeros((n, code_bytes(F, bits)), np.uint8)
    zmin = np.empty(n, np.float32)
    scale = np.empty(n, np.float32)
    _L().orc_quantize_rows_bits(n, F, bits, _p(X), F, _p(Q), Q.shape[1], _p(zmin), _p(scale), 1)
    return Q, zmin, scale


def dequant_rows_bits(Q, zmin, scale, F, bits):
    Q = _c(Q, np.uint8)
    n = Q.shape[0]
    out = np.empty((n, F), np.float32)
    _L().orc_dequant_rows_bits(n, F, bits, _p(Q), Q.shape[1], _p(_c(zmin, np.float32)),
                               _p(_c(scale, np.float32)), 1, _p(out), F)
    return out


def spmm_qbits(ptr, idx, val, n_local_cols, X_local, Q, zmin, scale, F, bits):
    """(Y, S) with halo columns holding b-bit codes."""
    ptr = _c(ptr, np.int64)
    idx = _c(idx, np.int32)
    val = _c(val, np.float32)
    X_local = np.ascontiguousarray(X_local, np.float32)
    Q = _c(Q, np.uint8)
    n = len(ptr) - 1
    Y = np.empty((n, F), np.float64)
    S = np.empty((n, F), np.float64)
    _L().orc_spmm_qbits(n, _p(ptr), _p(idx), _p(val), n_local_cols, _p(X_local),
                        X_local.shape[1] if X_local.ndim == 2 else F, bits, _p(Q), Q.shape[1],
                        _p(_c(zmin, np.float32)), _p(_c(scale, np.float32)), 1, F, _p(Y), _p(S))
    return Y, S


def bipartite_cover(eu, ev, n_u=None, n_v=None):
    """(matching size, cover_u bool[n_u], cover_v bool[n_v]) of a bipartite graph."""
    eu = _c(eu, np.int32)
    ev = _c(ev, np.int32)
    n_u = int(eu.max()) + 1 if n_u is None else n_u
    n_v = int(ev.max()) + 1 if n_v is None else n_v
    cu = np.zeros(max(n_u, 1), np.uint8)
    cv = np.zeros(max(n_v, 1), np.uint8)
    m = _L().orc_bipartite_cover(n_u, n_v, len(eu), _p(eu), _p(ev), _p(cu), _p(cv))
    return int(m), cu[:n_u].astype(bool), cv[:n_v].astype(bool)


def prepost_split(src, dst):
    """Algorithm 1 of Section 5.2 on a remote edge list (src on the sending
    worker, dst on the receiving one): the two endpoint sets are the sides of
    a bipartite graph, a minimum vertex cover is found, and an edge is a post-
    aggregation edge when its source is in the cover, else a pre-aggregation
    edge. Returns (is_post bool[n_edges], volume = |cover|, cover sources,
    cover destinations)."""
    src = np.asarray(src)
    dst = np.asarray(dst)
    us, eu = np.unique(src, return_inverse=True)
    vs, ev = np.unique(dst, return_inverse=True)
    m, cu, cv = bipartite_cover(eu.astype(np.int32), ev.astype(np.int32), len(us), len(vs))
    is_post = cu[eu]
    return is_post, m, us[cu], vs[cv]


# ---------------------------------------------------------------------------
# Whole-graph and sampled-row helpers.
# ---------------------------------------------------------------------------

class Graph:
    """Oracle matrices of one workload: CSR (rows = dst) and CSC, both with
    normalized values unless normalized=False (then every value is 1)."""

    def __init__(self, n_rows, n_cols, src, dst, flags, deg=None, normalized=True, mean=False):
        self.n_rows, self.n_cols = n_rows, n_cols
        self.csr_ptr, self.csr_idx = structure(n_rows, n_cols, src, dst, flags, False)
        self.csc_ptr, self.csc_idx = structure(n_rows, n_cols, src, dst, flags, True)
        if mean:
            self.deg = None
            self.csr_val, self.csc_val = mean_values(self.csr_ptr, self.csr_idx, self.csc_idx)
            return
        if deg is None:
            if n_rows != n_cols:
                raise ValueError("a rectangular graph needs a supplied degree array")
            deg = row_degrees(self.csr_ptr, self.csr_idx)
        self.deg = np.asarray(deg, np.int32)
        if len(self.deg) < max(n_rows, n_cols):
            raise ValueError("deg must cover every node id: max(n_rows, n_cols) entries")
        if normalized:
            self.csr_val = normalize(self.csr_ptr, self.csr_idx, self.deg)
            self.csc_val = normalize(self.csc_ptr, self.csc_idx, self.deg)
        else:
            self.csr_val = np.ones(len(self.csr_idx), np.float32)
            self.csc_val = np.ones(len(self.csc_idx), np.float32)

    @property
    def nnz(self):
        return len(self.csr_idx)

    def fwd(self, X):
        return spmm(self.csr_ptr, self.csr_idx, self.csr_val, X)

    def bwd(self, G):
        return spmm(self.csc_ptr, self.csc_idx, self.csc_val, G)


def mean_values(csr_ptr, csr_idx, csc_idx):
    """Values of the mean operator D^-1 A (GraphSAGE's mean AGGREGATE, Section
    2.1): entry (r, c) of A is 1 / (number of stored entries of row r), computed
    in double and rounded once to fp32; an empty row has no entries. Returns
    the values for A's CSR and for its transpose (whose entry (c, r) carries
    the value of row r of A)."""
    lens = np.diff(np.asarray(csr_ptr, np.int64)).astype(np.float64)
    rows = np.repeat(np.arange(len(lens)), np.diff(csr_ptr))
    csr_val = (1.0 / lens[rows]).astype(np.float32)
    csc_val = (1.0 / lens[np.asarray(csc_idx, np.int64)]).astype(np.float32)
    return csr_val, csc_val


def sampled(n_rows, n_cols, src, dst, flags, sel, transpose=False, deg=None):
    """(ptr, idx, val) of the listed rows of A (or A^T), normalized.

    deg: the supplied per-node degree array, or None to use the stored
    non-self entry count of each node's row of A (square graphs)."""
    sel = np.asarray(sel, np.int32)
    ptr, idx = rows_of(n_rows, n_cols, src, dst, flags, sel, transpose)
    if deg is not None:
        deg = np.asarray(deg, np.int32)
        deg_rows, deg_cols = deg[sel], deg[idx]
    else:
        nodes = np.unique(np.concatenate([sel, idx]))
        nptr, nidx = rows_of(n_rows, n_cols, src, dst, flags, nodes, False)
        owner = np.repeat(nodes, np.diff(nptr))
        nd = np.bincount(np.searchsorted(nodes, owner[nidx != owner]),
                         minlength=len(nodes)).astype(np.int32)
        deg_rows = nd[np.searchsorted(nodes, sel)]
        deg_cols = nd[np.searchsorted(nodes, idx)]
    val = normalize_listed(ptr, deg_rows, deg_cols)
    return ptr, idx, val


# ---------------------------------------------------------------------------
# Two-layer GCN training step (float64), Section 2.1: each layer aggregates
# then applies a linear transform; the order A (X W) keeps the aggregation on
# the narrower side. No bias, no dropout, no LayerNorm; ReLU between layers;
# mean negative log-likelihood of log-softmax over all nodes.
# ---------------------------------------------------------------------------

def _agg64(ptr, idx, val, H):
    """A H in float64 for float64 H (row order, double accumulation)."""
    H = np.ascontiguousarray(H, np.float64)
    ptr = _c(ptr, np.int64)
    idx = _c(idx, np.int32)
    val = _c(val, np.float32)
    n = len(ptr) - 1
    out = np.empty((n, H.shape[1]), np.float64)
    _L().orc_spmm_f64(n, _p(ptr), _p(idx), _p(val), H.ctypes.data, H.shape[1], H.shape[1],
                      _p(out))
    return out


def gcn_step(graph: Graph, X, W1, W2, labels):
    """Loss and weight gradients of the 2-layer GCN, all in float64.

    Returns dict(loss, dW1, dW2) and the intermediates Z1, A1, H1, Z2, logits,
    dlogits, dZ2, dH1 (before the ReLU mask), dZ1."""
    X = np.asarray(X, np.float64)
    W1 = np.asarray(W1, np.float64)
    W2 = np.asarray(W2, np.float64)
    y = np.asarray(labels)
    n = X.shape[0]
    fwd = lambda H: _agg64(graph.csr_ptr, graph.csr_idx, graph.csr_val, H)
    bwd = lambda H: _agg64(graph.csc_ptr, graph.csc_idx, graph.csc_val, H)
    Z1 = X @ W1
    A1 = fwd(Z1)
    H1 = np.maximum(A1, 0.0)
    Z2 = H1 @ W2
    logits = fwd(Z2)
    m = logits.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(logits - m).sum(axis=1))
    loss = float(np.mean(lse - logits[np.arange(n), y]))
    dlogits = np.exp(logits - lse[:, None])
    dlogits[np.arange(n), y] -= 1.0
    dlogits /= n
    dZ2 = bwd(dlogits)
    dW2 = H1.T @ dZ2
    dH1 = dZ2 @ W2.T
    dA1 = dH1 * (A1 > 0)
    dZ1 = bwd(dA1)
    dW1 = X.T @ dZ1
    return dict(loss=loss, dW1=dW1, dW2=dW2, Z1=Z1, A1=A1, H1=H1, Z2=Z2, logits=logits,
                dlogits=dlogits, dZ2=dZ2, dH1=dH1, dZ1=dZ1)


# ---------------------------------------------------------------------------
# 3-layer GraphSAGE training step with LayerNorm before each layer (the model
# of the evaluation, Table 2) and masked label propagation (Section 6.1 step 1,
# Lemma 2), all in float64.
# ---------------------------------------------------------------------------

def layernorm64(H, eps):
    """Row LayerNorm without affine parameters: (y, 1/sqrt(var + eps)) with the
    biased variance, in float64."""
    mu = H.mean(axis=1, keepdims=True)
    var = ((H - mu) ** 2).mean(axis=1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    return (H - mu) * rstd, rstd[:, 0]


def layernorm64_bwd(Y, rstd, dY):
    """Gradient of the row LayerNorm: rstd * (dY - mean(dY) - Y * mean(dY * Y))."""
    return rstd[:, None] * (dY - dY.mean(axis=1, keepdims=True)
                            - Y * (dY * Y).mean(axis=1, keepdims=True))


def sage_step(graph: Graph, X, params, labels, lp_mask=None, E=None, eps=1e-5, masks=None):
    """Loss and gradients of one step of the 3-layer GraphSAGE-mean model.

    graph: mean-normalized (Graph(..., mean=True)); params: the list
    [W_self1, W_neigh1, b1, W_self2, W_neigh2, b2, W_self3, W_neigh3, b3]
    (W [f_in x f_out], b [f_out]). Layer l: Y = LayerNorm(H), Z = D^-1 A Y,
    O = Y W_self + Z W_neigh + b, H = relu(O) after layers 1 and 2; the last O
    are the logits. Masked label propagation: rows with lp_mask = 1 get the
    embedding E[label] added to their input features and are left out of the
    loss; the loss is the mean softmax cross-entropy over the other rows (all
    rows without lp_mask). masks (optional): the ReLU patterns of layers 1 and
    2 to use in place of O > 0 (a unit whose pre-activation lies within
    rounding of 0 may fall either way in another precision). Returns
    dict(loss, grads (same order as params), dE or None, logits, acts: the
    float64 patterns O > 0 of the hidden layers, flip_margins: per hidden
    layer, |O| / (sum of the magnitudes of its terms) at every unit where the
    given mask differs from O > 0 (empty without masks), saved: per layer
    (Y, rstd, Z, pattern used), douts: per layer the gradient of the loss
    with respect to its output O)."""
    H = np.asarray(X, np.float64).copy()
    y = np.asarray(labels)
    n = H.shape[0]
    P = [np.asarray(p, np.float64) for p in params]
    if lp_mask is not None:
        m = np.asarray(lp_mask).astype(bool)
        H[m] += np.asarray(E, np.float64)[y[m]]
        loss_rows = ~m
    else:
        m = None
        loss_rows = np.ones(n, bool)
    fwd = lambda T: _agg64(graph.csr_ptr, graph.csr_idx, graph.csr_val, T)
    bwd = lambda T: _agg64(graph.csc_ptr, graph.csc_idx, graph.csc_val, T)
    saved = []
    flip_margins, acts = [], []
    for l in range(3):
        Ws, Wn, b = P[3 * l], P[3 * l + 1], P[3 * l + 2]
        Yl, rstd = layernorm64(H, eps)
        Zl = fwd(Yl)
        O = Yl @ Ws + Zl @ Wn + b
        if l < 2:
            own = O > 0
            act = own if masks is None else np.asarray(masks[l], bool)
            flip = act != own
            rows = np.flatnonzero(flip.any(axis=1))
            mag = (np.abs(Yl[rows]) @ np.abs(Ws) + np.abs(Zl[rows]) @ np.abs(Wn) + np.abs(b))
            flip_margins.append((np.abs(O[rows]) / mag)[flip[rows]])
            acts.append(own)
            H = O * act
        else:
            act = None
            H = O
        saved.append((Yl, rstd, Zl, act))
    logits = H
    mx = logits.max(axis=1, keepdims=True)
    lse = mx[:, 0] + np.log(np.exp(logits - mx).sum(axis=1))
    n_loss = int(loss_rows.sum())
    idx = np.flatnonzero(loss_rows)
    # no row in the loss (every label embedded): loss 0 and no gradient
    loss = float(np.sum(lse[idx] - logits[idx, y[idx]]) / n_loss) if n_loss else 0.0
    dO = np.exp(logits - lse[:, None])
    dO[idx, y[idx]] -= 1.0
    dO[~loss_rows] = 0.0
    dO /= max(n_loss, 1)
    grads = [None] * 9
    dE = None
    douts = [None] * 3
    for l in (2, 1, 0):
        Yl, rstd, Zl, _ = saved[l]
        douts[l] = dO
        grads[3 * l] = Yl.T @ dO
        grads[3 * l + 1] = Zl.T @ dO
        grads[3 * l + 2] = dO.sum(axis=0)
        if l == 0 and m is None:
            break
        dY = dO @ P[3 * l].T + bwd(dO @ P[3 * l + 1].T)
        dH = layernorm64_bwd(Yl, rstd, dY)
        if l > 0:
            dO = dH * saved[l - 1][3]
        else:
            dE = np.zeros_like(np.asarray(E, np.float64))
            np.add.at(dE, y[m], dH[m])
    return dict(loss=loss, grads=grads, dE=dE, logits=logits, acts=acts,
                flip_margins=flip_margins, saved=saved, douts=douts)

