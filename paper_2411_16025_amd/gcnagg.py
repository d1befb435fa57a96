"""Python binding of libgcnagg.so (argument marshalling only).

Every function has the name of the C entry point it wraps (include/gcnagg.h)
and passes device pointers of torch tensors plus the current torch stream.
All computation runs in the library's HIP kernels; there is no fallback: if
the library is missing or the call fails, an exception is raised.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgcnagg.so")

GCN_SYMMETRIZE = 1
GCN_ADD_SELF_LOOPS = 2
GCN_DT_F32 = 0
GCN_DT_BF16 = 1
GCN_Q8_USE_CSC = 1
GCN_Q_CODES_2BIT = 2
GCN_LAYERNORM = 1

STATUS = {0: "GCN_OK", 1: "GCN_EINVAL", 2: "GCN_ERANGE", 3: "GCN_ENOMEM", 4: "GCN_EHIP",
          5: "GCN_ESTATE"}

# every symbol include/gcnagg.h declares
GCN_GEMM_NN, GCN_GEMM_NT, GCN_GEMM_TN = 0, 1, 2

EXPORTS = ("gcn_build_csr", "gcn_normalize", "gcn_normalize_rc", "gcn_normalize_mean",
           "gcn_layernorm_fwd", "gcn_layernorm_bwd", "gcn_sage3_forward", "gcn_sage3_step",
           "gcn_prepost_split",
           "gcn_add_rows", "gcn_add_rows_q", "gcn_aggregate_fwd", "gcn_aggregate_bwd", "gcn_aggregate_fwd_noalloc",
           "gcn_aggregate_fwd_q8halo", "gcn_quantize_rows_u8", "gcn_layernorm_quantize",
           "gcn_gemm_f32", "gcn_relu",
           "gcn_relu_bwd", "gcn_softmax_xent", "gcn_gcn2_step", "gcn_graph_free",
           "gcn_graph_info", "gcn_graph_export", "gcn_graph_bins", "gcn_profile_enable",
           "gcn_profile_read", "gcn_last_error")


class GcnError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (STATUS.get(status, str(status)), message))
        self.status = status
        self.message = message


_lib = None


def lib():
    """Load libgcnagg.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libgcnagg.so is not built (%s); run "
                               "paper_2411_16025_amd.build.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, i64, u32, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32, ctypes.c_int
        L.gcn_build_csr.argtypes = [i64, i64, i64, P, P, u32, P, ctypes.POINTER(P)]
        L.gcn_normalize.argtypes = [P, P, P]
        L.gcn_normalize_rc.argtypes = [P, P, P, P]
        L.gcn_prepost_split.argtypes = [i64, i64, i64, P, P, P, P, P, P]
        L.gcn_add_rows.argtypes = [i64, i64, P, i64, P, i64, P, i64, P]
        L.gcn_add_rows_q.argtypes = [i64, i64, i32, P, i64, P, P, i64, P, i64, P, i64, P]
        L.gcn_aggregate_fwd.argtypes = [P, P, i64, i32, P, i64, i64, P]
        L.gcn_aggregate_bwd.argtypes = [P, P, i64, i32, P, i64, i64, P]
        L.gcn_aggregate_fwd_noalloc.argtypes = [P, P, i64, i32, P, i64, i64, P]
        L.gcn_aggregate_fwd_q8halo.argtypes = [P, i64, P, i64, P, i64, P, P, i64, P, i64, i64, u32,
                                               P]
        L.gcn_quantize_rows_u8.argtypes = [i64, i64, P, i64, P, i64, P, P, i64, P]
        L.gcn_layernorm_quantize.argtypes = [i64, i64, P, i64, P, P, ctypes.c_double, u32, i32, P,
                                             i64, P, i64, P, P, i64, P]
        L.gcn_gemm_f32.argtypes = [i32, i64, i64, i64, P, i64, P, i64, P, i64, P]
        L.gcn_relu.argtypes = [i64, i64, P, i64, P]
        L.gcn_relu_bwd.argtypes = [i64, i64, P, i64, P, i64, P]
        L.gcn_softmax_xent.argtypes = [i64, i64, P, i64, P, P, i64, P, P]
        L.gcn_gcn2_step.argtypes = [P, P, i64, i64, P, i64, P, i64, P, P, P, P, P]
        L.gcn_normalize_mean.argtypes = [P, P]
        L.gcn_layernorm_fwd.argtypes = [i64, i64, P, i64, ctypes.c_double, P, i64, P, P]
        L.gcn_layernorm_bwd.argtypes = [i64, i64, P, i64, P, P, i64, P, i64, P, i64, P, i64, P]
        L.gcn_sage3_step.argtypes = [P, P, i64, i64, i64, i64, P, P, P, P, ctypes.c_double, P,
                                     P, P, P]
        L.gcn_sage3_forward.argtypes = [P, P, i64, i64, i64, i64, P, P, P, P, ctypes.c_double, P,
                                        i64, P, i64, P, i64, P]
        L.gcn_graph_free.argtypes = [P]
        L.gcn_graph_free.restype = None
        L.gcn_graph_info.argtypes = [P, P, P, P]
        L.gcn_graph_export.argtypes = [P, i32, P, P, P, P]
        L.gcn_graph_bins.argtypes = [P, i32, i64, P, i32, P, P]
        L.gcn_profile_enable.argtypes = [i32]
        L.gcn_profile_read.argtypes = [P, P, P, i32, P]
        L.gcn_last_error.argtypes = []
        L.gcn_last_error.restype = ctypes.c_char_p
        for name in EXPORTS:
            if name not in ("gcn_graph_free", "gcn_last_error"):
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise GcnError(status, lib().gcn_last_error().decode())


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _dev(t, dtype=None, name="tensor"):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a CUDA (HIP) torch tensor" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must have dtype %s (got %s)" % (name, dtype, t.dtype))
    return t


def _rowmajor(t, name):
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("%s must be a 2-D row-major tensor (unit column stride)" % name)
    return t.stride(0)


class Graph:
    """Owner of a gcn_graph handle."""

    def __init__(self, handle: int):
        self._h = ctypes.c_void_p(handle)
        self.n_rows, self.n_cols, self.nnz = gcn_graph_info(self)

    @property
    def handle(self):
        if not self._h:
            raise GcnError(5, "graph already freed")
        return self._h

    def free(self):
        if self._h:
            lib().gcn_graph_free(self._h)
            self._h = ctypes.c_void_p(0)

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def gcn_build_csr(n_rows: int, n_cols: int, src: torch.Tensor, dst: torch.Tensor, flags: int,
                  stream=None) -> Graph:
    _dev(src, torch.int32, "src")
    _dev(dst, torch.int32, "dst")
    if src.numel() != dst.numel() or not src.is_contiguous() or not dst.is_contiguous():
        raise ValueError("src and dst must be contiguous and of equal length")
    out = ctypes.c_void_p(0)
    _check(lib().gcn_build_csr(n_rows, n_cols, src.numel(), src.data_ptr(), dst.data_ptr(), flags,
                               _stream(stream), ctypes.byref(out)))
    return Graph(out.value)


def gcn_normalize(g: Graph, deg: torch.Tensor | None = None, stream=None):
    if deg is not None:
        _dev(deg, torch.int32, "deg")
        if not deg.is_contiguous() or deg.numel() != max(g.n_rows, g.n_cols):
            raise ValueError("deg must be contiguous with max(n_rows, n_cols) entries")
    _check(lib().gcn_normalize(g.handle, deg.data_ptr() if deg is not None else None,
                               _stream(stream)))


def gcn_normalize_rc(g: Graph, deg_rows: torch.Tensor, deg_cols: torch.Tensor, stream=None):
    """Normalize with row degrees [n_rows] and column degrees [n_cols]."""
    for t, n, name in ((deg_rows, g.n_rows, "deg_rows"), (deg_cols, g.n_cols, "deg_cols")):
        _dev(t, torch.int32, name)
        if not t.is_contiguous() or t.numel() != n:
            raise ValueError("%s must be contiguous with %d entries" % (name, n))
    _check(lib().gcn_normalize_rc(g.handle, deg_rows.data_ptr(), deg_cols.data_ptr(),
                                  _stream(stream)))


def gcn_prepost_split(src, dst, n_src: int | None = None, n_dst: int | None = None):
    """Algorithm 1 on host int32 edge arrays: (is_post bool[n_edges],
    src_slot int32[n_src], dst_slot int32[n_dst], volume)."""
    src = np.ascontiguousarray(src, dtype=np.int32)
    dst = np.ascontiguousarray(dst, dtype=np.int32)
    if src.shape != dst.shape or src.ndim != 1:
        raise ValueError("src and dst must be 1-D arrays of one length")
    n_src = int(src.max()) + 1 if n_src is None else int(n_src)
    n_dst = int(dst.max()) + 1 if n_dst is None else int(n_dst)
    is_post = np.zeros(len(src), np.uint8)
    src_slot = np.zeros(max(n_src, 0), np.int32)
    dst_slot = np.zeros(max(n_dst, 0), np.int32)
    vol = ctypes.c_int64(0)
    ptr = lambda a: a.ctypes.data if a.size else None  # noqa: E731
    _check(lib().gcn_prepost_split(n_src, n_dst, len(src), ptr(src), ptr(dst), ptr(is_post),
                                   ptr(src_slot), ptr(dst_slot), ctypes.byref(vol)))
    return is_post.astype(bool), src_slot, dst_slot, int(vol.value)


def gcn_add_rows(P: torch.Tensor, idx: torch.Tensor, Y: torch.Tensor, stream=None):
    """Y[idx[j]] += P[j] in place (distinct idx)."""
    _dev(P, torch.float32, "P")
    _dev(Y, torch.float32, "Y")
    _dev(idx, torch.int32, "idx")
    if P.dim() != 2 or Y.dim() != 2 or P.shape[1] != Y.shape[1] or idx.numel() != P.shape[0]:
        raise ValueError("need P [n x F], idx [n], Y [m x F]")
    if not idx.is_contiguous():
        raise ValueError("idx must be contiguous")
    _check(lib().gcn_add_rows(P.shape[0], P.shape[1], P.data_ptr(), _rowmajor(P, "P"),
                              idx.data_ptr(), Y.shape[0], Y.data_ptr(), _rowmajor(Y, "Y"),
                              _stream(stream)))
    return Y


def gcn_add_rows_q(Q: torch.Tensor, zmin: torch.Tensor, scale: torch.Tensor, idx: torch.Tensor,
                   Y: torch.Tensor, bits: int = 8, F: int | None = None, stream=None):
    """Y[idx[j], f] += fmaf(q[j, f], scale[j], zmin[j]) in place (distinct idx);
    zmin / scale are 1-D with a common stride (the columns of an [n, 2] tensor
    give the paired layout)."""
    _dev(Q, torch.uint8, "Q")
    _dev(Y, torch.float32, "Y")
    _dev(idx, torch.int32, "idx")
    F = Y.shape[1] if F is None else F
    n = Q.shape[0]
    if Q.dim() != 2 or Y.dim() != 2 or Y.shape[1] != F or idx.numel() != n:
        raise ValueError("need Q [n x code bytes], idx [n], Y [m x F]")
    if not idx.is_contiguous():
        raise ValueError("idx must be contiguous")
    for t, nm in ((zmin, "zmin"), (scale, "scale")):
        _dev(t, torch.float32, nm)
        if t.dim() != 1 or t.numel() < n:
            raise ValueError("%s must be 1-D with at least %d entries" % (nm, n))
    ldp = zmin.stride(0)
    if scale.stride(0) != ldp or ldp < 1:
        raise ValueError("zmin and scale need the same positive stride")
    _check(lib().gcn_add_rows_q(n, F, bits, Q.data_ptr(), _rowmajor(Q, "Q"), zmin.data_ptr(),
                                scale.data_ptr(), ldp, idx.data_ptr(), Y.shape[0], Y.data_ptr(),
                                _rowmajor(Y, "Y"), _stream(stream)))
    return Y


def _dtype_code(t):
    if t.dtype == torch.float32:
        return GCN_DT_F32
    if t.dtype == torch.bfloat16:
        return GCN_DT_BF16
    raise TypeError("input must be float32 or bfloat16")


def gcn_aggregate_fwd(g: Graph, X: torch.Tensor, Y: torch.Tensor | None = None, stream=None):
    """Y = A_hat X (allocates Y if not given)."""
    _dev(X, None, "X")
    ldx = _rowmajor(X, "X")
    if X.shape[0] != g.n_cols:
        raise ValueError("X must have n_cols = %d rows" % g.n_cols)
    F = X.shape[1]
    if Y is None:
        Y = torch.empty((g.n_rows, F), dtype=torch.float32, device=X.device)
    _dev(Y, torch.float32, "Y")
    ldy = _rowmajor(Y, "Y")
    if tuple(Y.shape) != (g.n_rows, F):
        raise ValueError("Y must be n_rows x F")
    _check(lib().gcn_aggregate_fwd(g.handle, X.data_ptr(), ldx, _dtype_code(X), Y.data_ptr(), ldy,
                                   F, _stream(stream)))
    return Y


def gcn_aggregate_fwd_noalloc(g: Graph, X: torch.Tensor, Y: torch.Tensor, stream=None):
    """Y = A_hat X with the library's fixed partial-row array instead of an
    allocation (Y must be given; see include/gcnagg.h for the size limit)."""
    _dev(X, None, "X")
    ldx = _rowmajor(X, "X")
    if X.shape[0] != g.n_cols:
        raise ValueError("X must have n_cols = %d rows" % g.n_cols)
    F = X.shape[1]
    _dev(Y, torch.float32, "Y")
    ldy = _rowmajor(Y, "Y")
    if tuple(Y.shape) != (g.n_rows, F):
        raise ValueError("Y must be n_rows x F")
    _check(lib().gcn_aggregate_fwd_noalloc(g.handle, X.data_ptr(), ldx, _dtype_code(X),
                                           Y.data_ptr(), ldy, F, _stream(stream)))
    return Y


def gcn_aggregate_bwd(g: Graph, G: torch.Tensor, dX: torch.Tensor | None = None, stream=None):
    """dX = A_hat^T G (allocates dX if not given)."""
    _dev(G, None, "G")
    ldg = _rowmajor(G, "G")
    if G.shape[0] != g.n_rows:
        raise ValueError("G must have n_rows = %d rows" % g.n_rows)
    F = G.shape[1]
    if dX is None:
        dX = torch.empty((g.n_cols, F), dtype=torch.float32, device=G.device)
    _dev(dX, torch.float32, "dX")
    lddx = _rowmajor(dX, "dX")
    if tuple(dX.shape) != (g.n_cols, F):
        raise ValueError("dX must be n_cols x F")
    _check(lib().gcn_aggregate_bwd(g.handle, G.data_ptr(), ldg, _dtype_code(G), dX.data_ptr(),
                                   lddx, F, _stream(stream)))
    return dX


def gcn_aggregate_fwd_q8halo(g: Graph, n_local_cols: int, X_local, Q_halo, halo_min, halo_scale,
                             Y: torch.Tensor | None = None, use_csc: bool = False, F=None,
                             bits: int = 8, stream=None):
    """Y = A_hat [X_local; fmaf(Q, S, Z)] (or A_hat^T with use_csc).

    halo_min / halo_scale are 1-D tensors with a common stride ldp; the
    columns of an [n_halo, 2] tensor give the paired (Z, S) layout."""
    n_in, n_out = (g.n_rows, g.n_cols) if use_csc else (g.n_cols, g.n_rows)
    ldx = ldq = 0
    ldp = 1
    if X_local is not None:
        _dev(X_local, torch.float32, "X_local")
        ldx = _rowmajor(X_local, "X_local")
        F = X_local.shape[1] if F is None else F
        if X_local.shape[0] < n_local_cols:
            raise ValueError("X_local has fewer than n_local_cols rows")
    if Q_halo is not None:
        _dev(Q_halo, torch.uint8, "Q_halo")
        ldq = _rowmajor(Q_halo, "Q_halo")
        if F is None and bits == 2:
            raise ValueError("F must be given for 2-bit codes without X_local")
        F = Q_halo.shape[1] if F is None else F
        n_h = n_in - n_local_cols
        if Q_halo.shape[0] < n_h:
            raise ValueError("Q_halo has fewer than %d rows" % n_h)
        for t, nm in ((halo_min, "halo_min"), (halo_scale, "halo_scale")):
            _dev(t, torch.float32, nm)
            if t.dim() != 1 or t.numel() < n_h:
                raise ValueError("%s must be 1-D with at least %d entries" % (nm, n_h))
        ldp = halo_min.stride(0)
        if halo_scale.stride(0) != ldp or ldp < 1:
            raise ValueError("halo_min and halo_scale need the same positive stride")
    if F is None:
        raise ValueError("F is unknown")
    if Y is None:
        dev = (X_local if X_local is not None else Q_halo).device
        Y = torch.empty((n_out, F), dtype=torch.float32, device=dev)
    _dev(Y, torch.float32, "Y")
    ldy = _rowmajor(Y, "Y")
    if tuple(Y.shape) != (n_out, F):
        raise ValueError("Y must be %d x %d" % (n_out, F))
    ptr = lambda t: t.data_ptr() if t is not None else None
    _check(lib().gcn_aggregate_fwd_q8halo(
        g.handle, n_local_cols, ptr(X_local), ldx, ptr(Q_halo), ldq, ptr(halo_min),
        ptr(halo_scale), ldp, Y.data_ptr(), ldy, F,
        (GCN_Q8_USE_CSC if use_csc else 0) | (GCN_Q_CODES_2BIT if bits == 2 else 0),
        _stream(stream)))
    return Y


def gcn_quantize_rows_u8(X: torch.Tensor, Q=None, zmin=None, scale=None, paired=False,
                         stream=None):
    """Per-row uint8 codes and (zmin, scale) of an fp32 matrix.

    paired=True stores (Z, S) side by side in an [n, 2] tensor and returns
    its two columns (stride 2)."""
    _dev(X, torch.float32, "X")
    ldx = _rowmajor(X, "X")
    n, F = X.shape
    if Q is None:
        Q = torch.empty((n, F), dtype=torch.uint8, device=X.device)
    if zmin is None and scale is None and paired:
        zs = torch.empty((n, 2), dtype=torch.float32, device=X.device)
        zmin, scale = zs[:, 0], zs[:, 1]
    if zmin is None:
        zmin = torch.empty(n, dtype=torch.float32, device=X.device)
    if scale is None:
        scale = torch.empty(n, dtype=torch.float32, device=X.device)
    ldp = zmin.stride(0)
    if scale.stride(0) != ldp:
        raise ValueError("zmin and scale need the same stride")
    ldq = _rowmajor(Q, "Q")
    _check(lib().gcn_quantize_rows_u8(n, F, X.data_ptr(), ldx, Q.data_ptr(), ldq, zmin.data_ptr(),
                                      scale.data_ptr(), ldp, _stream(stream)))
    return Q, zmin, scale


def gcn_layernorm_quantize(X: torch.Tensor, bits: int = 8, layernorm: bool = True, gamma=None,
                           beta=None, eps: float = 1e-5, paired: bool = True, with_y: bool = False,
                           stream=None):
    """(Q, zmin, scale[, Y]): optional row LayerNorm, then b-bit codes (8 or 2,
    2-bit packed four per byte) with per-row zero point and scale."""
    _dev(X, torch.float32, "X")
    ldx = _rowmajor(X, "X")
    n, F = X.shape
    qb = F if bits == 8 else (F + 3) // 4
    Q = torch.empty((n, qb), dtype=torch.uint8, device=X.device)
    zs = torch.empty((n, 2), dtype=torch.float32, device=X.device)
    zmin, scale = (zs[:, 0], zs[:, 1]) if paired else (zs[:, 0].clone(), zs[:, 1].clone())
    Y = torch.empty((n, F), dtype=torch.float32, device=X.device) if with_y else None
    for t, nm in ((gamma, "gamma"), (beta, "beta")):
        if t is not None:
            _dev(t, torch.float32, nm)
            if t.numel() != F or not t.is_contiguous():
                raise ValueError("%s must hold F contiguous values" % nm)
    ptr = lambda t: t.data_ptr() if t is not None else None
    _check(lib().gcn_layernorm_quantize(n, F, X.data_ptr(), ldx, ptr(gamma), ptr(beta), eps,
                                        GCN_LAYERNORM if layernorm else 0, bits, ptr(Y),
                                        F if Y is not None else 0, Q.data_ptr(), qb,
                                        zmin.data_ptr(), scale.data_ptr(), zmin.stride(0),
                                        _stream(stream)))
    return (Q, zmin, scale, Y) if with_y else (Q, zmin, scale)


def gcn_gemm_f32(op: int, A: torch.Tensor, B: torch.Tensor, C: torch.Tensor | None = None,
                 stream=None):
    """C = A B (NN), A B^T (NT) or A^T B (TN) on the matrix cores, fp32."""
    for t, nm in ((A, "A"), (B, "B")):
        _dev(t, torch.float32, nm)
    lda, ldb = _rowmajor(A, "A"), _rowmajor(B, "B")
    if op == GCN_GEMM_NN:
        (M, K), (K2, N) = A.shape, B.shape
    elif op == GCN_GEMM_NT:
        (M, K), (N, K2) = A.shape, B.shape
    elif op == GCN_GEMM_TN:
        (K, M), (K2, N) = A.shape, B.shape
    else:
        raise ValueError("unknown op")
    if K != K2:
        raise ValueError("inner dimensions differ")
    if C is None:
        C = torch.empty((M, N), dtype=torch.float32, device=A.device)
    _dev(C, torch.float32, "C")
    ldc = _rowmajor(C, "C")
    if tuple(C.shape) != (M, N):
        raise ValueError("C must be %d x %d" % (M, N))
    _check(lib().gcn_gemm_f32(op, M, N, K, A.data_ptr(), lda, B.data_ptr(), ldb, C.data_ptr(), ldc,
                              _stream(stream)))
    return C


def gcn_relu(H: torch.Tensor, stream=None):
    """H = max(H, 0) in place."""
    _dev(H, torch.float32, "H")
    ld = _rowmajor(H, "H")
    _check(lib().gcn_relu(H.shape[0], H.shape[1], H.data_ptr(), ld, _stream(stream)))
    return H


def gcn_relu_bwd(H: torch.Tensor, dH: torch.Tensor, stream=None):
    """dH *= (H > 0) in place."""
    _dev(H, torch.float32, "H")
    _dev(dH, torch.float32, "dH")
    if H.shape != dH.shape:
        raise ValueError("H and dH shapes differ")
    _check(lib().gcn_relu_bwd(H.shape[0], H.shape[1], H.data_ptr(), _rowmajor(H, "H"),
                              dH.data_ptr(), _rowmajor(dH, "dH"), _stream(stream)))
    return dH


def gcn_softmax_xent(logits: torch.Tensor, labels: torch.Tensor, stream=None):
    """(loss device double scalar, dlogits) of the mean softmax cross-entropy."""
    _dev(logits, torch.float32, "logits")
    _dev(labels, torch.int32, "labels")
    n, C = logits.shape
    if labels.numel() != n or not labels.is_contiguous():
        raise ValueError("labels must be contiguous with one entry per row")
    d = torch.empty_like(logits)
    loss = torch.empty((), dtype=torch.float64, device=logits.device)
    _check(lib().gcn_softmax_xent(n, C, logits.data_ptr(), _rowmajor(logits, "logits"),
                                  labels.data_ptr(), d.data_ptr(), _rowmajor(d, "dlogits"),
                                  loss.data_ptr(), _stream(stream)))
    return loss, d


def gcn_gcn2_step(g: Graph, X: torch.Tensor, W1: torch.Tensor, W2: torch.Tensor,
                  labels: torch.Tensor, stream=None):
    """(loss, dW1, dW2) of one training step of the 2-layer GCN."""
    _dev(X, torch.float32, "X")
    for t, nm in ((W1, "W1"), (W2, "W2")):
        _dev(t, torch.float32, nm)
        if not t.is_contiguous():
            raise ValueError("%s must be contiguous" % nm)
    _dev(labels, torch.int32, "labels")
    f_in, hidden = W1.shape
    hidden2, n_classes = W2.shape
    if hidden2 != hidden or X.shape != (g.n_rows, f_in) or labels.numel() != g.n_rows:
        raise ValueError("shape mismatch")
    dW1 = torch.empty_like(W1)
    dW2 = torch.empty_like(W2)
    loss = torch.empty((), dtype=torch.float64, device=X.device)
    _check(lib().gcn_gcn2_step(g.handle, X.data_ptr(), _rowmajor(X, "X"), f_in, W1.data_ptr(),
                               hidden, W2.data_ptr(), n_classes, labels.data_ptr(),
                               dW1.data_ptr(), dW2.data_ptr(), loss.data_ptr(), _stream(stream)))
    return loss, dW1, dW2


def gcn_normalize_mean(g: Graph, stream=None):
    """Values of the mean operator D^-1 A (and its transpose)."""
    _check(lib().gcn_normalize_mean(g.handle, _stream(stream)))


def gcn_layernorm_fwd(X: torch.Tensor, eps: float = 1e-5, Y: torch.Tensor | None = None,
                      stream=None):
    """(Y, rstd): row LayerNorm without affine parameters, and 1/sqrt(var + eps)."""
    _dev(X, torch.float32, "X")
    n, F = X.shape
    if Y is None:
        Y = torch.empty((n, F), dtype=torch.float32, device=X.device)
    _dev(Y, torch.float32, "Y")
    rstd = torch.empty(n, dtype=torch.float32, device=X.device)
    _check(lib().gcn_layernorm_fwd(n, F, X.data_ptr(), _rowmajor(X, "X"), eps, Y.data_ptr(),
                                   _rowmajor(Y, "Y"), rstd.data_ptr(), _stream(stream)))
    return Y, rstd


def gcn_layernorm_bwd(Y: torch.Tensor, rstd: torch.Tensor, dY: torch.Tensor, dY2=None,
                      mask=None, dX: torch.Tensor | None = None, stream=None):
    """dX of the row LayerNorm for g = dY (+ dY2), zeroed where mask <= 0."""
    for t, nm in ((Y, "Y"), (rstd, "rstd"), (dY, "dY")):
        _dev(t, torch.float32, nm)
    n, F = Y.shape
    if dX is None:
        dX = torch.empty((n, F), dtype=torch.float32, device=Y.device)
    ptr = lambda t: t.data_ptr() if t is not None else None  # noqa: E731
    ld = lambda t, nm: _rowmajor(t, nm) if t is not None else 0  # noqa: E731
    _check(lib().gcn_layernorm_bwd(n, F, Y.data_ptr(), _rowmajor(Y, "Y"), rstd.data_ptr(),
                                   dY.data_ptr(), _rowmajor(dY, "dY"), ptr(dY2), ld(dY2, "dY2"),
                                   ptr(mask), ld(mask, "mask"), dX.data_ptr(), _rowmajor(dX, "dX"),
                                   _stream(stream)))
    return dX


def _sage_shapes(g, X, params):
    _dev(X, torch.float32, "X")
    if len(params) != 9:
        raise ValueError("params holds 9 tensors")
    for k, t in enumerate(params):
        _dev(t, torch.float32, "params[%d]" % k)
        if not t.is_contiguous():
            raise ValueError("params[%d] must be contiguous" % k)
    f_in, hidden = params[0].shape
    n_classes = params[6].shape[1]
    shapes = [(f_in, hidden), (f_in, hidden), (hidden,), (hidden, hidden), (hidden, hidden),
              (hidden,), (hidden, n_classes), (hidden, n_classes), (n_classes,)]
    if [tuple(t.shape) for t in params] != shapes:
        raise ValueError("parameter shapes must be %s" % shapes)
    if X.shape != (g.n_rows, f_in):
        raise ValueError("X must be [n x f_in]")
    return f_in, hidden, n_classes


def gcn_sage3_forward(g: Graph, X: torch.Tensor, params, labels=None, lp_mask=None, E=None,
                      eps: float = 1e-5, stream=None):
    """(H1, H2, logits) of the 3-layer GraphSAGE model (the step's forward pass)."""
    f_in, hidden, n_classes = _sage_shapes(g, X, params)
    if lp_mask is not None:
        _dev(lp_mask, torch.uint8, "lp_mask")
        _dev(E, torch.float32, "E")
        _dev(labels, torch.int32, "labels")
    n = g.n_rows
    H1 = torch.empty((n, hidden), dtype=torch.float32, device=X.device)
    H2 = torch.empty_like(H1)
    logits = torch.empty((n, n_classes), dtype=torch.float32, device=X.device)
    pa = (ctypes.c_void_p * 9)(*[t.data_ptr() for t in params])
    ptr = lambda t: t.data_ptr() if t is not None else None  # noqa: E731
    _check(lib().gcn_sage3_forward(g.handle, X.data_ptr(), _rowmajor(X, "X"), f_in, hidden,
                                   n_classes, pa, ptr(labels), ptr(lp_mask), ptr(E), eps,
                                   H1.data_ptr(), hidden, H2.data_ptr(), hidden, logits.data_ptr(),
                                   n_classes, _stream(stream)))
    return H1, H2, logits


def gcn_sage3_step(g: Graph, X: torch.Tensor, params, labels: torch.Tensor, lp_mask=None, E=None,
                   eps: float = 1e-5, stream=None):
    """(loss, grads, dE) of one step of the 3-layer GraphSAGE model.

    params: [W_self1, W_neigh1, b1, W_self2, W_neigh2, b2, W_self3, W_neigh3, b3]."""
    f_in, hidden, n_classes = _sage_shapes(g, X, params)
    _dev(labels, torch.int32, "labels")
    if labels.numel() != g.n_rows:
        raise ValueError("labels must have n entries")
    grads = [torch.empty_like(t) for t in params]
    dE = None
    if lp_mask is not None:
        _dev(lp_mask, torch.uint8, "lp_mask")
        _dev(E, torch.float32, "E")
        if tuple(E.shape) != (n_classes, f_in) or not E.is_contiguous():
            raise ValueError("E must be contiguous [n_classes x f_in]")
        dE = torch.empty_like(E)
    loss = torch.empty((), dtype=torch.float64, device=X.device)
    pa = (ctypes.c_void_p * 9)(*[t.data_ptr() for t in params])
    ga = (ctypes.c_void_p * 9)(*[t.data_ptr() for t in grads])
    _check(lib().gcn_sage3_step(g.handle, X.data_ptr(), _rowmajor(X, "X"), f_in, hidden, n_classes,
                                pa, labels.data_ptr(),
                                lp_mask.data_ptr() if lp_mask is not None else None,
                                E.data_ptr() if E is not None else None, eps, ga,
                                dE.data_ptr() if dE is not None else None, loss.data_ptr(),
                                _stream(stream)))
    return loss, grads, dE


def gcn_graph_info(g: Graph):
    a, b, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(lib().gcn_graph_info(g._h, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)))
    return a.value, b.value, c.value


def gcn_graph_export(g: Graph, which: int = 0, stream=None):
    """Host copies (ptr int64, idx int32, val float32) of A (0) or A^T (1)."""
    n_major = g.n_rows if which == 0 else g.n_cols
    ptr = np.empty(n_major + 1, np.int64)
    idx = np.empty(max(g.nnz, 1), np.int32)
    val = np.empty(max(g.nnz, 1), np.float32)
    _check(lib().gcn_graph_export(g.handle, which, ptr.ctypes.data, idx.ctypes.data,
                                  val.ctypes.data, _stream(stream)))
    return ptr, idx[:g.nnz], val[:g.nnz]


def gcn_graph_bins(g: Graph, which: int = 0, halo_from: int = -1, stream=None):
    """Per row-length class: dict(first_len, last_len, rows, entries, halo_entries)."""
    rec = np.zeros((16, 5), np.int64)
    n = ctypes.c_int(0)
    _check(lib().gcn_graph_bins(g.handle, which, halo_from, rec.ctypes.data, 16, ctypes.byref(n),
                                _stream(stream)))
    return [dict(first_len=int(a), last_len=int(b), rows=int(c), entries=int(d),
                 halo_entries=int(e)) for a, b, c, d, e in rec[:n.value]]


def gcn_profile_enable(on: bool = True):
    _check(lib().gcn_profile_enable(1 if on else 0))


def gcn_profile_read():
    """{kernel name: (launches, total ms)} of the launches since enabling."""
    cap = 64
    names = (ctypes.c_char_p * cap)()
    launches = np.zeros(cap, np.int64)
    ms = np.zeros(cap, np.float64)
    n = ctypes.c_int(0)
    _check(lib().gcn_profile_read(ctypes.cast(names, ctypes.c_void_p), launches.ctypes.data, ms.ctypes.data, cap,
                                  ctypes.byref(n)))
    return {names[i].decode(): (int(launches[i]), float(ms[i])) for i in range(min(n.value, cap))}
