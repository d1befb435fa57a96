"""Seeded synthetic inputs: graphs and feature matrices.

Python side of ``synth.cpp``: counter-based SplitMix64 random numbers, Erdos-
Renyi and RMAT edge lists (with rejection to non-power-of-two vertex counts
and a seeded relabelling permutation), one worker's partition of an RMAT
graph, uniform/normal features, Glorot weights and labels, plus the recipes
for the five workloads the aggregation path is measured and checked on.

Nothing here performs any step of the aggregation method (no CSR build, no
normalization, no aggregation, no quantization); both the GPU library's users
(tests, benchmark) and the CPU oracle's tests draw their inputs from here.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.cpp")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile libsynth.so with g++ (OpenMP)."""
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
        i64, u64, d = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
        lib.synth_splitmix64.argtypes = [u64, u64, i64, P]
        lib.synth_permutation.argtypes = [u64, i64, P]
        lib.synth_er_edges.argtypes = [u64, i64, i64, P, P]
        lib.synth_rmat_edges.argtypes = [u64, i64, i64, d, d, d, P, P, P]
        lib.synth_first_draws.argtypes = [i64, P, P, i64, P]
        lib.synth_first_draws.restype = i64
        lib.synth_nth_set.argtypes = [i64, P, i64]
        lib.synth_nth_set.restype = i64
        lib.synth_partition_select.argtypes = [i64, P, P, P, i64, i64, P]
        lib.synth_partition_select.restype = i64
        lib.synth_partition_emit.argtypes = [i64, P, P, P, i64, i64, P, P, P]
        lib.synth_partition_emit.restype = i64
        lib.synth_uniform.argtypes = [u64, i64, i64, i64, P]
        lib.synth_normal.argtypes = [u64, i64, i64, i64, P]
        lib.synth_glorot.argtypes = [u64, i64, i64, P]
        lib.synth_labels.argtypes = [u64, i64, ctypes.c_int32, P]
        lib.synth_bytes.argtypes = [u64, i64, i64, i64, P]
        lib.synth_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _p(a: np.ndarray) -> int:
    return a.ctypes.data


def splitmix64(seed: int, first: int, count: int) -> np.ndarray:
    out = np.empty(count, np.uint64)
    _L().synth_splitmix64(seed, first, count, _p(out))
    return out


def permutation(seed: int, n: int) -> np.ndarray:
    perm = np.empty(n, np.int32)
    _L().synth_permutation(seed, n, _p(perm))
    return perm


def er_edges(seed: int, n: int, m: int):
    """m ordered pairs uniform on [0, n)^2 -> (src, dst) int32 arrays."""
    src = np.empty(m, np.int32)
    dst = np.empty(m, np.int32)
    _L().synth_er_edges(seed, n, m, _p(src), _p(dst))
    return src, dst


RMAT_ABC = (0.57, 0.19, 0.19)  # d = 0.05


def rmat_edges(seed: int, n: int, m: int, perm_seed: int | None = None, abc=RMAT_ABC):
    """m RMAT draws over [0, n); relabelled through a seeded permutation."""
    perm = permutation(perm_seed, n) if perm_seed is not None else None
    src = np.empty(m, np.int32)
    dst = np.empty(m, np.int32)
    _L().synth_rmat_edges(seed, n, m, abc[0], abc[1], abc[2],
                          _p(perm) if perm is not None else None, _p(src), _p(dst))
    return src, dst


def first_draws(a: np.ndarray, b: np.ndarray, n: int):
    """(first, distinct): first[e] is True for the first draw of each unordered
    pair {a[e], b[e]} with a[e] != b[e]; distinct = number of such pairs."""
    a = np.ascontiguousarray(a, np.int32)
    b = np.ascontiguousarray(b, np.int32)
    first = np.empty(len(a), np.uint8)
    distinct = _L().synth_first_draws(len(a), _p(a), _p(b), n, _p(first))
    return first.view(bool), int(distinct)


def nth_set(flags: np.ndarray, k: int) -> int:
    """Index of the k-th (1-based) True entry, or -1."""
    flags = np.ascontiguousarray(flags).view(np.uint8)
    return int(_L().synth_nth_set(len(flags), _p(flags), k))


def partition_edges(seed: int, perm_seed: int, n_total: int, n_local: int, m: int,
                    target: int | None = None, abc=RMAT_ABC):
    """One worker's share of an undirected RMAT graph over [0, n_total): the
    draws {u, v} of rmat_edges(seed, n_total, m, perm_seed), in draw order;
    each emits "v contributes to row u" when u < n_local and "u contributes to
    row v" when v < n_local (a local-local pair emits both, so the local block
    stays symmetric); self pairs emit nothing (see synth.cpp).

    target (optional): stop once the distinct entries emitted reach exactly
    `target`; a draw whose new entries would pass it is left out.
    Returns (src, dst, raw_count): the entries, "src contributes to row dst",
    in draw order (duplicates included), and per vertex the number of draws
    taken that touch it.
    """
    src_d, dst_d = rmat_edges(seed, n_total, m, perm_seed=perm_seed, abc=abc)
    u, v = dst_d, src_d
    take = np.empty(m, np.uint8)
    if target is None:
        first = np.ones(m, np.uint8)
    else:
        first, _ = first_draws(u, v, n_total)
    used = _L().synth_partition_select(m, _p(u), _p(v), _p(first.view(np.uint8)), n_local,
                                       -1 if target is None else target, _p(take))
    if used < 0:
        raise ValueError("%d draws do not reach %d distinct entries" % (m, target))
    src = np.empty(2 * used, np.int32)
    dst = np.empty(2 * used, np.int32)
    raw = np.empty(n_total, np.int64)
    cnt = _L().synth_partition_emit(used, _p(u), _p(v), _p(take), n_local, n_total, _p(src),
                                    _p(dst), _p(raw))
    return src[:cnt].copy(), dst[:cnt].copy(), raw


def uniform(seed: int, n: int, f: int, ld: int | None = None) -> np.ndarray:
    ld = f if ld is None else ld
    x = np.zeros((n, ld), np.float32)
    _L().synth_uniform(seed, n, f, ld, _p(x))
    return x


def normal(seed: int, n: int, f: int, ld: int | None = None) -> np.ndarray:
    ld = f if ld is None else ld
    x = np.zeros((n, ld), np.float32)
    _L().synth_normal(seed, n, f, ld, _p(x))
    return x


def glorot(seed: int, fan_in: int, fan_out: int) -> np.ndarray:
    w = np.empty((fan_in, fan_out), np.float32)
    _L().synth_glorot(seed, fan_in, fan_out, _p(w))
    return w


def labels(seed: int, n: int, n_classes: int) -> np.ndarray:
    y = np.empty(n, np.int32)
    _L().synth_labels(seed, n, n_classes, _p(y))
    return y


def random_bytes(seed: int, n: int, f: int, ld: int | None = None) -> np.ndarray:
    ld = f if ld is None else ld
    q = np.zeros((n, ld), np.uint8)
    _L().synth_bytes(seed, n, f, ld, _p(q))
    return q


def num_threads() -> int:
    return _L().synth_num_threads()


# ---------------------------------------------------------------------------
# Workload recipes. Seeds: graph 1000+k, permutation 2000+k, X 3000+k,
# G 4000+k, weights/labels 5000+k for workload k.
# ---------------------------------------------------------------------------

SYMMETRIZE = 1
ADD_SELF_LOOPS = 2


@dataclass
class Workload:
    name: str
    n_rows: int
    n_cols: int
    src: np.ndarray
    dst: np.ndarray
    flags: int
    F: int
    deg: np.ndarray | None = None      # caller-supplied global degree (int32, length n_cols)
    n_local_cols: int | None = None    # columns >= this are int8 halo rows
    extra: dict = field(default_factory=dict)


def er_4096(k: int = 1) -> Workload:
    """ER graph: 4096 nodes, 65,536 uniform pairs, symmetrized, +I; F = 64."""
    src, dst = er_edges(1000 + k, 4096, 65536)
    return Workload("er4096_f64", 4096, 4096, src, dst, SYMMETRIZE | ADD_SELF_LOOPS, 64)


def rmat(scale: int, edge_factor: int, F: int, k: int, name: str | None = None,
         halo_fraction: float | None = None) -> Workload:
    """RMAT(.57,.19,.19,.05) over 2^scale nodes with edge_factor*2^scale draws,
    relabelled by a seeded permutation, symmetrized, +I."""
    n = 1 << scale
    src, dst = rmat_edges(1000 + k, n, edge_factor * n, perm_seed=2000 + k)
    nlc = None if halo_fraction is None else n - int(round(n * halo_fraction))
    return Workload(name or f"rmat{scale}_ef{edge_factor}_f{F}", n, n, src, dst,
                    SYMMETRIZE | ADD_SELF_LOOPS, F, n_local_cols=nlc)


def rmat20() -> Workload:
    """RMAT scale 20, edge factor 16, F = 128."""
    return rmat(20, 16, 128, 2)


def rmat24_q8() -> Workload:
    """RMAT scale 24, edge factor 32, F = 128; the last 25% of node ids are
    halo rows held as uint8 codes with per-row (min, scale)."""
    return rmat(24, 32, 128, 5, name="rmat24_ef32_f128_q8halo", halo_fraction=0.25)


def perm22(F: int = 128, k: int = 6) -> Workload:
    """Permutation graph over 2^22 nodes: row i holds the single entry
    (i, perm[i]), no self-loops. Every pass gathers each input row exactly
    once, so its traffic is known exactly: the workload on which hardware
    byte counters of a gather are checked."""
    n = 1 << 22
    perm = permutation(2000 + k, n)
    return Workload("perm22_f%d" % F, n, n, perm.copy(), np.arange(n, dtype=np.int32), 0, F)


def rmat24() -> Workload:
    """RMAT scale 24, edge factor 32, F = 128, every input row fp32."""
    return rmat(24, 32, 128, 5)


def product_like(n: int = 2_449_029, pairs: int = 61_859_140, k: int = 3,
                 max_draws: int = 68_000_000) -> Workload:
    """Product-graph-shaped RMAT: n nodes by rejection from the next power of
    two, permuted; draws are taken in order until they hold exactly `pairs`
    distinct undirected non-loop pairs; symmetrized, +I, so the graph stores
    2 * pairs + n entries (126,167,309 by default)."""
    src, dst = rmat_edges(1000 + k, n, max_draws, perm_seed=2000 + k)
    first, distinct = first_draws(src, dst, n)
    if distinct < pairs:
        raise ValueError("%d draws hold only %d distinct pairs" % (max_draws, distinct))
    m = nth_set(first, pairs) + 1
    return Workload(f"product_like_n{n}", n, n, src[:m].copy(), dst[:m].copy(),
                    SYMMETRIZE | ADD_SELF_LOOPS, 256, extra={"draws": m})


def partition_111m(n_local: int = 14_000_000, n_total: int = 20_000_000,
                   stored: int = 200_000_000, k: int = 4,
                   max_draws: int = 142_000_000) -> Workload:
    """One worker's partition of a large RMAT graph: n_local rows, columns
    over [0, n_total) (ids >= n_local are halo), self-loops on local rows, draws
    taken in order until the rows store exactly `stored` entries (self-loops
    included), normalization by a supplied global degree
    deg = floor(2.2 * raw_count)."""
    src, dst, raw = partition_edges(1000 + k, 2000 + k, n_total, n_local, max_draws,
                                    target=stored - n_local)
    deg = ((raw * 11) // 5).astype(np.int32)
    return Workload(f"partition_{n_local}x{n_total}", n_local, n_total, src, dst, ADD_SELF_LOOPS,
                    128, deg=deg)
