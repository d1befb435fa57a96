"""Generators: counter-based determinism and the shapes the workloads need."""

import hashlib
import os
import subprocess
import sys

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _digest_in_subprocess(threads):
    code = (
        "import hashlib, synth\n"
        "s, d = synth.rmat_edges(7, 3000, 50000, perm_seed=8)\n"
        "x = synth.normal(9, 300, 33)\n"
        "p, q, r = synth.partition_edges(10, 11, 5000, 3500, 20000)\n"
        "f, _ = synth.first_draws(s, d, 3000)\n"
        "t, u, v = synth.partition_edges(10, 11, 5000, 3500, 20000, target=12345)\n"
        "h = hashlib.sha256()\n"
        "[h.update(a.tobytes()) for a in (s, d, x, p, q, r, f, t, u, v)]\n"
        "print(h.hexdigest())\n")
    env = dict(os.environ, OMP_NUM_THREADS=str(threads), PYTHONPATH=ROOT)
    return subprocess.check_output([sys.executable, "-c", code], env=env, cwd=ROOT).strip()


def test_thread_count_independence():
    assert _digest_in_subprocess(1) == _digest_in_subprocess(5)


def test_splitmix64_reference_values():
    # SplitMix64 seeded with 0: first outputs of the published generator
    out = synth.splitmix64(0, 0, 3)
    assert list(out) == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_uniform_is_exact_grid():
    x = synth.uniform(1, 1000, 64)
    assert x.min() >= -1.0 and x.max() < 1.0
    k = (x.astype(np.float64) + 1.0) * 2.0**23
    assert np.array_equal(k, np.round(k))


def test_permutation_is_permutation():
    p = synth.permutation(3, 100003)
    assert np.array_equal(np.sort(p), np.arange(100003))
    assert not np.array_equal(p, np.arange(100003))


def test_rmat_quadrant_frequencies():
    # top-level quadrant of an unpermuted RMAT draw over 2^16 nodes
    n = 1 << 16
    src, dst = synth.rmat_edges(4, n, 200000)
    hu = (dst >> 15) & 1  # u -> dst
    hv = (src >> 15) & 1
    freq = [np.mean((hu == a) & (hv == b)) for a, b in ((0, 0), (0, 1), (1, 0), (1, 1))]
    assert np.allclose(freq, [0.57, 0.19, 0.19, 0.05], atol=0.005)


def test_rmat_rejection_keeps_range():
    src, dst = synth.rmat_edges(5, 1000, 100000, perm_seed=6)
    assert src.min() >= 0 and src.max() < 1000 and dst.max() < 1000


def test_partition_shape():
    src, dst, raw = synth.partition_edges(12, 13, 20000, 14000, 100000)
    assert dst.max() < 14000 and src.max() < 20000
    assert np.all(src != dst)
    assert raw.sum() <= 2 * 100000
    assert np.mean(src >= 14000) > 0.2  # halo columns are referenced


def test_first_draws_brute_force():
    rng = np.random.default_rng(5)
    a = rng.integers(0, 40, 3000).astype(np.int32)
    b = rng.integers(0, 40, 3000).astype(np.int32)
    first, distinct = synth.first_draws(a, b, 40)
    seen, want = set(), []
    for x, y in zip(a.tolist(), b.tolist()):
        k = (min(x, y), max(x, y))
        want.append(x != y and k not in seen)
        if x != y:
            seen.add(k)
    assert first.tolist() == want and distinct == len(seen)
    assert synth.nth_set(first, distinct) == max(i for i, w in enumerate(want) if w)
    assert synth.nth_set(first, distinct + 1) == -1


@pytest.mark.parametrize("target", [20000, 20001, 30123])
def test_partition_exact_entry_count(target):
    # distinct (row, col) entries of the emitted list reach exactly the target
    src, dst, raw = synth.partition_edges(14, 15, 20000, 14000, 100000, target=target)
    keys = np.unique(dst.astype(np.int64) * 20000 + src)
    assert len(keys) == target
    assert np.all(src != dst) and dst.max() < 14000
    # a taken draw adds 2 to the counts and emits at most 2 entries
    assert raw.sum() >= len(src)
    full, _, _ = synth.partition_edges(14, 15, 20000, 14000, 100000)
    # the taken draws are a prefix of the draws, save those left out
    assert len(src) <= len(full)
