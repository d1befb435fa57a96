"""gcn_aggregate_fwd_noalloc: the forward aggregation with the library's
fixed partial-row array, called through the C ABI, against
gcn_aggregate_fwd on the same inputs (identical bits: same kernels, same
summation order) and against the oracle (1e-5 * S). Two calls in a row on
graphs whose long rows write partial rows, the second on a smaller graph
and a narrower F; the over-capacity case fails with GCN_ERANGE before any
work; and the call takes nothing from the device's stream-ordered pool."""

import ctypes
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_close, dev, host, note

pytestmark = pytest.mark.gpu

FLAGS = synth.SYMMETRIZE | synth.ADD_SELF_LOOPS


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2411_16025_amd as pkg
    pkg.lib()
    return pkg


def build_with(G, n, m, seed, env):
    src, dst = synth.rmat_edges(seed, n, m, perm_seed=seed + 1)
    old = {k: os.environ.get(k) for k in env}
    os.environ.update(env)
    try:
        g = G.gcn_build_csr(n, n, dev(src), dev(dst), FLAGS)
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    G.gcn_normalize(g)
    return g, oracle.Graph(n, n, src, dst, FLAGS)


class Pool:
    """Used-memory counters of the current device's default memory pool (the
    one the library's stream-ordered temporaries come from)."""

    def __init__(self):
        import torch
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.pool = ctypes.c_void_p()
        assert self.hip.hipDeviceGetDefaultMemPool(ctypes.byref(self.pool),
                                                   torch.cuda.current_device()) == 0

    def get(self, attr):
        v = ctypes.c_uint64(0)
        assert self.hip.hipMemPoolGetAttribute(self.pool, attr, ctypes.byref(v)) == 0
        return v.value

    def reset_high(self):
        zero = ctypes.c_uint64(0)
        return self.hip.hipMemPoolSetAttribute(self.pool, 0x8, ctypes.byref(zero)) == 0

    def used(self):
        return self.get(0x7)

    def high(self):
        return self.get(0x8)


def test_noalloc_matches_fwd_twice_then_smaller(G):
    import torch
    cases = [
        # rows of more than one 256-entry chunk write partial rows
        ("chunked", 1 << 15, 16 << 15, 901, {"GCN_CHUNK_LEN": "256"}, 128),
        # every row over 48 entries cut at column blocks into pieces
        ("blocked", 1 << 13, 12 << 13, 903, {"GCN_BLOCK_MIN_COLS": "0", "GCN_COL_BLOCKS": "16",
                                             "GCN_SEGMENT_MIN": "8"}, 47),
    ]
    for name, n, m, seed, env, F in cases:
        note("noalloc %s n=%d F=%d" % (name, n, F))
        g, og = build_with(G, n, m, seed, env)
        X = synth.uniform(seed + 2, n, F)
        Xd = dev(X)
        want = G.gcn_aggregate_fwd(g, Xd)
        Y = torch.full((n, F), 7.0, device="cuda:0")
        G.gcn_aggregate_fwd_noalloc(g, Xd, Y)
        torch.cuda.synchronize()
        got = host(Y)
        assert np.array_equal(got.view(np.uint32), host(want).view(np.uint32)), name
        assert_close(got, *og.fwd(X), what="noalloc %s vs oracle" % name)
        g.free()


def test_noalloc_takes_nothing_from_the_pool(G):
    import torch
    note("noalloc pool counters")
    g, _ = build_with(G, 1 << 14, 16 << 14, 905, {"GCN_CHUNK_LEN": "256"})
    Xd = dev(synth.uniform(906, 1 << 14, 64))
    Y = torch.empty((1 << 14, 64), device="cuda:0")
    G.gcn_aggregate_fwd_noalloc(g, Xd, Y)  # first call on the device: symbol lookup
    torch.cuda.synchronize()
    pool = Pool()
    if not pool.reset_high() or pool.high() != pool.used():
        pytest.skip("the pool's high-water mark cannot be reset here")
    base = pool.used()
    G.gcn_aggregate_fwd_noalloc(g, Xd, Y)
    torch.cuda.synchronize()
    assert pool.high() == base, "the no-allocation call took pool memory"
    # the allocating call does take its partial rows from the pool
    assert pool.reset_high()
    G.gcn_aggregate_fwd(g, Xd)
    torch.cuda.synchronize()
    assert pool.high() > base
    g.free()


def test_noalloc_rejects_plans_beyond_its_array(G):
    import torch
    note("noalloc over capacity")
    # 16-entry pieces cut at every block: over a hundred thousand partial
    # rows of 256 floats, beyond the 2^24 floats of the array
    n = 1 << 17
    g, _ = build_with(G, n, 16 * n, 907, {"GCN_BLOCK_MIN_COLS": "0", "GCN_SEGMENT_MIN": "0",
                                           "GCN_PIECE_MAX": "16"})
    Xd = dev(synth.uniform(908, n, 256))
    Y = torch.full((n, 256), 7.0, device="cuda:0")
    with pytest.raises(G.GcnError) as e:
        G.gcn_aggregate_fwd_noalloc(g, Xd, Y)
    assert e.value.status == 2 and "no-allocation" in e.value.message
    torch.cuda.synchronize()
    assert bool(torch.all(Y == 7.0)), "output touched on error"
    # the allocating call runs the same graph
    G.gcn_aggregate_fwd(g, Xd, Y)
    torch.cuda.synchronize()
    g.free()
