"""gcn_aggregate_fwd_noalloc under stream capture, the use it exists for:
the call is captured once into a HIP graph (torch.cuda.CUDAGraph, which
drives stream capture and graph launch on ROCm) and the graph is replayed
three times, with new inputs copied into the captured input buffer and eager
work and synchronizations between the replays. Every replay must equal the
eager allocating call on the same inputs bit for bit (same kernels, same
summation order), and the oracle within 1e-5 * S. The graphs have rows long
enough to write partial rows (a chunked and a column-blocked plan), so the
library's fixed partial-row array is used inside the graph."""

import numpy as np
import pytest

import synth
from gpu_util import assert_close, dev, host, note
from test_zz_no_alloc import build_with

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2411_16025_amd as pkg
    pkg.lib()
    return pkg


@pytest.mark.parametrize("name,n,m,seed,env,F", [
    ("chunked", 1 << 14, 16 << 14, 921, {"GCN_CHUNK_LEN": "256"}, 64),
    ("blocked", 1 << 13, 12 << 13, 923, {"GCN_BLOCK_MIN_COLS": "0", "GCN_COL_BLOCKS": "16",
                                         "GCN_SEGMENT_MIN": "8"}, 47),
])
def test_noalloc_graph_replays(G, name, n, m, seed, env, F):
    import torch
    note("noalloc graph capture %s n=%d F=%d" % (name, n, F))
    g, og = build_with(G, n, m, seed, env)
    Xs = dev(synth.uniform(seed + 2, n, F))  # the captured input buffer
    Ys = torch.empty((n, F), device="cuda:0")
    G.gcn_aggregate_fwd_noalloc(g, Xs, Ys)  # eager first call: the symbol lookup
    torch.cuda.synchronize()
    side = torch.cuda.Stream()  # default priority
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        G.gcn_aggregate_fwd_noalloc(g, Xs, Ys)
    torch.cuda.synchronize()
    for rep in range(3):
        X = synth.uniform(seed + 10 + rep, n, F)
        Xs.copy_(dev(X))
        Ys.fill_(7.0)  # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = host(Ys)
        want = host(G.gcn_aggregate_fwd(g, dev(X)))
        torch.cuda.synchronize()
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (name, rep)
        if rep == 0:
            assert_close(got, *og.fwd(X), what="graph replay %s vs oracle" % name)
    del graph
    g.free()
