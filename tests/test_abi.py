"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments before touching the GPU (no compute calls here)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gcnagg.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gcn_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    import paper_2411_16025_amd as pkg
    return pkg.lib()


def test_exports_every_declared_symbol(L):
    import paper_2411_16025_amd as pkg
    names = declared_functions()
    assert len(names) >= 13
    assert sorted(pkg.EXPORTS) == names
    for n in names:
        assert hasattr(L, n), n


def test_binding_names_match_entry_points():
    import paper_2411_16025_amd as pkg
    for n in ("gcn_build_csr", "gcn_normalize", "gcn_aggregate_fwd", "gcn_aggregate_bwd",
              "gcn_aggregate_fwd_q8halo"):
        assert callable(getattr(pkg, n))


def _err(L):
    return L.gcn_last_error().decode()


def test_build_rejects_bad_arguments(L):
    out = ctypes.c_void_p(0)
    ref = ctypes.byref(out)
    fake = ctypes.c_void_p(0x1000)
    assert L.gcn_build_csr(0, 5, 0, None, None, 0, None, ref) == 1
    assert "positive" in _err(L)
    assert L.gcn_build_csr(5, -1, 0, None, None, 0, None, ref) == 1
    assert L.gcn_build_csr(5, 6, 0, None, None, 1, None, ref) == 1  # symmetrize, rectangular
    assert "square" in _err(L)
    assert L.gcn_build_csr(5, 5, 3, None, fake, 0, None, ref) == 1  # NULL src
    assert L.gcn_build_csr(5, 5, -2, fake, fake, 0, None, ref) == 1
    assert L.gcn_build_csr(5, 5, 0, None, None, 8, None, ref) == 1  # unknown flag
    assert L.gcn_build_csr(1 << 31, 5, 0, None, None, 0, None, ref) == 2
    assert L.gcn_build_csr(5, 5, 0, None, None, 0, None, None) == 1  # NULL out
    assert out.value is None


def test_calls_reject_null_and_corrupt_handles(L):
    assert L.gcn_normalize(None, None, None) == 1
    assert L.gcn_aggregate_fwd(None, None, 0, 0, None, 0, 4, None) == 1
    assert L.gcn_aggregate_bwd(None, None, 0, 0, None, 0, 4, None) == 1
    assert L.gcn_aggregate_fwd_q8halo(None, 0, None, 0, None, 0, None, None, 1, None, 0, 4, 0,
                                      None) == 1
    # a block of memory that is not a graph handle is reported as ESTATE
    junk = (ctypes.c_uint64 * 64)()
    assert L.gcn_graph_info(ctypes.cast(junk, ctypes.c_void_p), None, None, None) == 5
    assert "freed or corrupted" in _err(L)
    assert L.gcn_graph_export(ctypes.cast(junk, ctypes.c_void_p), 0, None, None, None, None) == 5
    L.gcn_graph_free(None)  # ignored


def test_quantize_rejects_bad_arguments(L):
    fake = ctypes.c_void_p(0x1000)
    assert L.gcn_quantize_rows_u8(4, 0, fake, 4, fake, 4, fake, fake, 1, None) == 1
    assert L.gcn_quantize_rows_u8(4, 8, fake, 4, fake, 8, fake, fake, 1, None) == 1  # ldx < F
    assert L.gcn_quantize_rows_u8(4, 8, None, 8, fake, 8, fake, fake, 1, None) == 1
    assert L.gcn_quantize_rows_u8(4, 8, fake, 8, fake, 8, fake, fake, 0, None) == 1  # ldp < 1
    assert L.gcn_quantize_rows_u8(0, 8, None, 8, None, 8, None, None, 1, None) == 0  # no rows


def test_last_error_is_per_thread(L):
    import threading
    assert L.gcn_build_csr(0, 5, 0, None, None, 0, None, None) == 1
    seen = []
    t = threading.Thread(target=lambda: seen.append(L.gcn_last_error()))
    t.start()
    t.join()
    assert seen == [b""]


def test_profile_toggle_without_launches(L):
    assert L.gcn_profile_enable(1) == 0
    n = ctypes.c_int(-1)
    assert L.gcn_profile_read(None, None, None, 0, ctypes.byref(n)) == 0
    assert n.value == 0
    assert L.gcn_profile_enable(0) == 0


def test_new_entry_points_reject_bad_arguments(L):
    import ctypes
    fake = ctypes.c_void_p(0x1000)
    junk = (ctypes.c_uint64 * 64)()
    jh = ctypes.cast(junk, ctypes.c_void_p)
    # normalization variants
    assert L.gcn_normalize_mean(None, None) == 1
    assert L.gcn_normalize_mean(jh, None) == 5
    assert L.gcn_normalize_rc(None, fake, fake, None) == 1
    assert L.gcn_normalize_rc(jh, fake, fake, None) == 5
    # LayerNorm forward / backward
    assert L.gcn_layernorm_fwd(-1, 4, fake, 4, 1e-5, fake, 4, None, None) == 1
    assert L.gcn_layernorm_fwd(4, 0, fake, 4, 1e-5, fake, 4, None, None) == 1
    assert L.gcn_layernorm_fwd(4, 8, fake, 4, 1e-5, fake, 8, None, None) == 1  # ldx < F
    assert L.gcn_layernorm_fwd(4, 8, None, 8, 1e-5, fake, 8, None, None) == 1
    assert L.gcn_layernorm_fwd(4, 8, fake, 8, -1.0, fake, 8, None, None) == 1  # eps < 0
    assert L.gcn_layernorm_fwd(0, 8, None, 8, 1e-5, None, 8, None, None) == 0  # no rows
    assert L.gcn_layernorm_bwd(4, 8, fake, 8, None, fake, 8, None, 0, None, 0, fake, 8, None) == 1
    assert L.gcn_layernorm_bwd(4, 8, fake, 8, fake, fake, 8, fake, 4, None, 0, fake, 8, None) == 1
    assert L.gcn_layernorm_bwd(0, 8, None, 8, None, None, 8, None, 0, None, 0, None, 8, None) == 0
    # GraphSAGE step and forward
    params = (ctypes.c_void_p * 9)(*([0x1000] * 9))
    grads = (ctypes.c_void_p * 9)(*([0x1000] * 9))
    assert L.gcn_sage3_step(None, fake, 4, 4, 8, 3, params, fake, None, None, 1e-5, grads, None,
                            fake, None) == 1
    assert L.gcn_sage3_step(jh, fake, 4, 4, 8, 3, params, fake, None, None, 1e-5, grads, None,
                            fake, None) == 5
    assert L.gcn_sage3_forward(None, fake, 4, 4, 8, 3, params, None, None, None, 1e-5, None, 0,
                               None, 0, None, 0, None) == 1
    # combine of received partial sums
    assert L.gcn_add_rows(0, 4, None, 4, None, 10, None, 4, None) == 0
    assert L.gcn_add_rows(3, 0, fake, 4, fake, 10, fake, 4, None) == 1
    assert L.gcn_add_rows(3, 8, fake, 4, fake, 10, fake, 8, None) == 1  # ldp < F
    assert L.gcn_add_rows(3, 4, None, 4, fake, 10, fake, 4, None) == 1
