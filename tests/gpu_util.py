"""Shared helpers of the GPU parity tests (host side only)."""

import sys

import numpy as np

import oracle


def note(msg):
    """Name the case about to run on the GPU (flushed, so it survives a crash)."""
    print("[gpu-case] " + msg, flush=True)
    sys.stdout.flush()


def dev(a, device="cuda:0"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def host(t):
    return t.detach().cpu().numpy()


def assert_close(y, ref, S, rel=1e-5, what=""):
    """|y - ref| <= rel * S elementwise, S = sum of |terms| from the oracle."""
    y = np.asarray(y, np.float64)
    err = np.abs(y - ref)
    bound = rel * S + 1e-30
    bad = err > bound
    if what and err.size:
        note("%s: max err/S %.2e over %d elements" % (what, float((err / np.maximum(S, 1e-300)).max()), err.size))
    if bad.any():
        idx = np.argwhere(bad)
        ratio = (err / np.maximum(S, 1e-300)).max()
        r, c = idx[0]
        raise AssertionError(
            "%s: %d of %d elements outside %.1e*S (max err/S %.3e); first at %s: got %r want %r S %r"
            % (what, bad.sum(), bad.size, rel, ratio, (int(r), int(c)), y[r, c], ref[r, c], S[r, c]))


def bf16_round(x):
    """Round fp32 to bf16 (round-half-even) and widen back to fp32, on the host."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) & 0xFFFF
    return (r.astype(np.uint32) << 16).view(np.float32)


def bf16_bits(x):
    """The bf16 bit patterns of bf16_round(x) as uint16."""
    return (bf16_round(x).view(np.uint32) >> 16).astype(np.uint16)


def oracle_graph(w, normalized=True):
    return oracle.Graph(w.n_rows, w.n_cols, w.src, w.dst, w.flags, deg=w.deg, normalized=normalized)
