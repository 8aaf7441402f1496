"""Helpers of the GPU parity tests: drive a Session and the oracle on the same
seeded inputs and compare bit patterns."""
from __future__ import annotations

import numpy as np


def f32_bits(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def assert_bits_equal(got, want, what: str) -> None:
    g = f32_bits(got) if np.asarray(got).dtype == np.float32 else np.asarray(got)
    w = f32_bits(want) if np.asarray(want).dtype == np.float32 else np.asarray(want)
    assert g.shape == w.shape, (what, g.shape, w.shape)
    bad = np.flatnonzero(g != w)
    if bad.size:
        i = int(bad[0])
        raise AssertionError(f"{what}: {bad.size} of {g.size} differ; first at {i}: got {got[i]!r} "
                             f"({int(g[i]):#x}) want {want[i]!r} ({int(w[i]):#x})")


def assert_bits_equal_nan(got, want, what: str) -> None:
    """assert_bits_equal, except that a NaN equals any NaN: the NaN an
    invalid operation (inf / inf) produces differs between the device and the
    host in sign and payload, which the arithmetic contract does not fix."""
    g, w = np.asarray(got), np.asarray(want)
    if g.dtype != np.float32:
        return assert_bits_equal(got, want, what)
    both = np.isnan(g) & np.isnan(w.astype(np.float32))
    g2, w2 = g.copy(), np.asarray(w, dtype=np.float32).copy()
    g2[both] = 0.0
    w2[both] = 0.0
    assert_bits_equal(g2, w2, what)


def to_device_grad16(sess, bits: np.ndarray):
    """Copy 16-bit gradient patterns (bf16 or fp16) into the session's
    gradient buffer on its compute stream."""
    import torch
    src = torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16))
    with torch.cuda.stream(sess.compute):
        sess.grad.view(torch.int16).copy_(src)


def load_state(sess, p, m=None, v=None, w=None):
    import torch
    with torch.cuda.stream(sess.compute):
        sess.master.copy_(torch.from_numpy(np.ascontiguousarray(p, dtype=np.float32)))
        if m is not None:
            sess.exp_avg.copy_(torch.from_numpy(np.ascontiguousarray(m, dtype=np.float32)))
        else:
            sess.exp_avg.zero_()
        if v is not None:
            sess.exp_avg_sq.copy_(torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32)))
        else:
            sess.exp_avg_sq.zero_()
        if sess.weight is not None:
            if w is not None:
                sess.weight.view(torch.int16).copy_(torch.from_numpy(np.ascontiguousarray(w, np.uint16)
                                                                     .view(np.int16)))
            else:
                sess.weight.copy_(sess.master.to(torch.bfloat16))
    sess.compute.synchronize()
