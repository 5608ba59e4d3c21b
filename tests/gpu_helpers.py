"""Shared helpers of the GPU parity tests (test infrastructure)."""
from __future__ import annotations

import sys

import numpy as np

# The bar for floating-point outputs (soft mask, grad_logits): elementwise
# |gpu - oracle| <= ATOL + RTOL * |oracle|.
RTOL = 1e-5
ATOL = 1e-6


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def bf16_bits(t) -> np.ndarray:
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def f32(t) -> np.ndarray:
    return t.detach().contiguous().cpu().numpy().astype(np.float32)


def assert_close(got, ref, what, rtol=RTOL, atol=ATOL, scale_aware=False):
    got = np.asarray(got, dtype=np.float64).reshape(-1)
    ref = np.asarray(ref, dtype=np.float64).reshape(-1)
    assert got.shape == ref.shape
    assert np.all(np.isfinite(got)), f"{what}: non-finite GPU values"
    a = atol * (np.abs(ref).max() if scale_aware and ref.size else 1.0)
    err = np.abs(got - ref)
    bound = a + rtol * np.abs(ref)
    bad = err > bound
    if bad.any():
        i = int(np.argmax(err - bound))
        raise AssertionError(
            f"{what}: {int(bad.sum())}/{ref.size} elements out of tolerance "
            f"(atol={a:.3g}, rtol={rtol}); worst at {i}: gpu={got[i]!r} oracle={ref[i]!r} "
            f"err={err[i]:.3g}")
    return float((err / np.maximum(bound, 1e-300)).max()) if ref.size else 0.0
