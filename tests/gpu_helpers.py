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


def assert_close(got, ref, what, rtol=RTOL, atol=ATOL, scale_aware=False, floor=None):
    """Elementwise |got - ref| <= atol + rtol |ref| (+ floor, when given: an
    extra per-element allowance for fp32 conditioning)."""
    got = np.asarray(got, dtype=np.float64).reshape(-1)
    ref = np.asarray(ref, dtype=np.float64).reshape(-1)
    assert got.shape == ref.shape
    assert np.all(np.isfinite(got)), f"{what}: non-finite GPU values"
    a = atol * (np.abs(ref).max() if scale_aware and ref.size else 1.0)
    err = np.abs(got - ref)
    bound = a + rtol * np.abs(ref)
    if floor is not None:
        bound = bound + np.asarray(floor, dtype=np.float64).reshape(-1)
    bad = err > bound
    if bad.any():
        i = int(np.argmax(err - bound))
        raise AssertionError(
            f"{what}: {int(bad.sum())}/{ref.size} elements out of tolerance "
            f"(atol={a:.3g}, rtol={rtol}); worst at {i}: gpu={got[i]!r} oracle={ref[i]!r} "
            f"err={err[i]:.3g}")
    return float((err / np.maximum(bound, 1e-300)).max()) if ref.size else 0.0


def key_ulp_sensitivity(oracle, kappa, sbar, n, tau, lam, trials=4, seed=0):
    """fp32 noise floor of dL/dphi: the largest change of the oracle's fp64
    gradient when every key moves by a random +-1 ulp (the keys are fp32, so
    any fp32 evaluation of the relaxation perturbs them at this level).
    kappa, sbar: [groups, m]."""
    rng = np.random.default_rng(seed)
    kappa = np.asarray(kappa, dtype=np.float32)
    groups, m = kappa.shape
    base = np.stack([oracle.relax_bwd(kappa[q].astype(np.float64), n, tau, sbar[q]) for q in range(groups)])
    sens = np.zeros_like(base)
    for _ in range(trials):
        sign = rng.choice(np.array([-1.0, 1.0], dtype=np.float32), size=kappa.shape)
        kp = np.nextafter(kappa, (np.float32(np.inf) * sign).astype(np.float32))
        pert = np.stack([oracle.relax_bwd(kp[q].astype(np.float64), n, tau, sbar[q]) for q in range(groups)])
        sens = np.maximum(sens, np.abs(pert - base))
    return sens / lam
