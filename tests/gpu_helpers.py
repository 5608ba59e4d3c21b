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


# The hardware-log noise of the kernels, N(x) = -log2(-log2 u(x)), against the
# exact noise g of the oracle: |N - (g log2(e) + log2(ln 2))| <= HW_NOISE_A +
# HW_NOISE_B |N| for every one of the 2^23 uniforms, and <= HW_NOISE_MAX
# (test_hardware_noise_bound checks both exhaustively).
HW_NOISE_A = 6e-7
HW_NOISE_B = 1e-7
HW_NOISE_MAX = 2.5e-6
LOG2E = 1.4426950408889634
LOG2_LN2 = float(np.log2(np.log(2.0)))


def backward_key_error(kappa, g, a):
    """Per-key bound (natural units) of how far the backward's keys may sit from
    the exact fp32 keys kappa = fl(a + g), a = fl(phi / lambda): the hardware
    noise bound above, the roundings of fl(log2(e) / lambda) and of a (3 units
    of 2^-24 |a|), of kappa and of the key's fma (2 units of 2^-24 |kappa|),
    plus 2 ulp of kappa for the fp32 evaluation of the relaxation."""
    kappa = np.abs(np.asarray(kappa, dtype=np.float64))
    N = np.abs(np.asarray(g, dtype=np.float64) * LOG2E + LOG2_LN2)
    a = np.abs(np.asarray(a, dtype=np.float64))
    u = 2.0 ** -24
    return np.log(2.0) * (HW_NOISE_A + HW_NOISE_B * N) + 3 * u * a + 6 * u * kappa


def key_error_floor(oracle, kappa, delta, sbar, n, tau, lam, factor=4.0):
    """Allowance for fp32 conditioning of dL/dphi: `factor` times the
    first-order worst case sum_i |grad(kappa + delta_i e_i) - grad(kappa)| of
    the oracle's fp64 gradient when each key moves by its bound delta_i.
    kappa, delta, sbar: [groups, m]."""
    kappa = np.asarray(kappa, dtype=np.float64)
    delta = np.asarray(delta, dtype=np.float64)
    groups, m = kappa.shape
    grad = lambda k: np.stack([oracle.relax_bwd(k[q], n, tau, sbar[q]) for q in range(groups)])
    base = grad(kappa)
    floor = np.zeros_like(base)
    for i in range(m):
        kp = kappa.copy()
        kp[:, i] += delta[:, i]
        floor += np.abs(grad(kp) - base)
    return factor * floor / lam
