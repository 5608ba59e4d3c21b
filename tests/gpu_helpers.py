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


# The fp32 rounding allowance of the relaxation's gradient.  The keys are fp32
# values by definition, and an fp32 evaluation of the recursion rounds its
# softmax arguments (the scaled keys, and in the log-domain form their per-step
# updates) at the level of a few units in the last place of the keys.  Where the
# gradient is ill-conditioned in the keys (unit-scale upstream gradients, small
# tau, near-dominant entries) no fp32 evaluation can be closer to the fp64
# oracle than that: the allowance is FP32_FLOOR_FACTOR times the first-order
# change sum_i |grad(kappa + ulp(kappa_i) e_i) - grad(kappa)| of the oracle's
# own fp64 gradient, per element.  It depends on the keys and the arithmetic
# only, never on the kernels.
FP32_FLOOR_FACTOR = 8.0


def bf16_rne_bits(x) -> np.ndarray:
    """bf16 patterns of fp32 values, round to nearest with ties to even
    (finite inputs)."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)


def soft_product_exact(W_bits, S, Ws_bits, what):
    """W_soft is bf16(W (.) S) for the kernel's own fp32 S, bit for bit: the
    fp32 product (one rounding) then the nearest bf16, ties to even."""
    w = (np.asarray(W_bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).reshape(-1)
    prod = w * np.asarray(S, dtype=np.float32).reshape(-1)  # fp32 multiply, round to nearest
    want = bf16_rne_bits(prod)
    got = np.asarray(Ws_bits, dtype=np.uint16).reshape(-1)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, (f"{what}: {bad.size} elements are not the rounded product; first at "
                           f"{bad[0]}: got 0x{got[bad[0]]:04x}, want 0x{want[bad[0]]:04x}")


def sbar_of(G_bits, W_bits) -> np.ndarray:
    """dL/dS = dL/dW_masked (.) W in fp64 (exact: a product of two bf16 values)."""
    g = (np.asarray(G_bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    w = (np.asarray(W_bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    return g.astype(np.float64) * w.astype(np.float64)


def fp32_key_floor(oracle, kappa, sbar, n, tau, lam, factor=FP32_FLOOR_FACTOR, threads=None):
    """Per-element fp32 allowance of dL/dphi (see above); kappa (fp32 keys)
    and sbar are [groups, m]."""
    k32 = np.asarray(kappa, dtype=np.float32)
    groups, m = k32.shape
    sb = np.asarray(sbar, dtype=np.float64).reshape(groups, m)
    threads = oracle.host_threads() if threads is None else threads
    base = oracle.relax_bwd_groups(k32.astype(np.float64), n, tau, sb, threads=threads)
    ulp = np.spacing(np.abs(k32)).astype(np.float64)
    floor = np.zeros_like(base)
    for i in range(m):
        kp = k32.astype(np.float64)
        kp[:, i] += ulp[:, i]
        floor += np.abs(oracle.relax_bwd_groups(kp, n, tau, sb, threads=threads) - base)
    return factor * floor / lam
