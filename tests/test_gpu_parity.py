"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.  Selected indices, hard masks and masked weights must be
bit-exact; the soft mask and grad_logits must be within 1e-5 relative /
1e-6 absolute (fp32 against the oracle's fp64).

The straight-through forward decides with keys from the hardware logarithm
and falls back to the exact keys where two keys are within its error margin;
its selections are compared bit for bit, with and without the soft mask, and
on inputs built so that keys tie or nearly tie (the margin's bound on the
hardware noise is pinned exhaustively here).  Every relaxation -- the soft
mask, the soft forward and every backward -- runs at the exact keys."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2608_23048_amd as roi
from paper_2608_23048_amd import workloads as wl
from tests.gpu_helpers import (HW_NOISE_A, HW_NOISE_B, HW_NOISE_MAX, LOG2_LN2, LOG2E,
                               assert_close, bf16_bits, f32, fp32_key_floor, sbar_of, say,
                               soft_product_exact)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available()
    roi.lib()  # raises if the HIP library is missing
    return torch.device("cuda:0")


def run_case(dev, rows, cols, n, m, tau, lam, seed, step, off, case_seed, w_std=wl.W_STD,
             grad_std=wl.GRAD_STD, logit_std=wl.LOGIT_STD, scale_aware=False, logits=None):
    import torch
    say(f"case rows={rows} cols={cols} {n}:{m} tau={tau} lam={lam} seed={seed} step={step} "
        f"off={off} case_seed={case_seed}")
    W, L, G = wl.small_case(rows, cols, case_seed, device=dev, w_std=w_std, logit_std=logit_std,
                            grad_std=grad_std)
    if logits is not None:
        L = torch.from_numpy(np.ascontiguousarray(logits, dtype=np.float32)).to(dev)
    Wm, S, idx = roi.mask_fwd(W, L, n, m, tau, lam, seed, step, off, want_soft=True)
    d = roi.mask_bwd(G, W, L, n, m, tau, lam, seed, step, off)
    torch.cuda.synchronize()
    tau32 = float(np.float32(tau))
    lam32 = float(np.float32(lam))
    Wm_o, S_o, idx_o = oracle.mask_fwd(bf16_bits(W), f32(L), n, m, tau32, lam32, seed, step, off)
    d_o = oracle.mask_bwd(bf16_bits(G), bf16_bits(W), f32(L), n, m, tau32, lam32, seed, step, off)
    assert np.array_equal(idx.cpu().numpy(), idx_o), "selected indices differ"
    assert np.array_equal(bf16_bits(Wm).reshape(-1), Wm_o), "masked weights differ"
    # the straight-through forward without the soft mask (hardware-key comparisons)
    Wm2, _, idx2 = roi.mask_fwd(W, L, n, m, tau, lam, seed, step, off, want_soft=False)
    Wm3, _, _ = roi.mask_fwd(W, L, n, m, tau, lam, seed, step, off, want_idx=False)
    torch.cuda.synchronize()
    assert np.array_equal(idx2.cpu().numpy(), idx_o), "selected indices differ (no soft mask)"
    assert np.array_equal(bf16_bits(Wm2).reshape(-1), Wm_o), "masked weights differ (no soft mask)"
    assert np.array_equal(bf16_bits(Wm3).reshape(-1), Wm_o), "masked weights differ (no indices)"
    rs = assert_close(f32(S), S_o, "soft mask")
    check_grad(d, d_o, L, G, W, n, m, tau32, lam32, seed, step, off, scale_aware)
    say(f"  ok: soft-mask err/bound {rs:.3f}")


def check_grad(d, d_o, L, G, W, n, m, tau32, lam32, seed, step, off, scale_aware):
    """grad_logits against the oracle.  At config scale: the plain bar
    (1e-6 absolute + 1e-5 relative).  In every case also the relative bar:
    1e-5 relative with the absolute term scaled to 1e-6 max|oracle|, plus
    the fp32 rounding allowance of the keys (gpu_helpers)."""
    got = f32(d).reshape(-1)
    if not scale_aware:
        assert_close(got, d_o, "grad_logits")
    kappa = oracle.keys(f32(L).reshape(-1), lam32, seed, step, off).reshape(-1, m)
    sbar = sbar_of(bf16_bits(G), bf16_bits(W)).reshape(-1, m)
    floor = fp32_key_floor(oracle, kappa, sbar, n, tau32, lam32)
    r = assert_close(got, d_o, "grad_logits (relative)", scale_aware=True, floor=floor)
    plain = np.abs(got - d_o) <= 1e-6 * np.abs(d_o).max() + 1e-5 * np.abs(d_o)
    say(f"  grad: err/bound {r:.3f}, {np.count_nonzero(~plain)}/{plain.size} elements "
        f"need the fp32 allowance")


# --------------------------------------------------------------------------- noise
def test_noise_words_and_gumbel_bit_exact(dev):
    import torch
    for seed, step, off, count in [(0, 0, 0, (1 << 20) + 3), (0xDEADBEEF12345678, 7, 1 << 34, 4099),
                                   (1, 2**40 + 3, 6525288448 - 4096, 4096),
                                   (3, 1, 2**34 - 40, 101)]:
        say(f"noise seed={seed} step={step} off={off} count={count}")
        words, g = roi.gumbel_noise(count, seed, step, off, device=dev)
        torch.cuda.synchronize()
        w = words.cpu().numpy().view(np.uint32)
        pick = np.unique(np.r_[np.arange(min(count, 2048)), np.arange(count - 7, count),
                               np.random.default_rng(seed % 1000).integers(0, count, 2000)])
        ref_w = np.array([oracle.philox_word(seed, step, off + int(i)) for i in pick], np.uint32)
        assert np.array_equal(w[pick], ref_w)
        ref_g = oracle.gumbel_from_words(w)
        assert np.array_equal(g.cpu().numpy().view(np.uint32), ref_g.view(np.uint32))


def test_gumbel_exhaustive_uniform_grid(dev):
    """All 2^23 uniforms of the grid (and random full words): bit-exact noise."""
    import torch
    say("gumbel grid 2^23")
    k = np.arange(1 << 23, dtype=np.uint32)
    rnd = np.random.default_rng(5).integers(0, 2**32, 1 << 20, dtype=np.uint64).astype(np.uint32)
    words = np.concatenate([k << np.uint32(9), (k << np.uint32(9)) | np.uint32(0x1FF), rnd])
    t = torch.from_numpy(words.view(np.int32)).to(dev)
    g = roi.gumbel_from_words(t)
    torch.cuda.synchronize()
    ref = oracle.gumbel_from_words(words)
    got = g.cpu().numpy()
    bad = np.flatnonzero(got.view(np.uint32) != ref.view(np.uint32))
    assert bad.size == 0, f"{bad.size} mismatches, first word {words[bad[0]]:#x}: " \
                          f"{got[bad[0]]!r} vs {ref[bad[0]]!r}"


# --------------------------------------------------------------------------- small cases
SMALL = [
    # rows, cols, n, m, tau, lam, seed, step, off
    (1, 4, 2, 4, 1.0, 1.0, 0, 0, 0),
    (37, 36, 2, 4, 1.0, 1.0, 3, 1, 0),           # 333 groups: ragged tail
    (64, 256, 2, 4, 0.5, 1.0, 11, 2, 4096),
    (130, 200, 2, 4, 0.1, 1.0, 5, 9, 8),
    (33, 64, 1, 4, 0.7, 1.0, 1, 0, 0),
    (33, 64, 3, 4, 1.3, 0.6, 2, 3, 12),
    (33, 64, 4, 4, 1.0, 1.0, 2, 3, 0),
    (48, 96, 4, 8, 0.5, 1.0, 7, 4, 0),
    (61, 88, 2, 8, 1.0, 2.0, 8, 5, 8),
    (61, 88, 1, 8, 0.3, 1.0, 8, 5, 8),
    (61, 88, 7, 8, 1.0, 1.0, 8, 5, 8),
    (61, 88, 8, 8, 0.9, 1.0, 9, 6, 0),
    (17, 8, 6, 8, 0.25, 0.5, 4, 2**33, 2**36),
    (23, 56, 5, 8, 2.0, 0.8, 3, 7, 0),           # tau > 1: the exp-domain power by exp2/log2
    # the Philox block index crosses a multiple of 2^32 inside the call
    (40, 64, 2, 4, 1.0, 1.0, 6, 3, 2**34 - 4 * 256),
    (25, 64, 4, 8, 0.5, 1.0, 6, 3, 2**35 - 8 * 100),
    # m = 16 and 32: groups spread over 4 and 8 lanes
    (37, 48, 8, 16, 1.0, 1.0, 2, 0, 0),
    (21, 80, 1, 16, 0.5, 1.0, 3, 7, 32),
    (21, 80, 15, 16, 0.7, 1.0, 3, 7, 16),
    (9, 64, 16, 16, 1.0, 1.0, 3, 1, 0),
    (33, 96, 16, 32, 1.0, 1.0, 4, 2, 0),
    (13, 64, 5, 32, 0.3, 0.8, 5, 3, 64),
    (13, 64, 31, 32, 1.0, 1.0, 5, 3, 32),
    (7, 32, 32, 32, 0.9, 1.0, 6, 4, 0),
    (20, 64, 8, 16, 0.5, 1.0, 7, 8, 2**34 - 16 * 40),
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "x".join(map(str, c[:4])))
def test_small_config_scale(dev, case):
    rows, cols, n, m, tau, lam, seed, step, off = case
    run_case(dev, rows, cols, n, m, tau, lam, seed, step, off, case_seed=rows * 1000 + cols)


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "x".join(map(str, c[:4])))
def test_small_unit_scale(dev, case):
    """Unit-scale W and upstream gradients (grad_logits of order 1/tau): the
    absolute 1e-6 term is scaled by the largest |oracle| value, and each
    element also gets the fp32 rounding allowance of its keys."""
    rows, cols, n, m, tau, lam, seed, step, off = case
    run_case(dev, rows, cols, n, m, tau, lam, seed, step, off, case_seed=7 + rows * cols,
             w_std=1.0, grad_std=1.0, logit_std=2.0, scale_aware=True)


def relaxation_form_logits(rows, cols, m, tau, lam, seed):
    """Logits laid out wave by wave (64 groups): calm groups (small key spans:
    the exp-domain recursion), groups with one key 100 tau / lambda above the
    rest (1 - mu of that key falls below FLT_MIN, so log(1 - mu) is floored),
    groups with two such keys, wide-spread groups, and waves mixing calm and
    dominant groups, which must all take the log-domain recursion together."""
    rng = np.random.default_rng(seed)
    groups = rows * cols // m
    L = rng.normal(0.0, 1.0, size=(groups, m))
    kind = (np.arange(groups) // 64) % 6
    mixed = (kind == 4) & (np.arange(groups) % 2 == 1)
    calm = (kind == 0) | ((kind == 4) & ~mixed)
    L[calm] *= 0.3
    big = 100.0 * tau * lam
    top = rng.integers(0, m, size=groups)
    second = (top + 1 + rng.integers(0, m - 1, size=groups)) % m
    spike = (kind == 1) | (kind == 2) | mixed | (kind == 5)
    L[spike, top[spike]] += big
    two = kind == 2
    L[two, second[two]] += 0.5 * big
    wide = kind == 3
    L[wide] *= 4.0
    return L.reshape(rows, cols).astype(np.float32)


RELAX_FORMS = [
    # rows, cols, n, m, tau, lam: 392 groups = 6 full waves of each kind + a tail
    (49, 32, 2, 4, 1.0, 1.0),
    (49, 32, 2, 4, 0.5, 1.0),
    (49, 32, 2, 4, 0.3, 1.0),
    (49, 32, 1, 4, 1.0, 1.0),
    (49, 32, 3, 4, 0.5, 0.7),
    (49, 64, 4, 8, 0.5, 1.0),
    (49, 64, 2, 8, 1.0, 2.0),
    (49, 64, 6, 8, 0.25, 1.0),
    (49, 128, 8, 16, 1.0, 1.0),
    (49, 256, 16, 32, 1.0, 1.0),
]


@pytest.mark.parametrize("case", RELAX_FORMS, ids=lambda c: "x".join(map(str, c[:5])))
def test_relaxation_forms_and_floor(dev, case):
    """Waves that take the exp-domain recursion, waves that must fall back to
    the log-domain one, and groups that reach the FLT_MIN floor of log(1 - mu)
    (so the backward's floor case runs), in one launch, against the oracle."""
    rows, cols, n, m, tau, lam = case
    logits = relaxation_form_logits(rows, cols, m, tau, lam, seed=rows * cols + n)
    run_case(dev, rows, cols, n, m, tau, lam, 3, 1, 0, case_seed=cols + n, w_std=1.0,
             grad_std=1.0, scale_aware=True, logits=logits)


def test_single_layer_896(dev):
    """One 896x896 linear layer, 2:4, tau = 1, seed 0, step 0: every output."""
    run_case(dev, 896, 896, 2, 4, 1.0, 1.0, 0, 0, 0, case_seed=0)


def test_hardware_noise_bound(dev):
    """The premise of the forward's guarded comparisons and of the backward's
    key error: over all 2^23 uniforms, the hardware-log noise N stays within
    HW_NOISE_MAX (the kernels' margin constant) and within HW_NOISE_A +
    HW_NOISE_B |N| of log2(e) g + log2(ln 2), g the oracle's exact noise."""
    import torch
    say("hardware noise bound, 2^23 uniforms")
    k = np.arange(1 << 23, dtype=np.uint32)
    words = np.concatenate([k << np.uint32(9), (k << np.uint32(9)) | np.uint32(0x1FF)])
    N = roi.fast_noise_from_words(torch.from_numpy(words.view(np.int32)).to(dev))
    torch.cuda.synchronize()
    N = N.cpu().numpy().astype(np.float64)
    g = oracle.gumbel_from_words(words).astype(np.float64)
    err = np.abs(N - (g * LOG2E + LOG2_LN2))
    say(f"  max error {err.max():.3g} (bound {HW_NOISE_MAX})")
    assert err.max() <= HW_NOISE_MAX
    assert np.all(err <= HW_NOISE_A + HW_NOISE_B * np.abs(N))


# --------------------------------------------------------------------------- ties
def test_ties_go_to_lowest_index(dev):
    """Logits equal to minus the noise make every key exactly +0.0: all keys
    tie and the kept entries are the lowest indices, in index order."""
    import torch
    for n, m in ((2, 4), (3, 8), (1, 4), (5, 8), (8, 16), (3, 16), (16, 32), (7, 32)):
        say(f"ties {n}:{m}")
        rows, cols, seed, step = 16, 64, 21, 4
        _, g = roi.gumbel_noise(rows * cols, seed, step, 0, device=dev, want_words=False)
        L = (-g).reshape(rows, cols).contiguous()
        # half of the groups: raise the last two entries so they win, in index order
        L2 = L.clone()
        L2.view(-1, m)[::2, m - 2:] += 1.0
        W = torch.randn(rows, cols, device=dev).to(torch.bfloat16)
        for logits in (L, L2):
            Wm, S, idx = roi.mask_fwd(W, logits, n, m, 1.0, 1.0, seed, step, 0, want_soft=True)
            torch.cuda.synchronize()
            Wm_o, S_o, idx_o = oracle.mask_fwd(bf16_bits(W), f32(logits), n, m, 1.0, 1.0, seed,
                                               step, 0)
            assert np.array_equal(idx.cpu().numpy(), idx_o)
            assert np.array_equal(bf16_bits(Wm).reshape(-1), Wm_o)
            assert_close(f32(S), S_o, "soft mask (ties)")
        idx0 = roi.mask_fwd(W, L, n, m, 1.0, 1.0, seed, step, 0)[2].cpu().numpy()
        assert np.all(idx0 == np.arange(n)[None, :])


NEAR = [(2, 4, 1.0), (1, 4, 1.0), (3, 4, 0.6), (4, 4, 1.0), (4, 8, 1.0), (2, 8, 2.0),
        (7, 8, 1.0), (8, 16, 1.0), (16, 32, 0.7)]


@pytest.mark.parametrize("case", NEAR, ids=lambda c: f"{c[0]}of{c[1]}-lam{c[2]}")
def test_near_ties_bit_exact(dev, case):
    """Logits built from the oracle's noise so that the keys of a group sit at
    exact ties, a few ulp apart, around the forward's comparison margin, and
    far apart: the selections must still be those of the exact keys, with and
    without the soft mask."""
    import torch
    n, m, lam = case
    rows, cols, seed, step, off = 64, 256, 31, 5, 4096
    groups = rows * cols // m
    say(f"near ties {n}:{m} lambda={lam}")
    g = oracle.keys(np.zeros(rows * cols, np.float32), 1.0, seed, step, off).astype(np.float64)
    rng = np.random.default_rng(n * 100 + m)
    base = rng.normal(0.0, 2.0, (groups, 1))
    base[::4] = 0.0  # logits -g (lambda = 1): keys exactly +0.0 where the step is 0
    steps = np.array([0.0, 0.0, 0.0, 1e-7, -1e-7, 4e-7, 2e-6, -2e-6, 1e-5, -1e-5, 2.5e-5, 4e-5,
                      -6e-5, 1e-4, 3e-4, 1.0, -1.0])
    target = base + rng.choice(steps, (groups, m))
    target[1::3] = base[1::3] + rng.normal(0.0, 1.0, (target[1::3].shape))  # well separated
    L = ((target.reshape(-1) - g) * lam).astype(np.float32).reshape(rows, cols)
    lam32 = float(np.float32(lam))
    kappa = oracle.keys(L.reshape(-1), lam32, seed, step, off).reshape(groups, m)
    gaps = np.abs(kappa[:, :, None] - kappa[:, None, :]) + np.eye(m)[None] * 1e30
    closest = gaps.min(axis=(1, 2))
    assert (closest < 5e-5).mean() > 0.5, "inputs not near ties"
    assert lam != 1.0 or (closest == 0).mean() > 0.05, "no exact ties"
    Lt = torch.from_numpy(L).to(dev)
    W = (torch.randn(rows, cols, generator=torch.Generator().manual_seed(m)) + 4.0)
    W = W.to(torch.bfloat16).to(dev)  # nonzero, so a wrong mask shows in W_masked
    Wm_o, S_o, idx_o = oracle.mask_fwd(bf16_bits(W), L, n, m, 0.5, lam32, seed, step, off)
    for want_soft in (False, True):
        Wm, S, idx = roi.mask_fwd(W, Lt, n, m, 0.5, lam, seed, step, off, want_soft=want_soft)
        torch.cuda.synchronize()
        assert np.array_equal(idx.cpu().numpy(), idx_o), f"indices differ (soft={want_soft})"
        assert np.array_equal(bf16_bits(Wm).reshape(-1), Wm_o), f"W_masked differs ({want_soft})"


# --------------------------------------------------------------------------- layout properties
@pytest.mark.parametrize("tau", [1.0, 0.5, 0.4])
def test_split_calls_equal_one_slab_call(dev, tau):
    """Per-tensor calls with cumulative elem_offset give exactly the outputs of
    one call over the back-to-back slab.  Tensor boundaries fall inside waves
    at every m, and the logits mix spreads so that groups of one wave disagree
    on which form of the relaxation their key spans allow: a group's bits must
    not depend on the groups that share its wave."""
    import torch
    shapes = [(128, 96), (33, 96), (32, 96), (128, 96), (200, 96), (96, 224), (7, 96)]
    offs = np.cumsum([0] + [r * c for r, c in shapes])
    total = int(offs[-1])
    gen = torch.Generator(device="cpu")
    gen.manual_seed(3)
    W = (torch.randn(total, generator=gen) * 0.02).to(torch.bfloat16).to(dev)
    spread = torch.where(torch.rand(total // 4, generator=gen) < 0.3, 6.0, 1.0)
    L = (torch.randn(total, generator=gen) * spread.repeat_interleave(4)).to(dev)
    G = (torch.randn(total, generator=gen) * 1e-3).to(torch.bfloat16).to(dev)
    for n, m in ((2, 4), (4, 8), (8, 16), (16, 32)):
        say(f"split vs slab {n}:{m} tau={tau}")
        Wm, S, idx = roi.mask_fwd(W, L, n, m, tau, 1.0, 9, 2, 0, want_soft=True)
        d = roi.mask_bwd(G, W, L, n, m, tau, 1.0, 9, 2, 0)
        for (r, c), o in zip(shapes, offs[:-1]):
            o = int(o)
            sl = slice(o, o + r * c)
            w_t, l_t, g_t = (W[sl].view(r, c), L[sl].view(r, c), G[sl].view(r, c))
            Wm_t, S_t, idx_t = roi.mask_fwd(w_t, l_t, n, m, tau, 1.0, 9, 2, o, want_soft=True)
            d_t = roi.mask_bwd(g_t, w_t, l_t, n, m, tau, 1.0, 9, 2, o)
            torch.cuda.synchronize()
            assert torch.equal(Wm_t.reshape(-1).view(torch.int16), Wm[sl].view(torch.int16))
            assert torch.equal(S_t.reshape(-1).view(torch.int32), S[sl].view(torch.int32)), \
                f"soft mask differs, tensor at {o}"
            assert torch.equal(idx_t, idx[o // m:(o + r * c) // m])
            assert torch.equal(d_t.reshape(-1).view(torch.int32), d[sl].view(torch.int32)), \
                f"grad_logits differs, tensor at {o}"


def grouped_inputs(dev, m, count=40, seed=5):
    """`count` separately allocated tensors of mixed shapes (cols % 32 == 0),
    one of them empty, with stack offsets except one piece placed just below
    a multiple of 2^34 elements, so that its noise crosses the boundary."""
    import torch
    rng = np.random.default_rng(seed)
    shapes = [(int(rng.integers(1, 90)), 32 * int(rng.integers(1, 9))) for _ in range(count)]
    shapes[3] = (0, 64)
    if count > 7:
        shapes[7] = (40, 96)
    gen = torch.Generator(device="cpu").manual_seed(seed)
    tensors, offsets, off = [], [], 0
    for i, (r, c) in enumerate(shapes):
        W = (torch.randn(r, c, generator=gen) * 0.02).to(torch.bfloat16).to(dev)
        L = torch.randn(r, c, generator=gen).to(dev)
        G = (torch.randn(r, c, generator=gen) * 1e-3).to(torch.bfloat16).to(dev)
        tensors.append((W, L, G))
        if i == 7:
            off = (1 << 34) - 32 * ((r * c // 2) // 32)
        offsets.append(off)
        off += r * c
    return tensors, offsets


@pytest.mark.parametrize("n,m", [(2, 4), (4, 8), (8, 16), (16, 32)])
def test_grouped_equals_single_calls(dev, n, m):
    """The grouped calls over separately allocated tensors give, bit for bit,
    the outputs of one single-tensor call per tensor (forward with and
    without S and indices, soft forward with them and alone, backward)."""
    import torch
    say(f"grouped vs single {n}:{m}")
    tensors, offs = grouped_inputs(dev, m)
    args = (n, m, 0.7, 1.0, 13, 4)
    for soft, want_soft, want_idx in ((False, False, True), (False, True, True),
                                      (False, False, False), (True, True, True),
                                      (True, False, False)):
        outs = roi.mask_fwd_grouped([(W, L) for W, L, _ in tensors], *args, offsets=offs,
                                    want_soft=want_soft, want_idx=want_idx, soft_forward=soft)
        for (W, L, _), off, (Wm, S, idx) in zip(tensors, offs, outs):
            Wm1, S1, idx1 = roi.mask_fwd(W, L, *args, elem_offset=off, want_soft=want_soft,
                                         want_idx=want_idx, soft_forward=soft)
            torch.cuda.synchronize()
            assert torch.equal(Wm.view(torch.int16), Wm1.view(torch.int16))
            if want_soft:
                assert torch.equal(S.view(torch.int32), S1.view(torch.int32))
            if want_idx:
                assert torch.equal(idx, idx1)
    ds = roi.mask_bwd_grouped([(G, W, L) for W, L, G in tensors], *args, offsets=offs)
    for (W, L, G), off, d in zip(tensors, offs, ds):
        d1 = roi.mask_bwd(G, W, L, *args, elem_offset=off)
        torch.cuda.synchronize()
        assert torch.equal(d.view(torch.int32), d1.view(torch.int32))


def test_grouped_against_oracle(dev):
    """A grouped call over separate tensors against the oracle, tensor by tensor."""
    import torch
    say("grouped vs oracle 2:4")
    tensors, offs = grouped_inputs(dev, 4, count=6, seed=9)
    n, m, tau, lam, seed, step = 2, 4, 0.5, 1.0, 3, 2
    outs = roi.mask_fwd_grouped([(W, L) for W, L, _ in tensors], n, m, tau, lam, seed, step,
                                offsets=offs, want_soft=True)
    ds = roi.mask_bwd_grouped([(G, W, L) for W, L, G in tensors], n, m, tau, lam, seed, step,
                              offsets=offs)
    torch.cuda.synchronize()
    for (W, L, G), off, (Wm, S, idx), d in zip(tensors, offs, outs, ds):
        Wm_o, S_o, idx_o = oracle.mask_fwd(bf16_bits(W), f32(L), n, m, tau, lam, seed, step, off)
        d_o = oracle.mask_bwd(bf16_bits(G), bf16_bits(W), f32(L), n, m, tau, lam, seed, step, off)
        assert np.array_equal(idx.cpu().numpy(), idx_o)
        assert np.array_equal(bf16_bits(Wm).reshape(-1), Wm_o)
        assert_close(f32(S), S_o, "soft mask (grouped)")
        assert_close(f32(d), d_o, "grad_logits (grouped)")


# --------------------------------------------------------------------------- fused AdamW
ADAMW = [(37, 36, 2, 4, 1.0, 1.0, 1, 1e-3), (64, 96, 2, 4, 0.1, 1.0, 7, 4e-4),
         (33, 64, 3, 4, 0.7, 0.6, 3, 1e-3), (61, 88, 4, 8, 0.5, 1.0, 2, 1e-3),
         (37, 48, 8, 16, 1.0, 1.0, 1, 1e-3), (13, 64, 5, 32, 0.3, 0.8, 12, 2e-4),
         (29, 40, 7, 8, 0.4, 1.7, 5, 1e-3)]


def adamw_state(rows, cols, seed):
    rng = np.random.default_rng(seed)
    m = rng.normal(0.0, 2e-5, (rows, cols)).astype(np.float32)
    v = (rng.random((rows, cols)) * 1e-9).astype(np.float32)
    return m, v


def adamw_rounding_check(got_p, got_m, got_v, g, phi0, m0, v0, hp, t, what):
    """The fused step's moments and logits against the oracle's AdamW applied
    to the kernel's own fp32 gradient g, so that only the step's fp32
    arithmetic is measured: each moment within a few units of rounding of its
    two terms (fp32 products and a fused multiply-add), and the logit within
    2 ulp plus 2e-6 of the update (approximate reciprocal and square root)."""
    lr, b1, b2, eps, wd = hp
    g = np.asarray(g, dtype=np.float64).reshape(-1)
    m0 = np.asarray(m0, dtype=np.float64).reshape(-1)
    v0 = np.asarray(v0, dtype=np.float64).reshape(-1)
    p_r, m_r, v_r = oracle.adamw(g, phi0, m0.astype(np.float32), v0.astype(np.float32), *hp, t)
    u = 2.0 ** -24
    tol_m = 4 * u * (b1 * np.abs(m0) + (1 - b1) * np.abs(g)) + 2 * u * np.abs(m_r)
    tol_v = 4 * u * (b2 * np.abs(v0) + (1 - b2) * g * g) + 2 * u * np.abs(v_r)
    for got, ref, tol, name in ((got_m, m_r, tol_m, "exp_avg"), (got_v, v_r, tol_v, "exp_avg_sq")):
        err = np.abs(np.asarray(got, dtype=np.float64).reshape(-1) - ref.reshape(-1))
        assert np.all(err <= tol), f"{what}: {name} off by {float((err - tol).max()):.3g}"
    decayed = np.asarray(phi0, dtype=np.float64).reshape(-1) * (1.0 - lr * wd)
    upd = p_r.reshape(-1) - decayed
    gp = np.asarray(got_p, dtype=np.float64).reshape(-1)
    # the moments' own rounding carried into the update -s m' / (sqrt(v' / bc2) + eps)
    step_size = lr / (1.0 - b1 ** t)
    den = np.sqrt(v_r.reshape(-1) / (1.0 - b2 ** t)) + eps
    carried = step_size * tol_m.reshape(-1) / den + \
        np.abs(upd) * tol_v.reshape(-1) / np.maximum(2.0 * v_r.reshape(-1), 1e-300)
    tol_p = 2 * np.spacing(np.abs(gp.astype(np.float32))).astype(np.float64) + \
        2e-6 * np.abs(upd) + carried
    err = np.abs(gp - p_r.reshape(-1))
    assert np.all(err <= tol_p), f"{what}: logits off by {float((err - tol_p).max()):.3g}"
    return tol_p


@pytest.mark.parametrize("scale", ["config", "unit"])
@pytest.mark.parametrize("case", ADAMW, ids=lambda c: "x".join(map(str, c[:4])) + f"-t{c[6]}")
def test_bwd_adamw_against_oracle(dev, case, scale):
    """The fused backward + AdamW step against the oracle's backward followed by
    its AdamW step; the gradient it also writes equals roi_mask_bwd's bit for
    bit.  At config scale (and with unit-scale W and upstream gradients, where
    the gradient is held to the relative bar with its fp32 allowance)."""
    import torch
    rows, cols, n, m, tau, lam, t, lr = case
    seed, step, off = 17, 3, 64
    unit = scale == "unit"
    say(f"bwd+adamw {rows}x{cols} {n}:{m} tau={tau} lam={lam} t={t} lr={lr} {scale} scale")
    if unit:
        W, L, G = wl.small_case(rows, cols, rows + cols + 1, device=dev, w_std=1.0, grad_std=1.0,
                                logit_std=2.0)
    else:
        W, L, G = wl.small_case(rows, cols, rows + cols, device=dev)
    m0, v0 = adamw_state(rows, cols, t)
    if unit:  # moments of the size a unit-scale gradient builds up
        m0, v0 = (m0 * 5e3).astype(np.float32), (v0 * 1e7).astype(np.float32)
    opt = roi.adamw_params(lr, t=t)
    Lg, mg, vg = L.clone(), torch.from_numpy(m0).to(dev), torch.from_numpy(v0).to(dev)
    d = torch.empty_like(L)
    roi.mask_bwd_adamw(G, W, Lg, mg, vg, n, m, tau, lam, seed, step, off, opt=opt, grad_out=d)
    d_ref = roi.mask_bwd(G, W, L, n, m, tau, lam, seed, step, off)
    torch.cuda.synchronize()
    assert torch.equal(d.view(torch.int32), d_ref.view(torch.int32))
    tau32, lam32 = float(np.float32(tau)), float(np.float32(lam))
    d_o = oracle.mask_bwd(bf16_bits(G), bf16_bits(W), f32(L), n, m, tau32, lam32, seed, step, off)
    check_grad(d, d_o, L, G, W, n, m, tau32, lam32, seed, step, off, scale_aware=unit)
    hp = [float(np.float32(x)) for x in (lr, 0.9, 0.95, 1e-8, 0.05)]
    # the step's own arithmetic, from the kernel's gradient
    tol_p = adamw_rounding_check(f32(Lg), f32(mg), f32(vg), f32(d), f32(L), m0, v0, hp, t,
                                 "fused AdamW")
    # The check is tight enough to see a wrong step: without the bias
    # corrections (t = 1) most logits fall outside it.
    if t > 1:
        p_nb, _, _ = oracle.adamw(f32(d).astype(np.float64), f32(L), m0, v0, *hp, 1)
        wrong = np.abs(f32(Lg).astype(np.float64).reshape(-1) - p_nb.reshape(-1)) > tol_p
        assert wrong.mean() > 0.5
    # and the logits against the oracle's own backward + AdamW: the gradient's
    # tolerance carried through the step (first order, from the oracle)
    p_o, _, _ = oracle.adamw(d_o, f32(L), m0, v0, *hp, t)
    got_d = f32(d).astype(np.float64).reshape(-1)
    p_g, _, _ = oracle.adamw(got_d, f32(L), m0, v0, *hp, t)
    moved = np.abs(p_g.reshape(-1) - p_o.reshape(-1))  # what the gradient difference moves
    assert np.all(np.abs(f32(Lg).astype(np.float64).reshape(-1) - p_o.reshape(-1))
                  <= moved + tol_p), "logits after AdamW"


def test_full_bwd_adamw_7b_stack(dev):
    """The fused backward + AdamW over the whole 7B stack in one call, as
    `bench.py --mode adamw` runs it (step 3 of the annealing: tau, the
    learning rate and AdamW's step count t = 4).  Sampled groups of the
    gradient, both moments and the updated logits against the oracle's
    backward followed by its AdamW step."""
    import torch
    name, n, m, step = "qwen2.5-7b-stack-2:4", 2, 4, 3
    work = wl.WORKLOADS[name]
    say(f"full bwd+adamw {name}: allocating {work.numel} weights and moments")
    W, L, G = wl.fill_slab(work, dev, step=step)
    gen = torch.Generator(device=dev).manual_seed(99)
    mom = torch.empty_like(L).normal_(0.0, 2e-5, generator=gen)
    sec = torch.empty_like(L).uniform_(0.0, 1e-9, generator=gen)
    tau = roi.anneal(1.0, 0.1, step, 9)
    lr = roi.anneal(1e-3, 1e-4, step, 9)
    ng = work.numel // m
    picks = sample_groups(work, ng, m, np.random.default_rng(777), 20000)
    pt = torch.from_numpy(picks).to(dev)
    take = lambda t: t.view(-1, m).index_select(0, pt)
    L0, m0, v0 = f32(take(L)), f32(take(mom)), f32(take(sec))
    d = torch.empty_like(L)
    roi.mask_bwd_adamw(G, W, L, mom, sec, n, m, tau, 1.0, 0, step, 0,
                       opt=roi.adamw_params(lr, t=step + 1), grad_out=d)
    torch.cuda.synchronize()
    say(f"  comparing {picks.size} sampled groups with the oracle")
    ge = picks.astype(np.uint64) * np.uint64(m)
    d_o = oracle.mask_bwd_groups(bf16_bits(take(G)), bf16_bits(take(W)), L0, ge, n, m,
                                 float(np.float32(tau)), 1.0, 0, step)
    hp = [float(np.float32(x)) for x in (lr, 0.9, 0.95, 1e-8, 0.05)]
    p_o, m_o, v_o = oracle.adamw(d_o, L0, m0, v0, *hp, step + 1)
    assert_close(f32(take(d)), d_o, "grad_logits (fused, full stack)")
    adamw_rounding_check(f32(take(L)), f32(take(mom)), f32(take(sec)), f32(take(d)), L0, m0, v0,
                         hp, step + 1, "fused AdamW (full stack)")
    assert_close(f32(take(L)), p_o, "logits after AdamW (full stack)")
    del W, L, G, mom, sec, d
    torch.cuda.empty_cache()


def test_bwd_adamw_three_steps(dev):
    """Three training steps (forward, fused backward + AdamW) with the
    temperatures and the learning rate annealed: the GPU state against the
    oracle carrying its own state, rounded to fp32 after each step."""
    import torch
    rows, cols, n, m = 96, 128, 2, 4
    W, L, _ = wl.small_case(rows, cols, 5, device=dev)
    Lg = L.clone()
    mg = torch.zeros_like(L)
    vg = torch.zeros_like(L)
    p_o = f32(L)
    m_o = np.zeros_like(p_o)
    v_o = np.zeros_like(p_o)
    gen = torch.Generator(device="cpu").manual_seed(8)
    for t in range(1, 4):
        tau = roi.anneal(1.0, 0.05, t - 1, 3)
        lam = roi.anneal(1.0, 0.5, t - 1, 3)
        lr = roi.anneal(1e-3, 1e-4, t - 1, 3)
        say(f"adamw chain t={t} tau={tau:.4f} lam={lam:.4f} lr={lr:.2e}")
        G = (torch.randn(rows, cols, generator=gen) * 1e-3).to(torch.bfloat16).to(dev)
        before = [f32(x) for x in (Lg, mg, vg)]
        d = torch.empty_like(Lg)
        roi.mask_bwd_adamw(G, W, Lg, mg, vg, n, m, tau, lam, 0, t, 0,
                           opt=roi.adamw_params(lr, t=t), grad_out=d)
        torch.cuda.synchronize()
        hp = [float(np.float32(x)) for x in (lr, 0.9, 0.95, 1e-8, 0.05)]
        # this step's arithmetic from the GPU's own state and gradient
        adamw_rounding_check(f32(Lg), f32(mg), f32(vg), f32(d), *before, hp, t,
                             f"AdamW step {t}")
        # the gradient at the GPU's logits, then the chain against the oracle
        # carrying its own state
        assert_close(f32(d), oracle.mask_bwd(bf16_bits(G), bf16_bits(W), before[0], n, m, tau,
                                             lam, 0, t, 0), f"grad_logits at step {t}")
        d_o = oracle.mask_bwd(bf16_bits(G), bf16_bits(W), p_o, n, m, tau, lam, 0, t, 0)
        p64, m64, v64 = oracle.adamw(d_o, p_o, m_o, v_o, *hp, t)
        assert_close(f32(Lg), p64, f"logits after step {t}")
        tol_g = 1e-6 + 1e-5 * np.abs(d_o)
        assert np.all(np.abs(f32(mg).reshape(-1) - m64) <= (1 - hp[1]) * tol_g + 1e-7 * np.abs(m64)
                      + 2 * np.abs(before[1].reshape(-1) - m_o.reshape(-1))), f"exp_avg, step {t}"
        assert np.all(np.abs(f32(vg).reshape(-1) - v64) <=
                      (1 - hp[2]) * (2 * np.abs(d_o) + tol_g) * tol_g + 1e-7 * v64
                      + 2 * np.abs(before[2].reshape(-1) - v_o.reshape(-1))), f"exp_avg_sq, step {t}"
        p_o, m_o, v_o = (x.astype(np.float32) for x in (p64, m64, v64))


def test_bwd_adamw_grouped_equals_single(dev):
    import torch
    say("bwd+adamw grouped vs single")
    tensors, offs = grouped_inputs(dev, 4, count=36, seed=21)
    opt = roi.adamw_params(1e-3, t=4)
    states = []
    for W, L, G in tensors:
        m0, v0 = adamw_state(W.shape[0], W.shape[1], W.numel())
        states.append((torch.from_numpy(m0).to(dev), torch.from_numpy(v0).to(dev)))
    grouped_state = [(L.clone(), mm.clone(), vv.clone()) for (_, L, _), (mm, vv) in
                     zip(tensors, states)]
    roi.mask_bwd_adamw_grouped([(G, W, p, mm, vv) for (W, _, G), (p, mm, vv) in
                                zip(tensors, grouped_state)], 2, 4, 0.5, 1.0, 9, 2,
                               offsets=offs, opt=opt)
    for (W, L, G), off, (mm, vv), (pg, mgr, vgr) in zip(tensors, offs, states, grouped_state):
        p1, m1, v1 = L.clone(), mm.clone(), vv.clone()
        roi.mask_bwd_adamw(G, W, p1, m1, v1, 2, 4, 0.5, 1.0, 9, 2, off, opt=opt)
        torch.cuda.synchronize()
        for a, b in ((pg, p1), (mgr, m1), (vgr, v1)):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32))


# --------------------------------------------------------------------------- final-mask export
EXPORT = [(37, 36, 2, 4), (5, 12, 2, 4), (64, 256, 2, 4), (33, 64, 1, 4), (33, 64, 3, 4),
          (21, 64, 4, 4), (61, 88, 4, 8), (61, 88, 2, 8), (61, 88, 7, 8), (37, 48, 8, 16),
          (21, 80, 1, 16), (13, 64, 5, 32), (7, 32, 31, 32), (9, 64, 16, 32)]


@pytest.mark.parametrize("case", EXPORT, ids=lambda c: "x".join(map(str, c)))
def test_export_bit_exact(dev, case):
    """The final mask (top-n of the logits) in every form, bit for bit against
    the oracle, with many exact ties; the 2:4 metadata over group counts that
    leave a partial last word."""
    import torch
    rows, cols, n, m = case
    say(f"export {rows}x{cols} {n}:{m}")
    W, L, _ = wl.small_case(rows, cols, rows * cols + n, device=dev)
    L = L.clone()
    L.view(-1, m)[::3] = torch.round(L.view(-1, m)[::3] * 2) / 2  # exact ties
    meta = n == 2 and m == 4
    Wm, vals, idx, mt = roi.mask_export(L, W, n, m, want_meta=meta)
    _, _, idx_only, mt_only = roi.mask_export(L, None, n, m, want_dense=False, want_values=False,
                                              want_meta=meta)
    torch.cuda.synchronize()
    Wm_o, vals_o, idx_o, mt_o = oracle.export(f32(L), bf16_bits(W), n, m, want_meta=meta)
    assert np.array_equal(bf16_bits(Wm).reshape(-1), Wm_o)
    assert np.array_equal(bf16_bits(vals), vals_o)
    assert np.array_equal(idx.cpu().numpy(), idx_o)
    assert np.array_equal(idx_only.cpu().numpy(), idx_o)
    if meta:
        assert np.array_equal(mt.cpu().numpy().view(np.uint32), mt_o)
        assert np.array_equal(mt_only.cpu().numpy().view(np.uint32), mt_o)


def test_export_full_7b_stack(dev):
    """The 7B-class stack at 2:4 in one call: sampled groups against the oracle,
    and on every group the metadata equals the indices and the compressed
    values equal the dense mask."""
    import torch
    work = wl.WORKLOADS["qwen2.5-7b-stack-2:4"]
    say(f"export full stack: {work.numel} weights")
    W, L, G = wl.fill_slab(work, dev)
    del G
    Wm, vals, idx, mt = roi.mask_export(L, W, 2, 4, want_meta=True)
    torch.cuda.synchronize()
    ng = work.numel // 4
    chunk = 1 << 26
    for g0 in range(0, ng, chunk):
        g1 = min(ng, g0 + chunk)
        ii = idx[g0:g1].long()
        assert bool((ii[:, 0] < ii[:, 1]).all())
        words = mt[g0 // 8:(g1 + 7) // 8].view(torch.int32)
        q = torch.arange(g0, g1, device=dev)
        nib = (words[(q - g0) // 8] >> (4 * (q % 8))) & 0xF
        assert torch.equal(nib & 3, ii[:, 0]) and torch.equal(nib >> 2, ii[:, 1])
        dense = torch.zeros((g1 - g0, 4), dtype=torch.int16, device=dev)
        dense.scatter_(1, ii, vals[g0:g1].view(torch.int16))
        assert torch.equal(dense, Wm[g0 * 4:g1 * 4].view(-1, 4).view(torch.int16))
        del ii, words, q, nib, dense
    picks = sample_groups(work, ng, 4, np.random.default_rng(77), 30000)
    pt = torch.from_numpy(picks).to(dev)
    take = lambda t: t.view(-1, 4).index_select(0, pt)
    _, vals_o, idx_o, _ = oracle.export(f32(take(L)), bf16_bits(take(W)), 2, 4)
    assert np.array_equal(idx.index_select(0, pt).cpu().numpy(), idx_o)
    assert np.array_equal(bf16_bits(vals.index_select(0, pt)), vals_o)
    del W, L, Wm, vals, idx, mt
    torch.cuda.empty_cache()


SPARSE_MM = [(16, 64, 16), (64, 256, 32), (48, 640, 48), (128, 3584, 32)]


@pytest.mark.parametrize("case", SPARSE_MM, ids=lambda c: "x".join(map(str, c)))
def test_export_feeds_sparse_mfma(dev, case):
    """The 2:4 export read as written by gfx950's sparse matrix core
    (v_smfmac_f32_16x16x64_bf16): W_sparse X^T from the compressed values and
    metadata equals the oracle's masked dense weights times X^T exactly
    (small-integer values, so every fp32 sum is exact)."""
    import torch
    from tests import sparse_mfma
    rows, cols, tokens = case
    say(f"export -> sparse MFMA: W {rows}x{cols}, X {tokens}x{cols}")
    rng = np.random.default_rng(rows * cols + tokens)
    Wi = rng.integers(-8, 9, size=(rows, cols)).astype(np.float32)
    Xi = rng.integers(-8, 9, size=(tokens, cols)).astype(np.float32)
    W = torch.from_numpy(Wi).to(dev).to(torch.bfloat16)
    X = torch.from_numpy(Xi).to(dev).to(torch.bfloat16)
    L = torch.from_numpy(rng.standard_normal((rows, cols)).astype(np.float32)).to(dev)
    _, vals, _, meta = roi.mask_export(L, W, 2, 4, want_dense=False, want_idx=False,
                                       want_meta=True)
    Y = sparse_mfma.matmul_2of4(vals, meta, X, rows, cols)
    torch.cuda.synchronize()
    Wm_o, _, _, _ = oracle.export(f32(L), bf16_bits(W), 2, 4)
    Wd = (Wm_o.astype(np.uint32) << 16).view(np.float32).reshape(rows, cols).astype(np.float64)
    ref = Wd @ Xi.astype(np.float64).T
    assert np.array_equal(Y.cpu().numpy().astype(np.float64), ref)


# --------------------------------------------------------------------------- categorical sampler
CAT = [(37, 36, 2, 4, 1.0, 1.0, 0), (64, 96, 2, 4, 0.3, 0.6, 5), (33, 64, 1, 4, 0.7, 1.0, 3),
       (33, 64, 3, 4, 1.3, 1.0, 1), (21, 64, 4, 4, 1.0, 1.0, 0), (61, 88, 2, 8, 0.5, 1.0, 7),
       (61, 88, 4, 8, 1.0, 2.0, 2 ** 33 + 5), (25, 64, 1, 8, 0.4, 1.0, 11),
       (25, 64, 7, 8, 1.0, 1.0, 0), (19, 96, 3, 8, 0.8, 1.0, 2 ** 40),
       # 8 candidates over several full 256-group chunks and a ragged one
       (70, 64, 1, 8, 0.6, 1.0, 9), (67, 48, 7, 8, 1.0, 0.8, 2 ** 32 - 100)]


def cat_fp32_floor(alpha, G_bits, W_bits, n, m, tau, lam, seed, step, goff):
    """fp32 rounding allowance of the categorical gradient (as fp32_key_floor
    for the item sampler): FP32_FLOOR_FACTOR times the first-order change of
    the fp64 softmax derivative y (ybar - <y, ybar>) / (tau lambda) when each
    fp32 key moves by one ulp.  The keys are the oracle's (candidate c of group
    Q has the noise of element 4 ceil(C / 4) Q + c)."""
    from tests.gpu_helpers import FP32_FLOOR_FACTOR
    A = np.asarray(alpha, dtype=np.float32)
    groups, C = A.shape
    B = (C + 3) // 4
    kappa = np.stack([oracle.keys(A[q], lam, seed, step, 4 * B * (goff + q))
                      for q in range(groups)]).astype(np.float32)
    masks = oracle.cat_candidates(n, m)
    member = ((masks[:, None] >> np.arange(m)[None, :]) & 1).astype(np.float64)  # [C, m]
    ybar = sbar_of(G_bits, W_bits).reshape(groups, m) @ member.T

    def grad(k):
        z = k / tau
        y = np.exp(z - z.max(axis=1, keepdims=True))
        y /= y.sum(axis=1, keepdims=True)
        return y * (ybar - (y * ybar).sum(axis=1, keepdims=True)) / (tau * lam)

    k64 = kappa.astype(np.float64)
    base = grad(k64)
    ulp = np.spacing(np.abs(kappa)).astype(np.float64)
    floor = np.zeros_like(base)
    for c in range(C):
        kp = k64.copy()
        kp[:, c] += ulp[:, c]
        floor += np.abs(grad(kp) - base)
    return FP32_FLOOR_FACTOR * floor


@pytest.mark.parametrize("scale", ["config", "unit"])
@pytest.mark.parametrize("case", CAT, ids=lambda c: "x".join(map(str, c[:4])))
def test_cat_sampler_against_oracle(dev, case, scale):
    """The categorical sampler: chosen candidates and masked weights bit-exact
    (with and without the soft mask), S and dL/dalpha within the float
    tolerance, against the oracle; large group offsets exercise Philox block
    indices above 2^32.  With unit-scale W and upstream gradients the gradient
    is also held to the relative bar with its fp32 allowance."""
    import torch
    rows, cols, n, m, tau, lam, goff = case
    C = roi.cat_num_candidates(n, m)
    unit = scale == "unit"
    say(f"cat {rows}x{cols} {n}:{m} C={C} tau={tau} lam={lam} goff={goff} {scale} scale")
    if unit:
        W, _, G = wl.small_case(rows, cols, rows + 3 * cols + n + 1, w_std=1.0, grad_std=1.0)
    else:
        W, _, G = wl.small_case(rows, cols, rows + 3 * cols + n)
    gen = torch.Generator(device="cpu").manual_seed(n * 100 + m)
    A = torch.randn(rows * cols // m, C, generator=gen) * (2.0 if unit else 1.0)
    W, G, A = W.to(dev), G.to(dev), A.to(dev)
    Wm, S, ch = roi.cat_mask_fwd(W, A, n, m, tau, lam, 9, 4, goff, want_soft=True)
    Wm2, _, ch2 = roi.cat_mask_fwd(W, A, n, m, tau, lam, 9, 4, goff)
    d = roi.cat_mask_bwd(G, W, A, n, m, tau, lam, 9, 4, goff)
    torch.cuda.synchronize()
    tau32, lam32 = float(np.float32(tau)), float(np.float32(lam))
    Wm_o, S_o, ch_o = oracle.cat_fwd(bf16_bits(W), f32(A), n, m, tau32, lam32, 9, 4, goff)
    d_o = oracle.cat_bwd(bf16_bits(G), bf16_bits(W), f32(A), n, m, tau32, lam32, 9, 4, goff)
    for a_, b_ in ((ch, ch2), (Wm, Wm2)):
        assert torch.equal(a_, b_)
    assert np.array_equal(ch.cpu().numpy(), ch_o), "chosen candidates differ"
    assert np.array_equal(bf16_bits(Wm).reshape(-1), Wm_o), "masked weights differ"
    assert_close(f32(S), S_o, "categorical soft mask")
    if not unit:
        assert_close(f32(d), d_o, "dL/dalpha")
    floor = cat_fp32_floor(f32(A), bf16_bits(G), bf16_bits(W), n, m, tau32, lam32, 9, 4, goff)
    r = assert_close(f32(d), d_o, "dL/dalpha (relative)", scale_aware=True, floor=floor)
    say(f"  dL/dalpha err/bound {r:.3f}")


def test_full_cat_7b_stack_2of4(dev):
    """The categorical sampler over the whole 7B stack at 2:4 in one call per
    direction, as `bench.py --mode cat` runs it (6 candidates per group; the
    backward staged through its LDS tile).  40 windows of 300 consecutive
    groups at random, unaligned places (so they cut across the tiles) against
    the oracle: choices and masked weights bit for bit, dL/dalpha within the
    tolerance."""
    import torch
    name, n, m, tau = "qwen2.5-7b-stack-2:4", 2, 4, 1.0
    work = wl.WORKLOADS[name]
    C = roi.cat_num_candidates(n, m)
    ng = work.numel // m
    say(f"full categorical {name}: allocating {work.numel} weights, {ng} x {C} logits")
    W, L, G = wl.fill_slab(work, dev)
    del L
    A = torch.empty((ng, C), dtype=torch.float32, device=dev)
    A.normal_(0.0, 1.0, generator=torch.Generator(device=dev).manual_seed(2468))
    Wm, _, ch = roi.cat_mask_fwd(W, A, n, m, tau, 1.0, 5, 2, 0)
    d = roi.cat_mask_bwd(G, W, A, n, m, tau, 1.0, 5, 2, 0)
    torch.cuda.synchronize()
    rng = np.random.default_rng(13579)
    starts = np.concatenate([[0, ng - 300], rng.integers(0, ng - 300, 38)])
    for g0 in starts.tolist():
        sl = slice(g0 * m, (g0 + 300) * m)
        Wm_o, _, ch_o = oracle.cat_fwd(bf16_bits(W[sl]), f32(A[g0:g0 + 300]), n, m, tau, 1.0, 5,
                                       2, g0, want_soft=False)
        d_o = oracle.cat_bwd(bf16_bits(G[sl]), bf16_bits(W[sl]), f32(A[g0:g0 + 300]), n, m, tau,
                             1.0, 5, 2, g0)
        assert np.array_equal(ch[g0:g0 + 300].cpu().numpy(), ch_o), f"choices differ at {g0}"
        assert np.array_equal(bf16_bits(Wm[sl]).reshape(-1), Wm_o), f"masked weights differ at {g0}"
        assert_close(f32(d[g0:g0 + 300]), d_o, f"dL/dalpha at group {g0}")
    del W, G, A, Wm, ch, d
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n,m", [(2, 4), (4, 8), (2, 8)])
def test_cat_ties_and_near_ties(dev, n, m):
    """Logits built from the oracle's noise so that candidate keys tie exactly
    or nearly: the choice must still be the exact keys' (lowest candidate on a
    tie), with the fast comparison's fallback exercised."""
    import torch
    rows, cols = 32, 64
    Gn = rows * cols // m
    C = roi.cat_num_candidates(n, m)
    B = (C + 3) // 4
    say(f"cat near ties {n}:{m}")
    # noise of every candidate: element 4 B Q + c
    Q = np.arange(Gn, dtype=np.uint64)
    elems = (4 * B * Q[:, None] + np.arange(C, dtype=np.uint64)[None, :]).reshape(-1)
    g = np.array([oracle.keys(np.zeros(1, np.float32), 1.0, 3, 6, int(e))[0] for e in elems],
                 dtype=np.float64).reshape(Gn, C)
    rng = np.random.default_rng(C)
    steps = np.array([0.0, 0.0, 1e-7, -3e-7, 2e-6, 1.5e-5, -2.5e-5, 4e-5, 1e-3, 1.0])
    target = rng.normal(0, 1, (Gn, 1)) + rng.choice(steps, (Gn, C))
    target[::4] = rng.choice(steps, (Gn, C))[::4]           # around 0: exact ties when step 0
    A = (target - g).astype(np.float32)
    A[::4][target[::4] == 0.0] = (-g[::4][target[::4] == 0.0]).astype(np.float32)
    W = (torch.randn(rows, cols, generator=torch.Generator().manual_seed(1)) + 3).to(torch.bfloat16)
    W, At = W.to(dev), torch.from_numpy(A).to(dev)
    Wm, _, ch = roi.cat_mask_fwd(W, At, n, m, 1.0, 1.0, 3, 6, 0)
    Wm_s, _, ch_s = roi.cat_mask_fwd(W, At, n, m, 1.0, 1.0, 3, 6, 0, want_soft=True)
    torch.cuda.synchronize()
    Wm_o, _, ch_o = oracle.cat_fwd(bf16_bits(W), A, n, m, 1.0, 1.0, 3, 6, 0, want_soft=False)
    assert np.array_equal(ch.cpu().numpy(), ch_o) and np.array_equal(ch_s.cpu().numpy(), ch_o)
    assert np.array_equal(bf16_bits(Wm).reshape(-1), Wm_o)
    assert np.array_equal(bf16_bits(Wm_s).reshape(-1), Wm_o)


def test_every_output_written_and_deterministic(dev):
    import torch
    W, L, G = wl.small_case(333, 64, 1, device=dev)
    for n, m in ((2, 4), (3, 8), (8, 16), (16, 32)):
        say(f"sentinel/determinism {n}:{m}")
        outs = []
        for _ in range(2):
            Wm = torch.full_like(W, float("nan"))
            S = torch.full_like(L, float("nan"))
            idx = torch.full((W.numel() // m, n), 255, dtype=torch.uint8, device=dev)
            d = torch.full_like(L, float("nan"))
            roi.mask_fwd(W, L, n, m, 0.8, 1.0, 4, 4, 0, want_soft=True,
                         out={"W_masked": Wm, "soft_mask": S, "sel_idx": idx})
            roi.mask_bwd(G, W, L, n, m, 0.8, 1.0, 4, 4, 0, out=d)
            torch.cuda.synchronize()
            assert not torch.isnan(Wm.float()).any() and not torch.isnan(S).any()
            assert not torch.isnan(d).any() and bool((idx < m).all())
            outs.append((Wm.view(torch.int16).clone(), S.view(torch.int32).clone(), idx.clone(),
                         d.view(torch.int32).clone()))
        for a, b in zip(*outs):
            assert torch.equal(a, b)


def test_empty_and_invalid_on_device(dev):
    import torch
    W = torch.empty(0, 8, dtype=torch.bfloat16, device=dev)
    L = torch.empty(0, 8, dtype=torch.float32, device=dev)
    Wm, S, idx = roi.mask_fwd(W, L, 2, 4, want_soft=True)
    assert Wm.numel() == 0 and idx.numel() == 0
    W = torch.zeros(4, 6, dtype=torch.bfloat16, device=dev)
    L = torch.zeros(4, 6, dtype=torch.float32, device=dev)
    with pytest.raises(roi.RoiError):
        roi.mask_fwd(W, L, 2, 4)
    with pytest.raises(roi.RoiError):
        roi.mask_fwd(W[:, :4].contiguous(), L[:, :4].contiguous(), 2, 4, tau=0.0, want_soft=True)


# --------------------------------------------------------------------------- full-size workloads
def sample_groups(workload, ngroups, m, rng, count):
    """Random groups plus the first and last group of every tensor."""
    edges = []
    for t in workload.tensors:
        g0 = t.offset // m
        g1 = (t.offset + t.numel) // m - 1
        edges += [g0, g1]
    picks = np.concatenate([rng.integers(0, ngroups, count), np.array(edges), [0, ngroups - 1]])
    return np.unique(picks)


def check_grad_whole(got, ref, kappa_of, sbar_of_groups, n, m, tau32, what):
    """Every element: the plain bar (1e-6 absolute + 1e-5 relative), then the
    relative bar (absolute term 1e-6 max|oracle|) with the fp32 allowance of
    the keys, which is computed only for the groups that need it."""
    from tests.gpu_helpers import ATOL, RTOL
    r = assert_close(got, ref, what)
    bound = ATOL * np.abs(ref).max() + RTOL * np.abs(ref)
    need = np.flatnonzero((np.abs(got - ref) > bound).reshape(-1, m).any(axis=1))
    floor = np.zeros(got.size)
    if need.size:
        fl = fp32_key_floor(oracle, kappa_of(need), sbar_of_groups(need), n, tau32, 1.0)
        floor.reshape(-1, m)[need] = fl
    assert_close(got, ref, what + " (relative)", scale_aware=True, floor=floor)
    worst = 0.0
    if need.size:
        e = np.abs(got - ref).reshape(-1, m)[need]
        worst = float((e / (bound.reshape(-1, m)[need] + floor.reshape(-1, m)[need])).max())
    say(f"  {what}: err/bound {r:.3f}; {need.size} of {got.size // m} groups over the relative "
        f"bar, worst at {worst:.3f} of it with the fp32 allowance")


def whole_layer_check(dev, work, tensors, W, L, G, Wm, S, idx, d, n, m, tau, step):
    """Every group of the given consecutive tensors (whole layers of the stack)
    against the oracle on the host's cores: indices and masked weights bit for
    bit, the soft mask and the gradient elementwise."""
    import time
    t0, t1 = work.tensors[tensors[0]], work.tensors[tensors[-1]]
    e0, e1 = t0.offset, t1.offset + t1.numel
    g0, g1 = e0 // m, e1 // m
    threads = oracle.host_threads()
    say(f"  whole-layer check: tensors {t0.name} .. {t1.name}, {e1 - e0} weights, "
        f"oracle on {threads} threads")
    Wb, Lh, Gb = bf16_bits(W[e0:e1]), f32(L[e0:e1]).reshape(-1), bf16_bits(G[e0:e1])
    tau32 = float(np.float32(tau))
    start = time.time()
    Wm_o, S_o, idx_o = oracle.mask_fwd(Wb, Lh, n, m, tau32, 1.0, 0, step, e0, want_soft=True,
                                       threads=threads)
    say(f"  oracle forward {time.time() - start:.1f} s")
    assert np.array_equal(idx[g0:g1].cpu().numpy(), idx_o), "selected indices differ"
    assert np.array_equal(bf16_bits(Wm[e0:e1]).reshape(-1), Wm_o), "masked weights differ"
    del Wm_o, idx_o
    r = assert_close(f32(S[e0:e1]).reshape(-1), S_o, "soft mask (whole layer)")
    say(f"  soft mask err/bound {r:.3f}")
    del S_o
    start = time.time()
    d_o = oracle.mask_bwd(Gb, Wb, Lh, n, m, tau32, 1.0, 0, step, e0, threads=threads)
    say(f"  oracle backward {time.time() - start:.1f} s")
    Wg, Gg, Lg = Wb.reshape(-1, m), Gb.reshape(-1, m), Lh.reshape(-1, m)
    kappa_of = lambda q: np.stack([oracle.keys(Lg[i], 1.0, 0, step, e0 + int(i) * m) for i in q])
    sbar_of_groups = lambda q: sbar_of(Gg[q], Wg[q])
    check_grad_whole(f32(d[e0:e1]).reshape(-1), d_o, kappa_of, sbar_of_groups, n, m, tau32,
                     "grad_logits (whole layer)")


def full_workload_check(dev, name, n, m, tau, step, count, whole=None):
    """The whole stack in one call (the benchmark's launch configuration):
    sampled groups against the oracle, structural properties on every group,
    and every group of the tensors in `whole` (whole layers) against the
    oracle on the host's cores."""
    import torch
    work = wl.WORKLOADS[name]
    say(f"full workload {name} {n}:{m} tau={tau} step={step}: allocating {work.numel} weights")
    W, L, G = wl.fill_slab(work, dev, step=step)
    Wm, _, idx = roi.mask_fwd(W, L, n, m, tau, 1.0, 0, step, 0, want_soft=False)
    d = roi.mask_bwd(G, W, L, n, m, tau, 1.0, 0, step, 0)
    torch.cuda.synchronize()
    if whole is not None:
        # the forward with the soft mask: the same selection, bit for bit
        Wm_s, S, idx_s = roi.mask_fwd(W, L, n, m, tau, 1.0, 0, step, 0, want_soft=True)
        torch.cuda.synchronize()
        assert torch.equal(idx_s, idx) and torch.equal(Wm_s.view(torch.int16), Wm.view(torch.int16))
        del Wm_s, idx_s
        whole_layer_check(dev, work, whole, W, L, G, Wm, S, idx, d, n, m, tau, step)
        del S
        torch.cuda.empty_cache()
    say("  kernels done; checking properties")
    ng = work.numel // m
    chunk = 1 << 26
    ar = torch.arange(m, device=dev, dtype=torch.uint8)
    for g0 in range(0, ng, chunk):
        g1 = min(ng, g0 + chunk)
        ii = idx[g0:g1].long()
        hard = torch.zeros((g1 - g0, m), dtype=torch.bool, device=dev)
        hard.scatter_(1, ii, True)
        assert bool((hard.sum(1) == n).all()), "a group does not keep exactly n entries"
        w = W[g0 * m:g1 * m].view(-1, m).view(torch.int16)
        wm = Wm[g0 * m:g1 * m].view(-1, m).view(torch.int16)
        assert torch.equal(wm, torch.where(hard, w, torch.zeros_like(w))), "W_masked != W (.) hard"
        assert bool(torch.isfinite(d[g0 * m:g1 * m]).all())
        del ii, hard, w, wm
    del ar
    rng = np.random.default_rng(1234 + step)
    picks = sample_groups(work, ng, m, rng, count)
    say(f"  comparing {picks.size} sampled groups with the oracle")
    pt = torch.from_numpy(picks).to(dev)
    take = lambda t: t.view(-1, m).index_select(0, pt)
    Wg, Lg, Gg = take(W), take(L), take(G)
    tau32 = float(np.float32(tau))
    ge = picks.astype(np.uint64) * np.uint64(m)
    Wm_o, _, idx_o = oracle.mask_fwd_groups(bf16_bits(Wg), f32(Lg), ge, n, m, tau32, 1.0, 0, step,
                                            want_soft=False)
    d_o = oracle.mask_bwd_groups(bf16_bits(Gg), bf16_bits(Wg), f32(Lg), ge, n, m, tau32, 1.0, 0,
                                 step)
    assert np.array_equal(idx.index_select(0, pt).cpu().numpy(), idx_o)
    assert np.array_equal(bf16_bits(take(Wm)), Wm_o)
    r = assert_close(f32(take(d)), d_o, f"grad_logits ({name})")
    say(f"  ok: grad err/bound {r:.3f}")
    del W, L, G, Wm, idx, d
    torch.cuda.empty_cache()


def test_full_qwen05b_stack_2of4(dev):
    full_workload_check(dev, "qwen2.5-0.5b-stack-2:4", 2, 4, 1.0, 0, 20000)


LAST_LAYER = list(range(27 * 7, 28 * 7))  # the seven tensors of layer 27 of a 28-layer stack


def test_full_qwen7b_layer_2of4(dev):
    """The 7B-class layer at 2:4: every group against the oracle."""
    full_workload_check(dev, "qwen2.5-7b-layer-2:4", 2, 4, 0.5, 0, 20000, whole=list(range(7)))


def test_full_qwen7b_layer_4of8(dev):
    """The 7B-class layer at 4:8: every group against the oracle."""
    full_workload_check(dev, "qwen2.5-7b-layer-4:8", 4, 8, 0.5, 0, 20000, whole=list(range(7)))


@pytest.mark.parametrize("step", [0, 9])
def test_full_qwen7b_stack_2of4(dev, step):
    """The whole 7B stack in one call at the first and the last annealing
    step: every group of its last layer (global offsets past 6e9) against the
    oracle, sampled groups elsewhere."""
    tau = roi.anneal(1.0, 0.1, step, 9)
    full_workload_check(dev, "qwen2.5-7b-stack-2:4", 2, 4, tau, step, 30000, whole=LAST_LAYER)


@pytest.mark.parametrize("name,n,m", [("qwen2.5-1.5b-stack-8:16", 8, 16),
                                      ("qwen2.5-1.5b-stack-16:32", 16, 32)])
def test_full_qwen15b_stack_wide(dev, name, n, m):
    """The 1.5B stack at 8:16 and 16:32 in one call: every group of its last
    layer against the oracle, sampled groups elsewhere."""
    full_workload_check(dev, name, n, m, 1.0, 0, 20000, whole=LAST_LAYER)


@pytest.mark.parametrize("name,n,m,tau,step", [("qwen2.5-7b-stack-2:4", 2, 4, 0.1, 9),
                                                 ("qwen2.5-1.5b-stack-16:32", 16, 32, 1.0, 0)])
def test_full_soft_forward_alone(dev, name, n, m, tau, step):
    """The soft forward with W_soft as its only output over a whole stack in
    one call, as `bench.py --mode soft` runs it: the 7B stack at its last
    annealing step (tau = 0.1, one group per lane) and the 1.5B stack at
    16:32 (a group over eight lanes).  Sampled groups against the oracle's
    W (.) S: within one bf16 rounding step plus the float tolerance."""
    import torch
    work = wl.WORKLOADS[name]
    say(f"full soft forward alone {name} {n}:{m} tau={tau}: allocating {work.numel} weights")
    W, L, G = wl.fill_slab(work, dev, step=step)
    del G
    Ws, _, _ = roi.mask_fwd(W, L, n, m, tau, 1.0, 0, step, 0, want_soft=False, want_idx=False,
                            soft_forward=True)
    torch.cuda.synchronize()
    ng = work.numel // m
    picks = sample_groups(work, ng, m, np.random.default_rng(4321 + step), 20000)
    say(f"  comparing {picks.size} sampled groups with the oracle")
    pt = torch.from_numpy(picks).to(dev)
    take = lambda t: t.view(-1, m).index_select(0, pt)
    Wg, Lg = take(W), take(L)
    ge = picks.astype(np.uint64) * np.uint64(m)
    _, S_o, _ = oracle.mask_fwd_groups(bf16_bits(Wg), f32(Lg), ge, n, m, float(np.float32(tau)),
                                       1.0, 0, step, want_soft=True)
    wf = (bf16_bits(Wg).astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(-1)
    ref = wf * S_o.reshape(-1)
    got = (bf16_bits(take(Ws)).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    ulp = np.where(ref != 0, 2.0 ** (np.floor(np.log2(np.abs(ref) + 1e-300)) - 7), 0.0)
    assert_close(got.reshape(-1), ref, f"W (.) S ({name})", floor=ulp)
    del W, L, Ws
    torch.cuda.empty_cache()


def check_sampled(dev, W, L, G, Wm, idx, d, n, m, tau, step, picks):
    """Sampled groups of a one-call slab against the oracle (indices and masked
    weights bit for bit, gradient within the tolerance)."""
    import torch
    pt = torch.from_numpy(picks).to(dev)
    take = lambda t: t.view(-1, m).index_select(0, pt)
    Wg, Lg = take(W), take(L)
    tau32 = float(np.float32(tau))
    ge = picks.astype(np.uint64) * np.uint64(m)
    if Wm is not None:
        Wm_o, _, idx_o = oracle.mask_fwd_groups(bf16_bits(Wg), f32(Lg), ge, n, m, tau32, 1.0, 0,
                                                step, want_soft=False)
        assert np.array_equal(idx.index_select(0, pt).cpu().numpy(), idx_o), "indices differ"
        assert np.array_equal(bf16_bits(take(Wm)), Wm_o), "masked weights differ"
    if d is not None:
        d_o = oracle.mask_bwd_groups(bf16_bits(take(G)), bf16_bits(Wg), f32(Lg), ge, n, m, tau32,
                                     1.0, 0, step)
        return assert_close(f32(take(d)), d_o, "grad_logits")
    return 0.0


def test_launch_beyond_2e32_work_items(dev):
    """A slab of 2^34 + 2^28 weights in one call.  Its first piece (2^34
    elements, up to the Philox block index's high-word change) needs 2^32
    work-items in the backward at m = 4 (one group per lane) and in both wide
    kernels at m = 16 (four elements per lane), one block more than a dispatch
    can hold: the grid is capped and its last 256 work-items run in the
    kernels' stride loops.  The second piece goes to a launch of its own.
    Sampled groups (random, around the 2^34 boundary, and those reached by
    the stride loops) against the oracle; every group keeps exactly n."""
    import torch
    E = (1 << 34) + (1 << 28)
    cols = 4096
    rows = E // cols
    say(f"beyond 2^32 work-items: allocating {E} weights")
    W = torch.empty(E, dtype=torch.bfloat16, device=dev)
    L = torch.empty(E, dtype=torch.float32, device=dev)
    gen = torch.Generator(device=dev).manual_seed(77)
    for c0 in range(0, E, 1 << 30):
        c1 = min(E, c0 + (1 << 30))
        L[c0:c1].normal_(0.0, 1.0, generator=gen)
        W[c0:c1] = (L[c0:c1] * 0.02).to(torch.bfloat16)  # any bf16 values of weight scale
    L.normal_(0.0, 1.0, generator=gen)
    torch.cuda.synchronize()
    rng = np.random.default_rng(99)
    for n, m, tau, step in ((2, 4, 0.7, 3), (8, 16, 1.0, 5)):
        ng = E // m
        first = (1 << 34) // m  # groups of the first piece
        # work-items of the largest grid of 256-thread blocks; the backward at
        # m = 4 has one group per work-item, the wide kernels m / 4 per group
        capped = (0xFFFFFFFF // 256) * 256
        in_grid = capped if m == 4 else capped // (m // 4)  # groups before the stride loop
        picks = np.unique(np.concatenate([
            rng.integers(0, ng, 4000), np.arange(first - 300, first + 300),
            np.arange(in_grid - 8, min(first, in_grid + 300)), [0, ng - 1]]))
        say(f"  {n}:{m}: forward")
        Wm, _, idx = roi.mask_fwd(W.view(rows, cols), L.view(rows, cols), n, m, tau, 1.0, 0, step,
                                  0, want_soft=False)
        torch.cuda.synchronize()
        chunk = 1 << 26
        for g0 in range(0, ng, chunk):
            g1 = min(ng, g0 + chunk)
            hard = torch.zeros((g1 - g0, m), dtype=torch.bool, device=dev)
            hard.scatter_(1, idx[g0:g1].long(), True)
            assert bool((hard.sum(1) == n).all()), "a group does not keep exactly n entries"
            del hard
        check_sampled(dev, W, L, None, Wm.view(-1), idx, None, n, m, tau, step, picks)
        del idx
        say(f"  {n}:{m}: backward")
        G = Wm.view(-1)  # the masked weights serve as an upstream gradient of bf16 values
        d = roi.mask_bwd(G.view(rows, cols), W.view(rows, cols), L.view(rows, cols), n, m, tau,
                         1.0, 0, step, 0)
        torch.cuda.synchronize()
        for g0 in range(0, E, 1 << 30):
            assert bool(torch.isfinite(d.view(-1)[g0:g0 + (1 << 30)]).all())
        r = check_sampled(dev, W, L, G, None, None, d.view(-1), n, m, tau, step, picks)
        say(f"  ok: {picks.size} sampled groups, grad err/bound {r:.3f}")
        del Wm, G, d
        torch.cuda.empty_cache()
    del W, L
    torch.cuda.empty_cache()


# --------------------------------------------------------------------------- pure soft forward
SOFT = [(37, 36, 2, 4, 1.0, 1.0, 3, 1, 0), (64, 96, 2, 4, 0.1, 1.0, 5, 9, 8),
        (33, 64, 3, 4, 1.3, 0.6, 2, 3, 12), (61, 88, 4, 8, 0.5, 1.0, 8, 5, 8),
        (37, 48, 8, 16, 1.0, 1.0, 2, 0, 0), (33, 96, 16, 32, 1.0, 1.0, 4, 2, 0),
        (13, 64, 5, 32, 0.3, 0.8, 5, 3, 64),
        # the exp-domain relaxation with powers by multiplication (tau = 1/2) and
        # by exp2 / log2 (tau = 0.7) in the wide kernels
        (37, 48, 8, 16, 0.5, 1.0, 6, 2, 16), (33, 96, 16, 32, 0.7, 1.3, 7, 4, 0)]


@pytest.mark.parametrize("case", SOFT, ids=lambda c: "x".join(map(str, c[:4])))
def test_soft_forward(dev, case):
    """Pure soft forward (the paper's default, without the straight-through
    estimator): W_soft = bf16(W (.) S).  Against W (.) S from the oracle's fp64
    S: within one bf16 rounding step plus the float tolerance; S and the
    indices as in the straight-through forward."""
    import torch
    rows, cols, n, m, tau, lam, seed, step, off = case
    say(f"soft forward rows={rows} cols={cols} {n}:{m} tau={tau} lam={lam}")
    W, L, _ = wl.small_case(rows, cols, rows * 7 + cols, device=dev, w_std=1.0)
    Ws, S, idx = roi.mask_fwd(W, L, n, m, tau, lam, seed, step, off, want_soft=True,
                              soft_forward=True)
    Wh, S2, idx2 = roi.mask_fwd(W, L, n, m, tau, lam, seed, step, off, want_soft=True)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2) and torch.equal(S.view(torch.int32), S2.view(torch.int32))
    soft_product_exact(bf16_bits(W), f32(S), bf16_bits(Ws), "W_soft against the kernel's S")
    tau32, lam32 = float(np.float32(tau)), float(np.float32(lam))
    _, S_o, idx_o = oracle.mask_fwd(bf16_bits(W), f32(L), n, m, tau32, lam32, seed, step, off)
    assert np.array_equal(idx.cpu().numpy(), idx_o)
    ref = (bf16_bits(W).astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(-1) \
        * S_o
    got = (bf16_bits(Ws).astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(-1)
    ulp = np.where(ref != 0, 2.0 ** (np.floor(np.log2(np.abs(ref) + 1e-300)) - 7), 0.0)
    assert_close(got, ref, "W (.) S", floor=ulp)


# the soft forward cases plus small temperatures and lambda != 1
SOFT_ONLY = SOFT + [(61, 88, 6, 8, 0.1, 1.0, 3, 2, 0), (21, 80, 8, 16, 0.1, 0.7, 9, 1, 32),
                    (21, 80, 12, 16, 0.1, 0.7, 9, 1, 32), (13, 64, 24, 32, 0.15, 1.0, 2, 5, 0),
                    (37, 48, 2, 4, 1.0, 0.01, 3, 1, 0)]


@pytest.mark.parametrize("case", SOFT_ONLY, ids=lambda c: "x".join(map(str, c[:6])))
def test_soft_forward_alone(dev, case):
    """The pure soft forward with W_soft as its only output (no S, no indices)
    has a kernel of its own (no selection).  It runs the relaxation at the
    exact keys, so its output is the soft forward's with S requested, bit for
    bit, and within one bf16 rounding step plus the float tolerance of
    W (.) S from the oracle's fp64 S."""
    import torch
    rows, cols, n, m, tau, lam, seed, step, off = case
    say(f"soft forward alone rows={rows} cols={cols} {n}:{m} tau={tau} lam={lam}")
    W, L, _ = wl.small_case(rows, cols, rows * 7 + cols, device=dev, w_std=1.0)
    Ws, S, idx = roi.mask_fwd(W, L, n, m, tau, lam, seed, step, off, want_soft=False,
                              want_idx=False, soft_forward=True)
    assert S is None and idx is None
    We, Se, _ = roi.mask_fwd(W, L, n, m, tau, lam, seed, step, off, want_soft=True,
                             soft_forward=True)
    torch.cuda.synchronize()
    assert torch.equal(Ws.view(torch.int16), We.view(torch.int16)), \
        "the soft forward alone differs from the soft forward with S"
    soft_product_exact(bf16_bits(W), f32(Se), bf16_bits(Ws), "W_soft against the kernel's S")
    tau32, lam32 = float(np.float32(tau)), float(np.float32(lam))
    _, S_o, _ = oracle.mask_fwd(bf16_bits(W), f32(L), n, m, tau32, lam32, seed, step, off)
    wf = (bf16_bits(W).astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(-1)
    ref = wf * S_o.reshape(-1)
    got = (bf16_bits(Ws).astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(-1)
    ulp = np.where(ref != 0, 2.0 ** (np.floor(np.log2(np.abs(ref) + 1e-300)) - 7), 0.0)
    assert_close(got, ref, "W (.) S", floor=ulp)


def test_stream_copy(dev):
    """The benchmark's data-movement reference copies every byte, including a
    ragged tail of the last block, and rejects bad arguments before launching."""
    import torch
    n = 16 * (256 * 37 + 5)
    src = torch.randint(0, 256, (n,), dtype=torch.uint8, device=dev)
    dst = torch.zeros_like(src)
    roi.stream_copy(src, dst)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    L = roi.lib()
    p = src.data_ptr()
    assert L.roi_stream_copy(p, dst.data_ptr(), 24, None) == roi.ROI_E_INVAL      # not a multiple of 16
    assert L.roi_stream_copy(p + 8, dst.data_ptr(), 32, None) == roi.ROI_E_INVAL  # misaligned
    assert L.roi_stream_copy(p, p + 16, 64, None) == roi.ROI_E_INVAL              # overlap
    assert L.roi_stream_copy(p, dst.data_ptr(), 0, None) == roi.ROI_OK
