"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: an
independent library implementation (rocRAND's Philox4x32-10, numpy/scipy
log and softmax, torch autograd, mpmath), a closed form derived from the
paper's recursion, exact rational arithmetic, brute-force enumeration of the
Weighted-Reservoir-Sampling law (Eq. 1, §3.1), or an invariant.  No GPU.
"""
from __future__ import annotations

import itertools
import json
import math
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest
from scipy import special, stats

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def ulp32(x: np.ndarray) -> np.ndarray:
    x = np.abs(np.asarray(x, dtype=np.float32))
    return np.spacing(x).astype(np.float64)


# --------------------------------------------------------------------------- Philox
@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available for the rocRAND reference")
    exe = str(tmp_path_factory.mktemp("rr") / "philox_ref")
    subprocess.run([hipcc, "-O1", "-w", "-o", exe, os.path.join(HERE, "rocrand_philox_ref.cpp")],
                   check=True, capture_output=True)
    return exe


def test_philox_matches_rocrand(rocrand_ref):
    """Philox4x32-10 (Salmon et al., SC'11) with counter (elem/4, step), key
    seed and word elem%4 equals rocRAND's engine at (seed, subsequence=step,
    offset=elem), an independent implementation of the same generator."""
    cases = [
        (0, 0, 0, 64),
        (1, 0, 0, 16),
        (0, 1, 0, 16),
        (0x0123456789ABCDEF, 9, 1000003, 37),
        (0xFFFFFFFF00000001, (1 << 32) + 5, (1 << 34) - 6, 40),  # counter crosses 2^32 blocks
        (42, 7, 6525288448 - 13, 29),  # near the end of the 7B-class stack
        (2**64 - 1, 2**64 - 1, 2**63 + 1, 11),
    ]
    text = "".join(f"{s} {st} {o} {c}\n" for s, st, o, c in cases)
    out = subprocess.run([rocrand_ref], input=text, capture_output=True, text=True, check=True)
    ref = [int(w, 16) for w in out.stdout.split()]
    mine = []
    for s, st, o, c in cases:
        mine += [oracle.philox_word(s, st, o + i) for i in range(c)]
    assert mine == ref


def test_philox_block_structure():
    """The four words of one call are the four elements of one block."""
    out = oracle.philox4x32_10([5, 0, 3, 0], [11, 0])
    assert [oracle.philox_word(11, 3, 20 + i) for i in range(4)] == list(out)


def test_philox_bit_balance():
    words = np.array([oracle.philox_word(0, 0, e) for e in range(1 << 16)], dtype=np.uint32)
    bits = np.unpackbits(words.view(np.uint8))
    # 2^21 fair bits: mean within 5 sigma of 1/2
    assert abs(bits.mean() - 0.5) < 5 * 0.5 / math.sqrt(bits.size)
    hist = np.bincount(words >> 24, minlength=256)
    chi2 = ((hist - hist.mean()) ** 2 / hist.mean()).sum()
    assert stats.chi2.sf(chi2, 255) > 1e-4


# --------------------------------------------------------------------------- uniform
def test_uniform_grid_exact_and_open():
    assert oracle.uniform(0) == 2.0 ** -24
    assert oracle.uniform(0xFFFFFFFF) == 1.0 - 2.0 ** -24
    rng = np.random.default_rng(1)
    for w in rng.integers(0, 2**32, 2000, dtype=np.uint64):
        u = oracle.uniform(int(w))
        k = int(w) >> 9
        assert u * 2**24 == 2 * k + 1
        assert 0.0 < u < 1.0


# --------------------------------------------------------------------------- deterministic log
def test_log_accuracy_every_mantissa():
    """Every fp32 mantissa in four binades (all 2^23 values each): the fp32
    result is within 1.5 ulp of numpy's fp64 log (error measured in ulp of the
    correctly rounded fp32 value, or absolutely near ln x = 0)."""
    mant = np.arange(1 << 23, dtype=np.uint32)
    for exp_bits in (126, 127, 100, 131):  # [0.5,1), [1,2), tiny, [16,32)
        x = ((np.uint32(exp_bits) << 23) | mant).view(np.float32)
        got = oracle.log32_array(x).astype(np.float64)
        ref = np.log(x.astype(np.float64))
        err = np.abs(got - ref) / np.maximum(ulp32(ref.astype(np.float32)), 2.0 ** -149)
        # near x = 1 the value is tiny; there the error is bounded relative to |ln x| by
        # the same 2 ulp (the reduction leaves m - 1 exact), so the ulp measure applies.
        assert err.max() <= 1.5, (exp_bits, err.max(), x[err.argmax()])


def test_log_special_values():
    assert oracle.log32(1.0) == 0.0
    for k in range(-24, 8):
        got = float(oracle.log32(2.0 ** k))
        assert abs(got - k * math.log(2)) <= float(ulp32(np.float32(k * math.log(2)))) + 1e-30


# --------------------------------------------------------------------------- Gumbel noise
@pytest.fixture(scope="module")
def gumbel_grid():
    k = np.arange(1 << 23, dtype=np.uint32)
    words = k << np.uint32(9)
    u = (2.0 * k.astype(np.float64) + 1.0) * 2.0 ** -24
    g = oracle.gumbel_from_words(words).astype(np.float64)
    return u, g


def test_gumbel_is_inverse_cdf(gumbel_grid):
    """Algorithm 1: g = -log(-log u) is the inverse of the Gumbel(0,1) CDF
    F(g) = exp(-exp(-g)).  Over all 2^23 grid values, g matches the fp64
    inverse CDF within the fp32 error budget of the two logarithms."""
    u, g = gumbel_grid
    ref = -np.log(-np.log(u))
    # inner log relative error (<= 2 ulp) becomes an absolute error in g; the
    # outer log adds <= 2 ulp of g.
    tol = 2.5 * 2.0 ** -23 + 2.5 * ulp32(ref.astype(np.float32))
    assert np.all(np.abs(g - ref) <= tol)
    assert np.all(np.abs(np.exp(-np.exp(-g)) - u) <= 4e-6 * np.maximum(u, 1e-3))


def test_gumbel_monotone_and_moments(gumbel_grid):
    u, g = gumbel_grid
    assert np.all(np.diff(g) >= 0)
    assert g.min() > -3.0 and g.max() < 17.0
    # midpoint rule over the full grid: E[g] = Euler-Mascheroni, Var[g] = pi^2/6
    assert abs(g.mean() - np.euler_gamma) < 2e-6
    assert abs(g.var() - math.pi ** 2 / 6) < 2e-5


def test_keys_use_scaled_logits():
    """§4.2.3: the trick is applied to phi / lambda; with the noise fixed the
    keys move by exactly the change of phi / lambda (up to fp32 rounding)."""
    phi = np.linspace(-3, 3, 64).astype(np.float32)
    k1 = oracle.keys(phi, 1.0, 3, 4, 128).astype(np.float64)
    k0 = oracle.keys(np.zeros_like(phi), 1.0, 3, 4, 128).astype(np.float64)
    k2 = oracle.keys(phi, 2.0, 3, 4, 128).astype(np.float64)
    assert np.allclose(k1 - k0, phi, atol=4e-6)
    assert np.allclose(k2 - k0, phi / 2.0, atol=4e-6)


# --------------------------------------------------------------------------- hard top-N
def test_topn_matches_sort_with_ties():
    rng = np.random.default_rng(7)
    for trial in range(3000):
        m = int(rng.choice([4, 8, 16, 32, 5, 3]))
        n = int(rng.integers(1, m + 1))
        kappa = rng.normal(size=m).astype(np.float32)
        if trial % 3 == 0:  # heavy ties, including -0 and +0
            kappa = rng.choice(np.array([0.0, -0.0, 1.0, -1.0], dtype=np.float32), size=m)
        order, hard = oracle.topn(kappa, n)
        ref = sorted(range(m), key=lambda j: (-float(kappa[j]), j))[:n]
        assert list(order) == ref
        assert hard.sum() == n and all(hard[j] for j in ref)


def test_minus_zero_ties_plus_zero():
    order, _ = oracle.topn(np.array([-0.0, 0.0, -1.0, -2.0], dtype=np.float32), 1)
    assert order[0] == 0
    order, _ = oracle.topn(np.array([-1.0, 0.0, -0.0, -2.0], dtype=np.float32), 2)
    assert list(order) == [1, 2]


# --------------------------------------------------------------------------- WRS law (Eq. 1)
def wrs_ordered_prob(w, order):
    """Eq. 1 (§3.1): product of w_{y_i} / (W - sum_{j<i} w_{y_j})."""
    total = sum(w)
    p = Fraction(1)
    used = Fraction(0)
    for y in order:
        p *= w[y] / (total - used)
        used += w[y]
    return p


def sample_selection(w, n, groups, lam=1.0, seed=0, step=0):
    m = len(w)
    phi = np.tile((lam * np.log(np.array([float(x) for x in w]))).astype(np.float32), groups)
    W = np.ones(phi.size, dtype=np.uint16) * 0x3F80
    _, _, idx = oracle.mask_fwd(W, phi, n, m, 1.0, lam, seed, step, 0, want_soft=False)
    return idx


@pytest.mark.parametrize("w,n,groups,ordered,lam", [
    ((Fraction(4, 10), Fraction(3, 10), Fraction(2, 10), Fraction(1, 10)), 2, 400_000, True, 1.0),
    ((Fraction(4, 10), Fraction(3, 10), Fraction(2, 10), Fraction(1, 10)), 2, 200_000, True, 0.5),
    ((Fraction(5), Fraction(1), Fraction(3), Fraction(1)), 1, 200_000, True, 1.0),
    ((Fraction(5), Fraction(1), Fraction(3), Fraction(1)), 3, 200_000, True, 1.0),
    (tuple(Fraction(k) for k in (8, 1, 2, 7, 3, 1, 5, 4)), 2, 200_000, True, 1.0),
    (tuple(Fraction(k) for k in (8, 1, 2, 7, 3, 1, 5, 4)), 4, 200_000, False, 1.0),
])
def test_selection_law_is_wrs(w, n, groups, ordered, lam):
    """Selection frequencies of the hard top-n equal brute-force enumeration
    of the WRS law: ordered tuples against Eq. 1 directly, unordered subsets
    against Eq. 1 summed over orderings (the mask distribution of §4.2.1)."""
    m = len(w)
    idx = sample_selection(w, n, groups, lam=lam, seed=12345, step=3)
    if ordered:
        outcomes = list(itertools.permutations(range(m), n))
        probs = np.array([float(wrs_ordered_prob(w, o)) for o in outcomes])
        code = np.zeros(idx.shape[0], dtype=np.int64)
        for k in range(n):
            code = code * m + idx[:, k]
        keys = [sum(o[k] * m ** (n - 1 - k) for k in range(n)) for o in outcomes]
    else:
        outcomes = list(itertools.combinations(range(m), n))
        probs = np.array([float(sum(wrs_ordered_prob(w, p) for p in itertools.permutations(c)))
                          for c in outcomes])
        code = np.zeros(idx.shape[0], dtype=np.int64)
        for k in range(n):
            code |= np.int64(1) << idx[:, k].astype(np.int64)
        keys = [sum(1 << j for j in c) for c in outcomes]
    assert abs(probs.sum() - 1.0) < 1e-12
    lookup = {kk: i for i, kk in enumerate(keys)}
    counts = np.zeros(len(outcomes))
    vals, cnt = np.unique(code, return_counts=True)
    for v, c in zip(vals, cnt):
        counts[lookup[int(v)]] += c
    expected = probs * idx.shape[0]
    keep = expected >= 5
    obs = np.append(counts[keep], counts[~keep].sum())
    exp_ = np.append(expected[keep], expected[~keep].sum())
    if exp_[-1] == 0:
        obs, exp_ = obs[:-1], exp_[:-1]
    chi2 = ((obs - exp_) ** 2 / exp_).sum()
    assert stats.chi2.sf(chi2, len(obs) - 1) > 1e-4, (chi2, len(obs))


def test_inclusion_probabilities_2of4():
    """Worked example derived from Eq. 1: w = (0.4, 0.3, 0.2, 0.1), 2:4.
    Inclusion probabilities sum to N."""
    w = (Fraction(4, 10), Fraction(3, 10), Fraction(2, 10), Fraction(1, 10))
    incl = [sum(wrs_ordered_prob(w, o) for o in itertools.permutations(range(4), 2) if j in o)
            for j in range(4)]
    assert sum(incl) == 2
    idx = sample_selection(w, 2, 400_000, seed=99)
    freq = np.array([(idx == j).any(axis=1).mean() for j in range(4)])
    assert np.allclose(freq, [float(x) for x in incl], atol=5 * 0.5 / math.sqrt(400_000))


# --------------------------------------------------------------------------- relaxation
def exact_relaxation_tau1(w, n):
    """S at tau = 1 in exact rational arithmetic.  With e = exp(alpha), the
    recursion of §3.2 reads mu = e / sum(e), e <- e (1 - mu): every quantity
    stays rational when the initial weights exp(kappa) are rational."""
    e = [Fraction(x) for x in w]
    S = [Fraction(0)] * len(e)
    for _ in range(n):
        t = sum(e)
        mu = [x / t for x in e]
        S = [s + x for s, x in zip(S, mu)]
        e = [x * (1 - y) for x, y in zip(e, mu)]
    return S


def test_relaxation_worked_example_exact():
    w = (Fraction(4, 10), Fraction(3, 10), Fraction(2, 10), Fraction(1, 10))
    S = oracle.relax_fwd(np.log([0.4, 0.3, 0.2, 0.1]), 2, 1.0)
    assert exact_relaxation_tau1(w, 2) == [Fraction(26, 35), Fraction(3, 5), Fraction(3, 7),
                                           Fraction(8, 35)]
    assert np.allclose(S, [26 / 35, 3 / 5, 3 / 7, 8 / 35], rtol=1e-14, atol=0)
    # S_j may exceed 1: M = 2, N = 2, p = (0.9, 0.1) gives (1.4, 0.6)
    assert np.allclose(oracle.relax_fwd(np.log([0.9, 0.1]), 2, 1.0), [1.4, 0.6], rtol=1e-14)


@pytest.mark.parametrize("m,n", [(4, 1), (4, 2), (4, 3), (4, 4), (8, 4), (8, 7), (16, 8), (32, 4),
                                 (5, 3)])
def test_relaxation_exact_rational_tau1(m, n):
    rng = np.random.default_rng(m * 100 + n)
    for _ in range(20):
        w = [Fraction(int(x), 64) for x in rng.integers(1, 256, size=m)]
        ref = exact_relaxation_tau1(w, n)
        S = oracle.relax_fwd(np.log([float(x) for x in w]), n, 1.0)
        assert np.allclose(S, [float(x) for x in ref], rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("tau", [0.1, 0.5, 1.0, 2.0])
def test_relaxation_closed_forms_n1_n2(tau):
    """N = 1: S = softmax(kappa / tau) (the Gumbel-softmax).  N = 2:
    S = p + p (1-p)^(1/tau) / sum(p (1-p)^(1/tau)), p = softmax(kappa/tau)
    (one step of the §3.2 recursion in closed form)."""
    rng = np.random.default_rng(int(tau * 100))
    for m in (4, 8, 16):
        for _ in range(30):
            kappa = rng.normal(scale=2.0, size=m)
            p = special.softmax(kappa / tau)
            assert np.allclose(oracle.relax_fwd(kappa, 1, tau), p, rtol=1e-12, atol=1e-300)
            q = p * (1.0 - p) ** (1.0 / tau)
            assert np.allclose(oracle.relax_fwd(kappa, 2, tau), p + q / q.sum(), rtol=1e-11,
                               atol=1e-300)


def test_relaxation_invariants():
    rng = np.random.default_rng(3)
    for _ in range(500):
        m = int(rng.choice([4, 8, 16, 32]))
        n = int(rng.integers(1, m + 1))
        tau = float(rng.choice([0.1, 0.3, 1.0, 3.0]))
        kappa = rng.normal(scale=3.0, size=m)
        S = oracle.relax_fwd(kappa, n, tau)
        assert abs(S.sum() - n) < 1e-12 * n * m
        assert np.all(S >= 0) and np.all(S <= n)
        perm = rng.permutation(m)
        assert np.allclose(oracle.relax_fwd(kappa[perm], n, tau), S[perm], rtol=1e-12, atol=1e-300)
        assert np.allclose(oracle.relax_fwd(kappa + 5.25, n, tau), S, rtol=1e-12, atol=1e-300)


def test_relaxation_zero_temperature_limit_is_hard_topn():
    """tau -> 0: every softmax becomes the one-hot of the current maximum and
    log(1 - mu) removes it, so S tends to the hard top-n mask."""
    rng = np.random.default_rng(5)
    for _ in range(300):
        m = int(rng.choice([4, 8, 16]))
        n = int(rng.integers(1, m + 1))
        kappa = rng.permutation(np.arange(m, dtype=np.float64)) * 0.5  # gaps >= 0.5
        _, hard = oracle.topn(kappa.astype(np.float32), n)
        S = oracle.relax_fwd(kappa, n, 1e-3)
        assert np.allclose(S, hard, atol=1e-12)


def test_relaxation_large_temperature_is_uniform():
    kappa = np.array([3.0, -1.0, 0.5, 2.0, 0.0, 1.0, -2.0, 4.0])
    assert np.allclose(oracle.relax_fwd(kappa, 3, 1e9), 3 / 8, atol=1e-8)


# --------------------------------------------------------------------------- backward
def test_backward_n1_closed_form():
    """N = 1: the softmax Jacobian, dkappa = (1/tau) p (sbar - <p, sbar>)."""
    rng = np.random.default_rng(11)
    for _ in range(200):
        m = int(rng.choice([4, 8, 16]))
        tau = float(rng.choice([0.2, 1.0, 2.5]))
        kappa = rng.normal(scale=2, size=m)
        sbar = rng.normal(size=m)
        p = special.softmax(kappa / tau)
        ref = p * (sbar - p @ sbar) / tau
        assert np.allclose(oracle.relax_bwd(kappa, 1, tau, sbar), ref, rtol=1e-11, atol=1e-14)


@pytest.mark.parametrize("m,n", [(4, 2), (4, 3), (4, 4), (8, 4), (16, 8), (5, 3), (32, 16)])
@pytest.mark.parametrize("tau", [1.0, 0.5, 0.3, 2.0])
def test_backward_matches_finite_differences(m, n, tau):
    rng = np.random.default_rng(m * 1000 + n * 10 + int(tau * 10))
    for _ in range(4):
        kappa = rng.normal(scale=1.5, size=m)
        sbar = rng.normal(size=m)
        got = oracle.relax_bwd(kappa, n, tau, sbar)
        h = 1e-6
        fd = np.empty(m)
        for j in range(m):
            kp, km = kappa.copy(), kappa.copy()
            kp[j] += h
            km[j] -= h
            fd[j] = (oracle.relax_fwd(kp, n, tau) - oracle.relax_fwd(km, n, tau)) @ sbar / (2 * h)
        assert np.allclose(got, fd, rtol=1e-6, atol=1e-8 * np.abs(sbar).max()), (got, fd)


def torch_relaxation(kappa, n, tau):
    """The §3.2 recursion written literally with torch ops, for autograd."""
    import torch
    alpha = kappa
    S = torch.zeros_like(kappa)
    for _ in range(n):
        mu = torch.softmax(alpha / tau, dim=-1)
        S = S + mu
        alpha = alpha + torch.log1p(-mu)
    return S


@pytest.mark.parametrize("m,n", [(4, 2), (8, 4), (8, 7), (16, 8), (32, 16)])
def test_backward_matches_torch_autograd(m, n):
    import torch
    rng = np.random.default_rng(m + 31 * n)
    for tau in (1.0, 0.5, 2.0):
        for _ in range(10):
            kappa = rng.normal(scale=1.0, size=m)
            sbar = rng.normal(size=m)
            k = torch.tensor(kappa, dtype=torch.float64, requires_grad=True)
            S = torch_relaxation(k, n, tau)
            (S * torch.tensor(sbar, dtype=torch.float64)).sum().backward()
            ref = k.grad.numpy()
            got = oracle.relax_bwd(kappa, n, tau, sbar)
            assert np.allclose(got, ref, rtol=1e-8, atol=1e-11)
            assert np.allclose(oracle.relax_fwd(kappa, n, tau), S.detach().numpy(), rtol=1e-12)


def mp_relaxation(kappa, n, tau):
    import mpmath as mp
    alpha = list(kappa)
    S = [mp.mpf(0)] * len(alpha)
    for _ in range(n):
        a_max = max(alpha)
        e = [mp.exp((a - a_max) / tau) for a in alpha]
        t = mp.fsum(e)
        mu = [x / t for x in e]
        S = [s + x for s, x in zip(S, mu)]
        alpha = [a + mp.log(mp.fsum(mu[:j] + mu[j + 1:])) for j, a in enumerate(alpha)]
    return S


@pytest.mark.parametrize("kappa,n,tau", [
    ([30.0, 0.0, 0.5, -1.0], 2, 1.0),     # first pick nearly certain: 1 - mu ~ 1e-13
    ([30.0, 0.0, 0.5, -1.0], 3, 1.0),
    ([25.0, 24.0, 0.0, -3.0], 3, 1.0),
    ([12.0, 0.0, 0.3, -1.0], 2, 2.0),      # tau > 1
    ([12.0, 0.0, 0.3, -1.0, 1.0, 2.0, -0.5, 0.7], 4, 0.5),
    ([8.0, 0.0, 0.3, -1.0], 2, 0.3),       # omega^(1/tau) tiny but no floor
])
def test_backward_extreme_keys_mpmath(kappa, n, tau):
    """Keys with a dominant entry, where a naive reverse sweep cancels
    catastrophically: compare with 60-digit finite differences of the
    recursion evaluated in mpmath."""
    import mpmath as mp
    mp.mp.dps = 60
    m = len(kappa)
    rng = np.random.default_rng(17)
    sbar = rng.normal(size=m)
    got = oracle.relax_bwd(np.array(kappa), n, tau, sbar)
    h = mp.mpf("1e-25")
    ref = []
    for j in range(m):
        kp = [mp.mpf(x) for x in kappa]
        km = [mp.mpf(x) for x in kappa]
        kp[j] += h
        km[j] -= h
        sp, sm = mp_relaxation(kp, n, mp.mpf(tau)), mp_relaxation(km, n, mp.mpf(tau))
        ref.append(float(mp.fsum((a - b) * mp.mpf(float(s)) for a, b, s in zip(sp, sm, sbar))
                         / (2 * h)))
    ref = np.array(ref)
    assert np.allclose(got, ref, rtol=1e-9, atol=1e-12 * np.abs(sbar).max()), (got, ref)
    S = oracle.relax_fwd(np.array(kappa), n, tau)
    Smp = np.array([float(x) for x in mp_relaxation([mp.mpf(x) for x in kappa], n, mp.mpf(tau))])
    assert np.allclose(S, Smp, rtol=1e-12, atol=1e-300)


# The floored branch: where 1 - mu falls below FLT_MIN the log is floored at
# log(FLT_MIN) and passes no derivative (the stable form of the §3.2 update).
FLT_MIN = float(np.finfo(np.float32).tiny)


def mp_relaxation_floored(kappa, n, tau, floor=True):
    """The §3.2 recursion in mpmath with the floor written out: alpha_j +=
    log(max(omega_j, FLT_MIN)) with omega_j the sum of the other entries over
    the total.  Returns S and, per step, the omegas that fed an update."""
    import mpmath as mp
    fmin = mp.mpf(FLT_MIN)
    alpha = list(kappa)
    S = [mp.mpf(0)] * len(alpha)
    omegas = []
    for k in range(n):
        a_max = max(alpha)
        e = [mp.exp((a - a_max) / tau) for a in alpha]
        t = mp.fsum(e)
        mu = [x / t for x in e]
        S = [s + x for s, x in zip(S, mu)]
        om = [mp.fsum(e[:j] + e[j + 1:]) / t for j in range(len(e))]
        if k + 1 < n:
            omegas.append(om)
        alpha = [a + mp.log(max(o, fmin) if floor else o) for a, o in zip(alpha, om)]
    return S, omegas


def mp_floored_gradient(kappa, n, tau, sbar, floor=True):
    """60-digit central differences of sum_j sbar_j S_j; the step is far too
    small to move any omega across the floor, so this is the exact derivative
    of the floored recursion."""
    import mpmath as mp
    mp.mp.dps = 60
    h = mp.mpf("1e-25")
    out = []
    for j in range(len(kappa)):
        kp = [mp.mpf(x) for x in kappa]
        km = [mp.mpf(x) for x in kappa]
        kp[j] += h
        km[j] -= h
        sp, _ = mp_relaxation_floored(kp, n, mp.mpf(tau), floor)
        sm, _ = mp_relaxation_floored(km, n, mp.mpf(tau), floor)
        out.append(float(mp.fsum((a - b) * mp.mpf(float(s)) for a, b, s in zip(sp, sm, sbar))
                         / (2 * h)))
    return np.array(out)


FLOOR_CASES = [
    # The first pick's 1 - mu is ~e^-100 (or smaller), below FLT_MIN, and the
    # floored entry's alpha = kappa + log(FLT_MIN) still counts at later steps,
    # so the floor changes both S and its derivative.
    ([100.0, 0.0, 0.5, -1.0], 2, 1.0),
    ([100.0, 0.0, 0.5, -1.0], 3, 1.0),
    ([89.5, 0.0, 0.5, -1.0], 3, 1.0),        # floored entry competes again at step 2
    ([100.0, 0.0, 0.25, -0.5], 2, 0.5),
    ([100.0, 0.0, 0.25, -0.5], 3, 0.5),
    ([250.0, 0.0, 0.5, -1.0], 3, 1.0),       # floored at steps 1 and 2
    ([200.0, 0.0, 1.0, -1.0, 0.4, -0.3, 0.8, 0.1], 4, 2.0),
    ([100.0, 0.0, 0.3, -0.6, 0.1, -0.2, 0.5, 0.2], 3, 0.6),
]


@pytest.mark.parametrize("kappa,n,tau", FLOOR_CASES)
def test_floored_branch_forward_and_backward_mpmath(kappa, n, tau):
    """Forward S and backward dS of the oracle's floored branch (keep = 1 for
    a floored entry's carried gradient, and no 1/omega term) against the
    recursion with the floor written out in mpmath and differentiated by
    60-digit central differences."""
    import mpmath as mp
    mp.mp.dps = 60
    m = len(kappa)
    sbar = np.random.default_rng(29 + m + n).normal(size=m)
    S_mp, omegas = mp_relaxation_floored([mp.mpf(x) for x in kappa], n, mp.mpf(tau))
    # the case really reaches the floor at an updating step, and no omega sits
    # near it (the finite difference must not cross it)
    om = np.array([[float(o) for o in row] for row in omegas])
    assert (om < FLT_MIN).any(), "case does not reach the floor"
    assert np.all((om < 0.5 * FLT_MIN) | (om > 2.0 * FLT_MIN))
    S = oracle.relax_fwd(np.array(kappa), n, tau)
    assert np.allclose(S, np.array([float(x) for x in S_mp]), rtol=1e-12, atol=1e-300)
    ref = mp_floored_gradient(kappa, n, tau, sbar)
    got = oracle.relax_bwd(np.array(kappa), n, tau, sbar)
    assert np.allclose(got, ref, rtol=1e-9, atol=1e-12 * np.abs(sbar).max()), (got, ref)
    # The floor changes the derivative: the unfloored recursion's gradient
    # differs, so a sweep that ignored the floor would fail the check above.
    unfloored = mp_floored_gradient(kappa, n, tau, sbar, floor=False)
    assert np.abs(unfloored - ref).max() > 1e-3 * np.abs(ref).max()


@pytest.mark.parametrize("kappa,n,tau", FLOOR_CASES)
def test_floored_branch_matches_torch_autograd_with_clamp(kappa, n, tau):
    """The same branch through torch fp64 autograd: the update written as
    alpha + log(clamp(omega, min=FLT_MIN)), omega the sum of the other
    exponentials over the total (clamp passes no gradient below its bound)."""
    import torch
    m = len(kappa)
    sbar = np.random.default_rng(31 + m + n).normal(size=m)
    k = torch.tensor(kappa, dtype=torch.float64, requires_grad=True)
    others_of = 1.0 - torch.eye(m, dtype=torch.float64)
    alpha, S = k, torch.zeros_like(k)
    for step in range(n):
        e = torch.exp((alpha - alpha.max().detach()) / tau)
        t = e.sum()
        S = S + e / t
        if step + 1 < n:
            alpha = alpha + torch.log(torch.clamp(others_of @ e / t, min=FLT_MIN))
    (S * torch.tensor(sbar, dtype=torch.float64)).sum().backward()
    got = oracle.relax_bwd(np.array(kappa), n, tau, sbar)
    assert np.allclose(got, k.grad.numpy(), rtol=1e-9, atol=1e-12 * np.abs(sbar).max())
    assert np.allclose(oracle.relax_fwd(np.array(kappa), n, tau), S.detach().numpy(), rtol=1e-12)


def test_floored_branch_planted_mistake_is_caught():
    """A plausible slip in the floored branch -- carrying a floored entry's
    gradient with the unfloored factor (omega + tau - 1) / tau instead of 1 --
    is far outside the tolerance of the pins above.  The slip is emulated on
    the CPU by a literal fp64 sweep of the derivation, checked first to agree
    with the oracle when written correctly."""
    def sweep(kappa, n, tau, sbar, slip):
        m = len(kappa)
        alpha = np.array(kappa, dtype=np.float64)
        recs = []
        for _ in range(n):
            e = np.exp((alpha - alpha.max()) / tau)
            t = e.sum()
            mu = e / t
            om = np.array([(e.sum() - e[j]) if e[j] < 0.5 * t else np.delete(e, j).sum()
                           for j in range(m)]) / t
            fl = om < FLT_MIN
            recs.append((mu, om, fl))
            alpha = alpha + np.log(np.maximum(om, FLT_MIN))
        a = np.zeros(m)
        for k in range(n - 1, -1, -1):
            mu, om, fl = recs[k]
            nxt = k < n - 1
            mubar = sbar - (np.where(fl, 0.0, a / om) if nxt else 0.0)
            others = np.array([np.delete(mu * mubar, i).sum() for i in range(m)])
            soft = mu / tau * (om * sbar - others)
            keep = (om + (tau - 1.0)) / tau
            if not slip:
                keep = np.where(fl, 1.0, keep)
            a = (a * keep if nxt else 0.0) + soft
        return a

    kappa, n, tau = [100.0, 0.0, 0.5, -1.0], 3, 1.0
    sbar = np.random.default_rng(37).normal(size=4)
    ref = mp_floored_gradient(kappa, n, tau, sbar)
    tol = dict(rtol=1e-9, atol=1e-12 * np.abs(sbar).max())
    assert np.allclose(sweep(kappa, n, tau, sbar, slip=False), ref, **tol)
    assert np.allclose(oracle.relax_bwd(np.array(kappa), n, tau, sbar), ref, **tol)
    assert not np.allclose(sweep(kappa, n, tau, sbar, slip=True), ref, **tol)


def test_backward_uniform_upstream_is_zero():
    """sum_j S_j = N for every kappa, so a constant upstream gradient has zero
    derivative."""
    rng = np.random.default_rng(23)
    for _ in range(300):
        m = int(rng.choice([4, 8, 16, 32]))
        n = int(rng.integers(1, m + 1))
        tau = float(rng.choice([0.1, 0.5, 1.0]))
        kappa = rng.normal(scale=2, size=m)
        c = float(rng.normal())
        d = oracle.relax_bwd(kappa, n, tau, np.full(m, c))
        assert np.abs(d).max() <= 1e-12 * abs(c) * m / tau


# --------------------------------------------------------------------------- whole arrays
def test_fwd_outputs_consistent():
    rng = np.random.default_rng(29)
    m, n = 4, 2
    numel = 4096
    W = (rng.normal(scale=0.02, size=numel).astype(np.float32).view(np.uint32) >> 16).astype(
        np.uint16)
    W[::7] = 0x8000  # some -0.0 weights
    phi = rng.normal(size=numel).astype(np.float32)
    Wm, S, idx = oracle.mask_fwd(W, phi, n, m, 0.5, 1.0, 1, 2, 64)
    hard = np.zeros((numel // m, m), dtype=bool)
    np.put_along_axis(hard, idx.astype(np.int64), True, axis=1)
    assert np.all(hard.sum(1) == n)
    assert np.array_equal(Wm, np.where(hard.reshape(-1), W, np.uint16(0)))
    assert np.allclose(S.reshape(-1, m).sum(1), n, atol=1e-12)
    kappa = oracle.keys(phi, 1.0, 1, 2, 64).reshape(-1, m)
    for q in range(0, numel // m, 97):
        order, _ = oracle.topn(kappa[q], n)
        assert list(order) == list(idx[q])
        assert np.allclose(S.reshape(-1, m)[q], oracle.relax_fwd(kappa[q].astype(np.float64), n,
                                                                 0.5), rtol=1e-15)


def test_groups_entry_matches_contiguous():
    rng = np.random.default_rng(31)
    m, n, numel = 8, 4, 8 * 300
    W = rng.integers(0, 65536, numel).astype(np.uint16)
    W = np.where((W & 0x7F80) == 0x7F80, np.uint16(0x3F80), W)  # no inf/nan patterns
    phi = rng.normal(size=numel).astype(np.float32)
    G = rng.integers(0, 65536, numel).astype(np.uint16)
    G = np.where((G & 0x7F80) == 0x7F80, np.uint16(0x3F80), G)
    off = 4 * 12345
    Wm, S, idx = oracle.mask_fwd(W, phi, n, m, 0.7, 1.3, 5, 6, off)
    d = oracle.mask_bwd(G, W, phi, n, m, 0.7, 1.3, 5, 6, off)
    sel = np.array([3, 0, 299, 150])
    ge = off + sel * m
    Wg, Sg, ig = oracle.mask_fwd_groups(W.reshape(-1, m)[sel], phi.reshape(-1, m)[sel], ge, n, m,
                                        0.7, 1.3, 5, 6)
    dg = oracle.mask_bwd_groups(G.reshape(-1, m)[sel], W.reshape(-1, m)[sel],
                                phi.reshape(-1, m)[sel], ge, n, m, 0.7, 1.3, 5, 6)
    assert np.array_equal(Wg, Wm.reshape(-1, m)[sel])
    assert np.array_equal(ig, idx[sel])
    assert np.array_equal(Sg, S.reshape(-1, m)[sel])
    assert np.array_equal(dg, d.reshape(-1, m)[sel])


@pytest.mark.parametrize("threads", [2, 3, 7, 16])
def test_threaded_oracle_is_the_scalar_oracle(threads):
    """The threaded entry points only split the groups over threads: the same
    bits as the scalar loop for any thread count, including more threads than
    groups and a ragged split."""
    rng = np.random.default_rng(41 + threads)
    for m, n, groups, tau, lam in [(4, 2, 1001, 1.0, 1.0), (8, 4, 13, 0.5, 0.7),
                                   (32, 16, 5, 1.0, 1.0), (16, 8, 2, 0.3, 1.0)]:
        numel = m * groups
        W = (rng.normal(0, 0.02, numel).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        G = (rng.normal(0, 1e-3, numel).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        phi = rng.normal(size=numel).astype(np.float32)
        off = 4 * 777
        ref = oracle.mask_fwd(W, phi, n, m, tau, lam, 9, 4, off)
        got = oracle.mask_fwd(W, phi, n, m, tau, lam, 9, 4, off, threads=threads)
        for a, b in zip(ref, got):
            assert np.array_equal(a, b)
        d_ref = oracle.mask_bwd(G, W, phi, n, m, tau, lam, 9, 4, off)
        d_got = oracle.mask_bwd(G, W, phi, n, m, tau, lam, 9, 4, off, threads=threads)
        assert np.array_equal(d_ref, d_got)
        kappa = rng.normal(scale=2.0, size=(groups, m))
        sbar = rng.normal(size=(groups, m))
        many = oracle.relax_bwd_groups(kappa, n, tau, sbar, threads=threads)
        for q in range(groups):
            assert np.array_equal(many[q], oracle.relax_bwd(kappa[q], n, tau, sbar[q]))


def test_bwd_chains_straight_through_and_lambda():
    """dL/dphi = (1/lambda) dS/dkappa^T (G (.) W): the straight-through backward
    treats W_masked as W (.) S."""
    rng = np.random.default_rng(37)
    m, n, numel = 4, 2, 64
    Wf = rng.normal(scale=0.5, size=numel).astype(np.float32)
    Gf = rng.normal(size=numel).astype(np.float32)
    W = (Wf.view(np.uint32) >> 16).astype(np.uint16)
    G = (Gf.view(np.uint32) >> 16).astype(np.uint16)
    phi = rng.normal(size=numel).astype(np.float32)
    lam = float(np.float32(0.8))  # the oracle takes fp32 temperatures
    tau = float(np.float32(0.9))
    d = oracle.mask_bwd(G, W, phi, n, m, tau, lam, 2, 3, 0)
    kappa = oracle.keys(phi, lam, 2, 3, 0).astype(np.float64).reshape(-1, m)
    Wd = (W.astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(-1, m)
    Gd = (G.astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(-1, m)
    for q in range(numel // m):
        ref = oracle.relax_bwd(kappa[q], n, tau, Gd[q] * Wd[q]) / lam
        assert np.allclose(d.reshape(-1, m)[q], ref, rtol=1e-15, atol=0)


def test_argument_checks():
    W = np.zeros(8, dtype=np.uint16)
    phi = np.zeros(8, dtype=np.float32)
    for bad in [dict(n=0, m=4), dict(n=5, m=4), dict(n=2, m=3)]:
        with pytest.raises(ValueError):
            oracle.mask_fwd(W, phi, bad["n"], bad["m"], 1.0, 1.0, 0, 0)
    with pytest.raises(ValueError):
        oracle.mask_fwd(W, phi, 2, 4, 0.0, 1.0, 0, 0)
    with pytest.raises(ValueError):
        oracle.mask_fwd(W, phi, 2, 4, 1.0, -1.0, 0, 0)


# --------------------------------------------------------------------------- annealing
def test_anneal_schedule_paper_hyperparameters():
    """§4.2.3 exponential annealing with the appendix's settings: starts at
    the initial value, reaches the final value at T_anneal, stays there, and
    decays by a constant ratio per step."""
    hp = json.load(open(os.path.join(HERE, "golden", "hyperparameters.json")))
    T = hp["t_anneal"]
    for a, b in ((hp["tau_init"], hp["tau_end"]), (hp["lambda_init"], hp["lambda_end"])):
        vals = np.array([oracle.anneal(a, b, t, T) for t in range(hp["training_steps"] + 1)])
        assert vals[0] == a
        assert math.isclose(vals[T], b, rel_tol=1e-12)
        assert np.all(vals[T:] == b) or np.allclose(vals[T:], b, rtol=1e-12)
        ratios = vals[1:T] / vals[: T - 1]
        assert np.allclose(ratios, (b / a) ** (1.0 / T), rtol=1e-10)
    # 10-step schedule from 1.0 to 0.1 reaching 0.1 at the last step
    taus = [oracle.anneal(1.0, 0.1, t, 9) for t in range(10)]
    assert taus[0] == 1.0 and math.isclose(taus[9], 0.1, rel_tol=1e-12)


# --------------------------------------------------------------------------- AdamW on the logits
def _torch_adamw_step(phi, m, v, g, lr, b1, b2, eps, wd, t):
    """One step of PyTorch's AdamW (fp64, CPU) from an explicit state."""
    import torch
    p = torch.tensor(np.asarray(phi, np.float64), requires_grad=True)
    opt = torch.optim.AdamW([p], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd, foreach=False)
    opt.state[p] = {"step": torch.tensor(float(t - 1), dtype=torch.float64),
                    "exp_avg": torch.tensor(np.asarray(m, np.float64)),
                    "exp_avg_sq": torch.tensor(np.asarray(v, np.float64))}
    p.grad = torch.tensor(np.asarray(g, np.float64))
    opt.step()
    st = opt.state[p]
    return p.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()


@pytest.mark.parametrize("t,lr", [(1, 1e-3), (2, 1e-3), (7, 5e-4), (100, 2e-4), (1500, 1e-4)])
def test_adamw_matches_torch(t, lr):
    """The oracle's AdamW step against PyTorch's AdamW implementation (fp64) on
    random states, with the appendix's betas and weight decay."""
    rng = np.random.default_rng(t)
    n = 4096
    phi = rng.normal(0, 1, n).astype(np.float32)
    m = (rng.normal(0, 1e-4, n)).astype(np.float32)
    v = (rng.random(n) * 1e-8).astype(np.float32)
    g = rng.normal(0, 1e-4, n)
    got = oracle.adamw(g, phi, m, v, lr, 0.9, 0.95, 1e-8, 0.05, t)
    ref = _torch_adamw_step(phi, m, v, g, lr, 0.9, 0.95, 1e-8, 0.05, t)
    for a, b in zip(got, ref):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-18)


def test_adamw_closed_forms():
    """From a zero state at t = 1 the step is phi (1 - lr wd) - lr g / (|g| + eps);
    a zero gradient with zero moments only decays; lr = 0 changes nothing."""
    rng = np.random.default_rng(11)
    phi = rng.normal(0, 1, 1000).astype(np.float32)
    g = rng.normal(0, 1e-3, 1000)
    z = np.zeros(1000, np.float32)
    lr, wd, eps = 1e-3, 0.05, 1e-8
    p, m, v = oracle.adamw(g, phi, z, z, lr, 0.9, 0.95, eps, wd, 1)
    phi64 = phi.astype(np.float64)
    np.testing.assert_allclose(p, phi64 * (1 - lr * wd) - lr * g / (np.abs(g) + eps), rtol=1e-14)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-14)
    np.testing.assert_allclose(v, 0.05 * g * g, rtol=1e-14)
    p, _, _ = oracle.adamw(np.zeros(1000), phi, z, z, lr, 0.9, 0.95, eps, wd, 5)
    np.testing.assert_allclose(p, phi64 * (1 - lr * wd), rtol=1e-15)
    m0 = rng.normal(0, 1, 1000).astype(np.float32)
    v0 = rng.random(1000).astype(np.float32)
    p, m, v = oracle.adamw(g, phi, m0, v0, 0.0, 0.9, 0.95, eps, wd, 3)
    np.testing.assert_array_equal(p, phi.astype(np.float64))
    with pytest.raises(ValueError):
        oracle.adamw(g, phi, z, z, lr, 0.9, 0.95, eps, wd, 0)


# --------------------------------------------------------------------------- final-mask export
def test_export_worked_example():
    """Hand-computed: phi = (0.1, 0.9, 0.5, 0.2) keeps {1, 2} (nibble 1 | 2 << 2 = 9);
    phi = (3, 3, 1, 3) ties at 3 and keeps the lower indices {0, 1} (nibble 4,
    in bits 4..7): one metadata word 9 + 64 = 73."""
    phi = np.array([0.1, 0.9, 0.5, 0.2, 3, 3, 1, 3], np.float32)
    W = np.arange(1, 9, dtype=np.uint16)
    Wm, vals, idx, meta = oracle.export(phi, W, 2, 4, want_meta=True)
    assert Wm.tolist() == [0, 2, 3, 0, 5, 6, 0, 0]
    assert vals.tolist() == [[2, 3], [5, 6]] and idx.tolist() == [[1, 2], [0, 1]]
    assert meta.tolist() == [73]


def decompress(vals, idx, m):
    """Dense [G, m] from the compressed values and their indices."""
    G, n = vals.shape
    dense = np.zeros((G, m), dtype=vals.dtype)
    np.put_along_axis(dense, idx.astype(np.int64), vals, axis=1)
    return dense.reshape(-1)


@pytest.mark.parametrize("n,m", [(2, 4), (1, 4), (3, 4), (4, 8), (2, 8), (8, 16), (16, 32)])
def test_export_is_the_lambda_to_zero_limit_of_the_sampler(n, m):
    """§4.2.3 anneals lambda towards 0.  With lambda = 2^-40 and |phi| >= 2^-10,
    phi / lambda is exact and one ulp of it exceeds twice any |g|, so the
    sampler's keys equal phi * 2^40 exactly: its selection (ties included) must
    be the exported top-n of the logits, and its masked weights the exported
    dense mask."""
    rng = np.random.default_rng(n * 64 + m)
    G = 4000
    phi = rng.normal(0, 1, (G, m))
    phi = np.sign(phi) * np.maximum(np.abs(phi), 2.0 ** -10)
    phi[::3] = np.round(phi[::3] * 2) / 2 + 0.25  # many exact ties, all nonzero
    phi = phi.astype(np.float32).reshape(-1)
    W = rng.integers(1, 0x7F00, phi.size, dtype=np.uint16)
    Wm_s, _, idx_s = oracle.mask_fwd(W, phi, n, m, 1.0, 2.0 ** -40, 7, 3, 0, want_soft=False)
    Wm, vals, idx, meta = oracle.export(phi, W, n, m, want_meta=(n == 2 and m == 4))
    assert np.array_equal(np.sort(idx_s, axis=1), idx)
    assert np.array_equal(Wm_s, Wm)
    assert np.array_equal(decompress(vals, idx, m), Wm)
    if meta is not None:  # 2:4 metadata: two 2-bit fields per group, 8 groups per word
        q = np.arange(G)
        nib = (meta[q // 8] >> (4 * (q % 8))) & 0xF
        assert np.array_equal(np.stack([nib & 3, nib >> 2], axis=1), idx)


# --------------------------------------------------------------------------- categorical sampler
@pytest.mark.parametrize("n,m", [(1, 4), (2, 4), (3, 4), (4, 4), (1, 8), (2, 8), (4, 8), (7, 8)])
def test_cat_candidates_are_the_lexicographic_subsets(n, m):
    import itertools
    got = oracle.cat_candidates(n, m)
    ref = [sum(1 << j for j in comb) for comb in itertools.combinations(range(m), n)]
    assert got.tolist() == ref


@pytest.mark.parametrize("m", [4, 8])
def test_cat_with_one_kept_entry_is_the_item_sampler(m):
    """At n = 1 the candidates are the single entries, candidate c of group Q
    draws the noise of element m Q + c, and Gumbel-Softmax over one logit per
    entry is the item sampler's top-1 relaxation: both oracles must agree
    (choice, masked weights exactly; S and the gradient to rounding)."""
    rng = np.random.default_rng(m)
    G, off, tau, lam = 3000, 17, 0.4, 0.7
    bf = lambda x: (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    W = bf(rng.normal(0, 1, G * m))
    Gb = bf(rng.normal(0, 1, G * m))
    phi = rng.normal(0, 1, G * m).astype(np.float32)
    Wm_c, S_c, ch = oracle.cat_fwd(W, phi, 1, m, tau, lam, 5, 2, off)
    Wm_r, S_r, idx = oracle.mask_fwd(W, phi, 1, m, tau, lam, 5, 2, off * m)
    assert np.array_equal(ch, idx[:, 0]) and np.array_equal(Wm_c, Wm_r)
    np.testing.assert_allclose(S_c, S_r, rtol=1e-13, atol=1e-15)
    d_c = oracle.cat_bwd(Gb, W, phi, 1, m, tau, lam, 5, 2, off)
    d_r = oracle.mask_bwd(Gb, W, phi, 1, m, tau, lam, 5, 2, off * m)
    np.testing.assert_allclose(d_c, d_r, rtol=1e-10, atol=1e-12 * np.abs(d_r).max())


@pytest.mark.parametrize("n,m,lam", [(2, 4, 1.0), (2, 4, 0.5), (2, 8, 1.0), (4, 8, 1.0)])
def test_cat_choice_follows_softmax(n, m, lam):
    """Gumbel-max: the chosen candidate is distributed as softmax(alpha / lambda)."""
    from scipy.stats import chisquare
    rng = np.random.default_rng(n * 10 + m)
    C = oracle.cat_candidates(n, m).size
    a = rng.normal(0, 1, C).astype(np.float32)
    G = 200000 if C < 30 else 60000
    alpha = np.tile(a, G)
    W = np.ones(G * m, dtype=np.uint16)
    _, _, ch = oracle.cat_fwd(W, alpha, n, m, 1.0, lam, 11, 3, 0, want_soft=False)
    p = np.exp(a.astype(np.float64) / np.float32(lam))
    p /= p.sum()
    counts = np.bincount(ch, minlength=C)
    ok = p * G >= 5
    stat = chisquare(counts[ok], p[ok] * G * counts[ok].sum() / (p[ok] * G).sum())
    assert stat.pvalue > 1e-4


def test_cat_invariants_and_gradient():
    """S sums to n, lies in [0, 1], tends to the hard mask as tau -> 0; a uniform
    upstream gradient gives zero; the backward matches central differences of
    <sbar, S> in fp64."""
    rng = np.random.default_rng(3)
    bf = lambda x: (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    for n, m in ((2, 4), (2, 8), (4, 8)):
        C = oracle.cat_candidates(n, m).size
        G = 300
        alpha = rng.normal(0, 1, G * C).astype(np.float32)
        W = bf(rng.normal(0, 1, G * m))
        Wm, S, ch = oracle.cat_fwd(W, alpha, n, m, 0.6, 1.0, 4, 1, 9)
        np.testing.assert_allclose(S.reshape(G, m).sum(1), n, rtol=1e-12)
        assert S.min() >= 0 and S.max() <= 1 + 1e-12
        _, S0, ch0 = oracle.cat_fwd(W, alpha, n, m, 1e-4, 1.0, 4, 1, 9)
        hard = (Wm != 0).reshape(G, m)
        np.testing.assert_allclose(S0.reshape(G, m)[::7], hard[::7], atol=1e-6)
        one = np.full(G * m, 0x3F80, np.uint16)  # bf16 1.0 for W and G: sbar = 1
        d = oracle.cat_bwd(one, one, alpha, n, m, 0.6, 1.0, 4, 1, 9)
        assert np.abs(d).max() < 1e-12
        # central differences of L(alpha) = <sbar, S(alpha)> on a few groups,
        # divided by the actual change of the (fp32) key of that candidate
        Gb = bf(rng.normal(0, 1, G * m))
        B = (C + 3) // 4
        sbar = ((Gb.astype(np.uint32) << 16).view(np.float32).astype(np.float64) *
                (W.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
        d = oracle.cat_bwd(Gb, W, alpha, n, m, 0.6, 1.0, 4, 1, 9)
        for q in (0, 17, 123):
            for c in (0, C // 2, C - 1):
                h = np.float32(2.0 ** -10)
                ap, am = alpha.copy(), alpha.copy()
                ap[q * C + c] += h
                am[q * C + c] -= h
                Sp = oracle.cat_fwd(W, ap, n, m, 0.6, 1.0, 4, 1, 9)[1]
                Sm = oracle.cat_fwd(W, am, n, m, 0.6, 1.0, 4, 1, 9)[1]
                e = 4 * B * (9 + q) + c
                kp = float(oracle.keys(ap[q * C + c:q * C + c + 1], 1.0, 4, 1, e)[0])
                km = float(oracle.keys(am[q * C + c:q * C + c + 1], 1.0, 4, 1, e)[0])
                fd = (sbar @ Sp - sbar @ Sm) / (kp - km)
                assert abs(fd - d[q * C + c]) <= 1e-4 * np.abs(d).max(), (n, m, q, c, fd)
