"""Host-side checks of the GPU tests' own helpers (no GPU needed)."""
import numpy as np
import pytest

from tests.gpu_helpers import bf16_rne_bits, soft_product_exact


def _torch_bf16_bits(x):
    import torch
    t = torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_bf16_rounding_matches_torch():
    """The host rounding used to check W_soft is round to nearest, ties to
    even: equal to torch's float32 -> bfloat16 conversion on random values,
    on exact ties (both parities of the kept bit), on values one fp32 ulp to
    either side of a tie, and at the ends of the range."""
    rng = np.random.default_rng(7)
    x = np.concatenate([rng.standard_normal(200000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 200000),
                        rng.standard_normal(1000).astype(np.float32)])
    hi = rng.integers(0, 1 << 16, 4096, dtype=np.uint32) & 0x7F7F  # finite patterns
    ties = ((hi << 16) | 0x8000).view(np.float32)                 # exactly halfway
    below = ((hi << 16) | 0x7FFF).view(np.float32)
    above = ((hi << 16) | 0x8001).view(np.float32)
    ends = np.array([0.0, -0.0, 1e-45, -1e-45, 1.1754942e-38, 3.3895e38, -3.3895e38,
                     3.4028235e38], dtype=np.float32)
    for v in (x, ties, -ties, below, above, ends):
        assert np.array_equal(bf16_rne_bits(v), _torch_bf16_bits(v))


def test_soft_product_check_rejects_truncation():
    """The exact W_soft check accepts the rounded product and rejects the
    truncated one (a planted slip)."""
    rng = np.random.default_rng(3)
    W = (rng.standard_normal(4096).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    S = rng.random(4096).astype(np.float32)
    w = (W.astype(np.uint32) << 16).view(np.float32)
    prod = w * S
    soft_product_exact(W, S, bf16_rne_bits(prod), "rounded")
    truncated = (prod.view(np.uint32) >> 16).astype(np.uint16)
    assert not np.array_equal(truncated, bf16_rne_bits(prod))
    with pytest.raises(AssertionError):
        soft_product_exact(W, S, truncated, "truncated")
