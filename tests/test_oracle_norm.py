"""Pins for the oracle's RMSNorm (App. D.2, Fig. "precision-mapping"; reading
R14): a hand-worked row, the intermediate bf16 rounding, exact special cases,
scaling laws, and agreement with torch's float32 RMSNorm formula."""

import numpy as np
import pytest
import torch

from oracle import mx_oracle as O
from tests.calib_cases import f32_bits


def _vals(bits):
    return O.bf16_bits_to_f64(bits)


def test_hand_worked_row():
    # x = (3, 4, 0, 0): mean square 25/4, r = 1/2.5 = 0.4, fp32(0.4) = 13421773 * 2^-25;
    # 3 r = 40265319 * 2^-25 -> fp32 10066330 * 2^-23 = 1.20000005 -> bf16 154/128 = 1.203125;
    # 4 r = 1.60000002 (exact) -> bf16 205/128 = 1.6015625
    y = O.rmsnorm_bf16(f32_bits([[3, 4, 0, 0]]), f32_bits([1, 1, 1, 1]), 0.0)
    assert _vals(y).tolist() == [[1.203125, 1.6015625, 0.0, 0.0]]


def test_intermediate_bf16_rounding():
    # gamma 1.5: 1.5 * 1.203125 = 1.8046875 exactly (231/128); one rounding of
    # 1.5 * 1.20000005 would give 230/128 = 1.796875 instead
    y = O.rmsnorm_bf16(f32_bits([[3, 4, 0, 0]]), f32_bits([1.5, -2, 1, 1]), 0.0)
    assert _vals(y).tolist() == [[1.8046875, -3.203125, 0.0, 0.0]]


@pytest.mark.parametrize("c", [2.0 ** -20, 0.25, 1.0, 8.0, -64.0])
def test_constant_rows_give_gamma(c):
    # mean square c^2, r = 1/|c| exactly (a power of two), x r = sign(c)
    rng = np.random.default_rng(3)
    g = f32_bits(rng.standard_normal(96).astype(np.float32))
    y = O.rmsnorm_bf16(f32_bits(np.full((2, 96), c, np.float32)), g, 0.0)
    want = g if c > 0 else g ^ np.uint16(0x8000)
    assert np.array_equal(y[0], want) and np.array_equal(y[1], want)


def test_power_of_two_scaling():
    rng = np.random.default_rng(4)
    x = f32_bits(rng.standard_normal((5, 128)).astype(np.float32))
    g = f32_bits(rng.standard_normal(128).astype(np.float32))
    y = O.rmsnorm_bf16(x, g, 0.0)
    for k in (-9, 5):
        xs = O.f64_to_bf16_bits(_vals(x) * 2.0 ** k)
        assert np.array_equal(O.rmsnorm_bf16(xs, g, 0.0), y)  # the norm removes the scale exactly
    g2 = O.f64_to_bf16_bits(_vals(g) * 4.0)
    assert np.array_equal(_vals(O.rmsnorm_bf16(x, g2, 0.0)), 4.0 * _vals(y))


def test_eps_dominates_zero_rows():
    # an all-zero row stays zero; eps keeps the factor finite
    y = O.rmsnorm_bf16(np.zeros((1, 64), np.uint16), f32_bits(np.ones(64)), 1e-6)
    assert not np.any(_vals(y))


def test_matches_torch_float32_formula():
    """torch's float32 RMSNorm, as bf16 frameworks write it: mean of squares
    and rsqrt in float32 (their rounding can differ from the float64 factor
    by an ulp), the product cast to bf16, times the weight, cast again."""
    rng = np.random.default_rng(5)
    L, K, eps = 64, 4096, 1e-5
    x = (rng.standard_normal((L, K)) * np.exp(rng.normal(0, 1, K))).astype(np.float32)
    g = (1 + 0.1 * rng.standard_normal(K)).astype(np.float32)
    xb, gb = f32_bits(x), f32_bits(g)
    xt = torch.from_numpy(xb.view(np.int16)).view(torch.bfloat16)
    gt = torch.from_numpy(gb.view(np.int16)).view(torch.bfloat16)
    h = xt.float()
    h = h * torch.rsqrt(h.pow(2).mean(-1, keepdim=True) + eps)
    ref = (gt * h.to(torch.bfloat16)).view(torch.int16).numpy().view(np.uint16)
    ours = O.rmsnorm_bf16(xb, gb, eps)
    diff = np.abs(ours.astype(np.int32) - ref.astype(np.int32))
    assert diff.max() <= 2  # a one-ulp factor difference can move each of the two roundings
    assert np.mean(diff == 0) > 0.99

