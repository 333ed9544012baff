"""Pins for the oracle's offline calibration (Sec. 3.1 "Offline Channel
Assignment Strategy", Def. 1 eq. quantization-threshold, Appendix
"Derivations"): closed-form thresholds, a hand-built case whose groups are
known, invariance under exact power-of-two scaling, stability of the sort, and
a brute force with exact rationals."""

from fractions import Fraction

import numpy as np
import pytest

from oracle import mx_oracle as O
from paper_2508_02343_amd import workloads as W
from tests.calib_cases import boundary_case


def test_thresholds_closed_form():
    # T(4) = 2^1 * 2^3 / 6 * t/254 = (8/3) t/254 ;  T(6) = 2^3 * 2^5 / 28 * t/254 = (64/7) t/254
    for t in (1.0, 254.0, 1000.0, 2.0 ** -20):
        assert O.quantization_threshold(O.E2M1, t) == pytest.approx(8 / 3 * t / 254, rel=1e-15)
        assert O.quantization_threshold(O.E3M2, t) == pytest.approx(64 / 7 * t / 254, rel=1e-15)


def _bits(a):
    return W.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def test_hand_built_groups():
    """t = max|X| = 127: T(4) = 4/3, T(6) = 32/7 ~ 4.571.  Channels with mean
    1 go to G4, mean 3 to G6, mean 12 to G8 (32 of each, shuffled)."""
    rng = np.random.default_rng(0)
    K = 96
    means = np.repeat([1.0, 3.0, 12.0], 32)
    order = rng.permutation(K)
    m = means[order]
    x = np.stack([m * 0.5, m * 1.5])  # two rows: mean |x| = m
    x[1, order.tolist().index(64)] = 127.0  # the tensor's max, in a mean-12 channel (its mean becomes 33.5)
    sigma, split = O.calibrate(_bits(x))
    assert split == (32, 32, 32)
    M = np.abs(x).mean(axis=0)
    assert np.all(np.diff(M[sigma]) >= 0)
    assert set(sigma[:32]) == set(np.flatnonzero(M == 1.0))
    assert set(sigma[32:64]) == set(np.flatnonzero(M == 3.0))


def test_rounding_to_blocks_moves_channels_up():
    """40 channels under T(4), 20 between, 36 above: p4 = 32 and
    p4 + p6 = 32 * floor(60/32) = 32, so G6 is empty and 64 channels go to G8."""
    rng = np.random.default_rng(1)
    m = np.concatenate([np.full(40, 1.0), np.full(20, 3.0), np.full(36, 12.0)])
    x = np.stack([m, m])
    x[0, 95] = 127.0
    assert O.calibrate(_bits(x[:, rng.permutation(96)]))[1] == (32, 0, 64)


def test_power_of_two_scaling_invariance():
    w = W.LLAMA_ATTN
    xb = w.x_bits(64)
    s0, p0 = O.calibrate(xb)
    for k in (-7, 3):
        xs = O.f64_to_bf16_bits(O.bf16_bits_to_f64(xb) * 2.0 ** k)
        s, p = O.calibrate(xs)
        assert np.array_equal(s, s0) and p == p0


def test_equal_means_keep_index_order():
    x = np.ones((3, 64), np.float32)
    x[:, 5] = 4.0
    sigma, _ = O.calibrate(_bits(x))
    assert list(sigma[:63]) == [j for j in range(64) if j != 5] and sigma[63] == 5


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_brute_force_rationals(seed):
    rng = np.random.default_rng(seed)
    L, K = 5, 64
    x = (rng.standard_normal((L, K)) * np.exp2(rng.integers(-2, 6, K))).astype(np.float32)
    bits = _bits(x)
    xf = [[Fraction(float(v)) for v in row] for row in O.bf16_bits_to_f64(bits)]
    M = [sum(abs(xf[i][j]) for i in range(L)) / L for j in range(K)]
    t = max(abs(v) for row in xf for v in row)
    T4 = Fraction(2) * 8 / 6 * t / 254
    T6 = Fraction(8) * 32 / 28 * t / 254
    n4 = sum(1 for v in M if v <= T4)
    n6 = sum(1 for v in M if T4 < v <= T6)
    expect_split = (n4 // 32 * 32, (n4 + n6) // 32 * 32 - n4 // 32 * 32, K - (n4 + n6) // 32 * 32)
    expect_sigma = sorted(range(K), key=lambda j: (M[j], j))
    sigma, split = O.calibrate(bits)
    assert list(sigma) == expect_sigma
    assert split == expect_split


def test_rejects_bad_input():
    with pytest.raises(ValueError):
        O.calibrate(np.zeros((0, 32), np.uint16))
    with pytest.raises(ValueError):
        O.calibrate(np.zeros((2, 40), np.uint16))


def test_e2m3_threshold_uses_its_own_constants():
    # E2M3: b = 1, q_max = 7.5 -> T(6) = 2 * 32 / 7.5 * t/254 = (64/7.5) t/254, below E3M2's (64/7) t/254
    assert O.quantization_threshold(O.E2M3, 254.0) == pytest.approx(64 / 7.5, rel=1e-15)
    m = np.concatenate([np.full(32, 1.0), np.full(32, 8.8), np.full(32, 20.0)])
    x = np.stack([m, m])
    x[0, 95] = 254.0  # t = 254: T(4) = 8/3, T(6) = 64/7 ~ 9.14 (E3M2) or 8.53 (E2M3)
    assert O.calibrate(_bits(x))[1] == (32, 32, 32)
    assert O.calibrate(_bits(x), (O.E2M1, O.E2M3, O.E4M3))[1] == (32, 0, 64)


def test_means_exactly_at_the_thresholds_take_the_narrower_group():
    x = boundary_case()
    M = O.channel_abs_mean(_bits(x))
    assert M[31] == O.quantization_threshold(O.E2M1, 254.0) == 8 / 3
    assert M[63] == O.quantization_threshold(O.E3M2, 254.0) == 64 / 7
    assert O.calibrate(_bits(x))[1] == (32, 32, 32)
    # nudging either boundary channel up by one bf16 step moves the block boundary
    y = x.copy()
    y[20, 31] = 16.125
    assert O.calibrate(_bits(y))[1] == (0, 64, 32)
    y = x.copy()
    y[20, 63] = 32.25
    assert O.calibrate(_bits(y))[1] == (32, 0, 64)


def test_subnormal_channels_are_not_flushed():
    from tests.calib_cases import subnormal_case

    bits = subnormal_case()
    M = O.channel_abs_mean(bits)
    assert M[5] == 2.0 ** -133 and M[9] == 2.0 ** -126
    sigma, split = O.calibrate(bits)
    assert list(sigma) == [j for j in range(32) if j not in (5, 9)] + [5, 9]
    assert split == (0, 0, 32)  # 31 channels at or below T(4): rounds down to 0
