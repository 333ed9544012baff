"""CPU check of the GPU norm test's handling of row factors near an fp32
rounding midpoint (the rows it compares against both fp32 candidates)."""

import numpy as np

from tests.test_gpu_norm import factor_candidates


def test_exact_fp32_values_have_one_candidate():
    r = np.array([1.0, 0.5, float(np.float32(0.1))])
    r32, alt, amb = factor_candidates(r, 4096)
    assert not amb.any() and np.array_equal(r32, alt)


def test_midpoints_get_the_other_neighbour():
    a = np.float32(1.25)
    up = np.nextafter(a, np.float32(2))
    mid = (float(a) + float(up)) / 2  # exactly representable in float64
    for r in (mid, np.nextafter(mid, 0.0), np.nextafter(mid, 2.0)):
        r32, alt, amb = factor_candidates(np.array([r]), 4096)
        assert amb[0]
        assert {float(r32[0]), float(alt[0])} == {float(a), float(up)}


def test_far_from_midpoints_is_unambiguous():
    a = np.float32(3.0)
    up = np.nextafter(a, np.float32(4))
    quarter = float(a) + (float(up) - float(a)) / 4  # a quarter step: far from both midpoints
    r32, alt, amb = factor_candidates(np.array([quarter]), 4096)
    assert not amb[0] and r32[0] == a
