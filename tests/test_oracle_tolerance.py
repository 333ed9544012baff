"""Pins of the GEMM output bound |y - ref| <= 2^-8 |ref| + 1e-3 rms(ref)
(the oracle's gemm_tolerance and the test helper that applies it) against
hand-worked values: a wrong power of two, a mean in place of the rms, or an
rms over a row instead of the matrix fails one of them."""

import os

import numpy as np
import pytest

from oracle import mx_oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "gemm_tolerance_hand.txt")


def _cases():
    out = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        shape, ref, tol = (f.split() for f in line.split("|"))
        r, c = int(shape[0]), int(shape[1])
        out.append((np.array(ref, float).reshape(r, c), np.array(tol, float).reshape(r, c)))
    return out


CASES = _cases()


def test_fixture_has_cases():
    assert len(CASES) == 4


@pytest.mark.parametrize("ref,tol", CASES)
def test_hand_worked_bounds(ref, tol):
    got = O.gemm_tolerance(ref)
    assert got.shape == ref.shape
    np.testing.assert_allclose(got, tol, rtol=1e-12, atol=1e-15)


def test_bound_is_inclusive_and_tight():
    """The check passes an error equal to the bound (where the subtraction is
    exact: a zero reference) and errors just inside it, and fails an error
    just outside it, element by element and in both directions."""
    from tests.gpu_helpers import assert_gemm_close

    ref, tol = CASES[0]
    zero = ref == 0
    assert np.any(zero)
    assert_gemm_close(np.where(zero, tol, ref), ref)
    assert_gemm_close(np.where(zero, -tol, ref), ref)
    assert_gemm_close(ref + tol * (1 - 1e-9), ref)
    assert_gemm_close(ref - tol * (1 - 1e-9), ref)
    for i in range(ref.size):
        for sign in (1, -1):
            y = ref.copy().reshape(-1)
            y[i] += sign * tol.reshape(-1)[i] * (1 + 1e-9)
            with pytest.raises(AssertionError):
                assert_gemm_close(y.reshape(ref.shape), ref)
