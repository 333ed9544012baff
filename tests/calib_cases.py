"""Hand-built calibration inputs shared by the oracle pins and the GPU tests
(inputs only: no arithmetic of the method)."""

import numpy as np

from paper_2508_02343_amd import workloads as W


def f32_bits(a) -> np.ndarray:
    return W.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def boundary_case() -> np.ndarray:
    """float32 [21, 96] with max|X| = 254 (so max|X|/254 = 1): channel 31
    sums to 56, mean fl(56/21) = fl(8/3) = T(4) of E2M1; channel 63 sums to
    192, mean fl(64/7) = T(6) of E3M2.  Every partial sum is a small integer,
    exact in any order.  Channels 0-30 have mean 1, 32-62 mean 5, 64-95 mean
    20 (channel 95 holds the 254)."""
    L = 21
    x = np.zeros((L, 96), np.float32)
    x[:, :31] = 1.0
    x[:20, 31], x[20, 31] = 2.0, 16.0
    x[:, 32:63] = 5.0
    x[:20, 63], x[20, 63] = 8.0, 32.0
    x[:, 64:] = 20.0
    x[0, 95] = 254.0
    return x


def subnormal_case() -> np.ndarray:
    """bf16 bits [6, 32]: channel 5 holds the smallest subnormal (2^-133)
    in every row, channel 9 the smallest normal (2^-126), the rest zeros.
    Zero channels sort first (in index order), then 5, then 9; flushing
    subnormals to zero would tie channel 5 with the zeros instead."""
    x = np.zeros((6, 32), np.uint16)
    x[:, 5] = 0x0001
    x[:, 9] = 0x8080  # -2^-126: the sign does not matter
    return x
