"""Pins for the oracle's block scale, reorder, packing and mixed GEMM.

Checks against invariants of the MX rule (Sec. 2.1), the quantisation-error
bound (Sec. 2.1, eq. "quantization-error", with |gamma| <= 1/2 grid step), an
independent brute-force quantiser with exact rational arithmetic, torch's
float8 decoding, and hand-computed bit layouts.
"""

import math
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import mx_oracle as O
from paper_2508_02343_amd import workloads as W


def _rand_blocks(rng, R, nblk, spread=12):
    x = rng.standard_normal((R, nblk * 32)) * np.exp2(rng.integers(-spread, spread, (R, nblk))).repeat(32, 1)
    return x


@pytest.mark.parametrize("name", ["E2M1", "E3M2", "E2M3", "E4M3", "E5M2"])
def test_scale_invariant_and_error_bound(name):
    f = O.FORMATS[name]
    rng = np.random.default_rng(5)
    x = _rand_blocks(rng, 64, 8)
    codes, e = O.quantize_blocks(x, f)
    amax = np.abs(x).reshape(64, 8, 32).max(2)
    # 2^(e+emax) <= amax < 2^(e+emax+1) whenever e is not clamped
    lo = np.exp2(e + f.emax)
    assert np.all(lo <= amax) and np.all(amax < 2 * lo)
    # |x - s*Q(x)| <= s * (grid step at |x/s|) / 2 unless |x/s| saturates
    dq = O.dequantize_blocks(codes, e, f)
    s = np.exp2(e).repeat(32, 1)
    v = np.abs(x) / s
    _, ex = np.frexp(v)
    step = np.exp2(np.maximum(ex - 1, f.emin) - f.mbits)
    unsat = v <= f.max_normal
    err = np.abs(x - dq)
    assert np.all(err[unsat] <= 0.5 * step[unsat] * s[unsat])
    assert np.all(np.abs(dq[~unsat]) == f.max_normal * s[~unsat])


@pytest.mark.parametrize("name", ["E2M1", "E3M2", "E4M3"])
def test_power_of_two_equivariance(name):
    f = O.FORMATS[name]
    rng = np.random.default_rng(6)
    x = _rand_blocks(rng, 16, 4, spread=4)
    c0, e0 = O.quantize_blocks(x, f)
    for k in (-9, -1, 1, 5, 40):
        ck, ek = O.quantize_blocks(np.ldexp(x, k), f)
        np.testing.assert_array_equal(ck, c0)
        np.testing.assert_array_equal(ek, e0 + k)


def test_zero_blocks():
    x = np.zeros((2, 64))
    x[1, :32] = -0.0
    x[1, 32:] = 1.0
    for f in (O.E2M1, O.E3M2, O.E4M3):
        c, e = O.quantize_blocks(x, f)
        assert e[0, 0] == -127 and e[0, 1] == -127 and e[1, 0] == -127
        assert np.all(c[0] == 0)
        assert np.all(c[1, :32] == 1 << (f.bits - 1))


def test_pack_layouts_hand():
    # FP4: even element in the low nibble
    assert O.pack_fp4(np.array([[0x1, 0x2, 0xF, 0x0]]))[0].tolist() == [0x21, 0x0F]
    # FP6: little-endian bit stream, code i at bits 6i..6i+5
    assert O.pack_fp6(np.array([[0x01, 0, 0, 0]]))[0].tolist() == [0x01, 0, 0]
    assert O.pack_fp6(np.array([[0, 0x01, 0, 0]]))[0].tolist() == [0x40, 0, 0]
    assert O.pack_fp6(np.array([[0, 0, 0x3F, 0]]))[0].tolist() == [0, 0xF0, 0x03]
    assert O.pack_fp6(np.array([[0, 0, 0, 0x3F]]))[0].tolist() == [0, 0, 0xFC]
    rng = np.random.default_rng(1)
    c6 = rng.integers(0, 64, (3, 64))
    np.testing.assert_array_equal(O.unpack_fp6(O.pack_fp6(c6), 64), c6)
    c4 = rng.integers(0, 16, (3, 64))
    np.testing.assert_array_equal(O.unpack_fp4(O.pack_fp4(c4), 64), c4)


def _rand_bf16(rng, shape, scale=1.0):
    return W.f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def test_reorder_is_gather_then_quantize():
    rng = np.random.default_rng(2)
    K = 256
    x = _rand_bf16(rng, (5, K))
    perm = rng.permutation(K).astype(np.int32)
    split = (128, 64, 64)
    a = O.quantize_mixed(x, perm, split)
    b = O.quantize_mixed(x[:, perm], np.arange(K), split)
    for f in ("q4", "q6", "q8", "sc"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    # with the identity permutation the groups are plain column slices
    xi = O.bf16_bits_to_f64(x)
    c4, _ = O.quantize_blocks(xi[:, :128], O.E2M1)
    np.testing.assert_array_equal(O.element_codes(O.quantize_mixed(x, np.arange(K), split))[0], c4)


def test_permuting_inside_a_block_permutes_codes():
    rng = np.random.default_rng(4)
    x = _rand_bf16(rng, (3, 96))
    split = (32, 32, 32)
    base = O.quantize_mixed(x, np.arange(96), split)
    inner = np.arange(96)
    for blk in range(3):
        inner[blk * 32:(blk + 1) * 32] = blk * 32 + rng.permutation(32)
    moved = O.quantize_mixed(x, inner, split)
    np.testing.assert_array_equal(moved.sc, base.sc)
    for cb, cm, lo in zip(O.element_codes(base), O.element_codes(moved), (0, 32, 64)):
        np.testing.assert_array_equal(cm, cb[:, inner[lo:lo + 32] - lo])


def test_split_and_perm_validation():
    x = np.zeros((1, 64), np.uint16)
    with pytest.raises(ValueError):
        O.quantize_mixed(x, np.arange(64), (32, 16, 16))
    with pytest.raises(ValueError):
        O.quantize_mixed(x, np.arange(64), (32, 32, 32))
    with pytest.raises(ValueError):
        O.quantize_mixed(x, np.zeros(64, np.int32), (64, 0, 0))


# ---- mixed GEMM ------------------------------------------------------------


def _quant_pair(rng, M, N, K, split, formats=O.PARTITION_FORMATS):
    perm = rng.permutation(K).astype(np.int32)
    xa = _rand_bf16(rng, (M, K))
    xa[:, perm[-32:]] = W.f32_to_bf16_bits(O.bf16_bits_to_f64(xa[:, perm[-32:]]).astype(np.float32) * 25)
    xw = _rand_bf16(rng, (N, K), 0.02)
    return (O.quantize_mixed(xa, perm, split, formats), O.quantize_mixed(xw, perm, split, formats), xa, xw,
            perm)


def test_gemm_is_sum_of_partition_gemms():
    rng = np.random.default_rng(8)
    K = 256
    split = (128, 64, 64)
    a, w, *_ = _quant_pair(rng, 7, 9, K, split)
    y = O.gemm_mixed(a, w)
    da, dw = O.dequantize_mixed(a), O.dequantize_mixed(w)
    parts = [da[:, lo:hi] @ dw[:, lo:hi].T for lo, hi in ((0, 128), (128, 192), (192, 256))]
    np.testing.assert_allclose(y, parts[0] + parts[1] + parts[2], rtol=1e-13, atol=1e-13)


def test_all_fp8_split_equals_plain_mxfp8_gemm_via_torch_decode():
    rng = np.random.default_rng(9)
    K = 128
    a, w, *_ = _quant_pair(rng, 6, 5, K, (0, 0, K))
    y = O.gemm_mixed(a, w)

    def torch_dq(t):
        vals = torch.from_numpy(np.ascontiguousarray(t.q8)).view(torch.float8_e4m3fn).double().numpy()
        e = t.sc.astype(np.int64) - 127
        return vals * np.exp2(e).repeat(32, 1)

    np.testing.assert_allclose(y, torch_dq(a) @ torch_dq(w).T, rtol=1e-13, atol=0)


def test_all_fp4_split_matches_e2m1_lookup_gemm():
    rng = np.random.default_rng(10)
    K = 128
    a, w, *_ = _quant_pair(rng, 4, 3, K, (K, 0, 0))
    lut = [0, 0.5, 1, 1.5, 2, 3, 4, 6]

    def dq(t):
        lo = t.q4 & 0xF
        hi = t.q4 >> 4
        codes = np.empty((t.rows, K), np.int64)
        codes[:, 0::2], codes[:, 1::2] = lo, hi
        mag = np.array(lut)[codes & 7] * np.where(codes & 8, -1, 1)
        return mag * np.exp2(t.sc.astype(np.int64) - 127).repeat(32, 1)

    np.testing.assert_allclose(O.gemm_mixed(a, w), dq(a) @ dq(w).T, rtol=1e-13, atol=0)


# Brute force: an independent quantiser (exhaustive nearest value, scale found
# by stepping powers of two) and an exact rational triple loop.

def _bf_scale(block, f):
    amax = max(abs(v) for v in block)
    if amax == 0:
        return -127
    t = 0
    while Fraction(2) ** t > amax:
        t -= 1
    while Fraction(2) ** (t + 1) <= amax:
        t += 1
    return max(-127, min(127, t - f.emax))


_VALS = {}


def _bf_value(v, f):
    if f.name not in _VALS:
        _VALS[f.name] = sorted((Fraction(f.decode(c)), c) for c in range(1 << (f.bits - 1))
                               if f.is_finite_code(c))
    vals = _VALS[f.name]
    a = abs(v)
    d = min(abs(a - q) for q, _ in vals)
    ties = [(q, c) for q, c in vals if abs(a - q) == d]
    # on a tie between two neighbours take the even code (mantissa LSB 0)
    best = ties[0][0] if len(ties) == 1 else [q for q, c in ties if c % 2 == 0][0]
    return best if v >= 0 else -best


def _bf_quantize(row, p, f):
    out = []
    for b in range(0, len(row), 32):
        blk = [Fraction(v) for v in row[b:b + 32]]
        e = _bf_scale(blk, f)
        s = Fraction(2) ** e
        out += [_bf_value(v / s, f) * s for v in blk]
    return out


@pytest.mark.parametrize("split", [(32, 0, 0), (0, 32, 0), (0, 0, 32)])
def test_brute_force_single_block_32x32(split):
    _brute_force_case(32, 32, 32, split, seed=sum(i * v for i, v in enumerate(split)))


def _brute_force_case(M, N, K, split, seed, fmts=(O.E2M1, O.E3M2, O.E4M3)):
    rng = np.random.default_rng(seed)
    a, w, xa, xw, perm = _quant_pair(rng, M, N, K, split, fmts)
    y = O.gemm_mixed(a, w)
    fa = O.bf16_bits_to_f64(xa)[:, perm]
    fw = O.bf16_bits_to_f64(xw)[:, perm]
    bounds = np.cumsum((0,) + tuple(split))

    def q(rowv):
        out = []
        for (lo, hi), f in zip(zip(bounds[:-1], bounds[1:]), fmts):
            out += _bf_quantize(rowv[lo:hi], hi - lo, f)
        return out

    qa = [q(fa[i]) for i in range(M)]
    qw = [q(fw[j]) for j in range(N)]
    for i in range(M):
        for j in range(N):
            exact = sum(x * z for x, z in zip(qa[i], qw[j]))
            assert abs(Fraction(y[i, j]) - exact) <= abs(exact) * Fraction(1, 2 ** 45) + Fraction(1, 2 ** 200)


@pytest.mark.parametrize("split", [(32, 0, 0), (0, 32, 0), (0, 0, 32), (64, 0, 32), (32, 32, 32), (0, 64, 32)])
def test_brute_force_small(split):
    K = sum(split)
    _brute_force_case(4, 3, K, split, seed=K + split[0])


@pytest.mark.parametrize("split", [(0, 32, 0), (0, 0, 32), (32, 32, 32), (0, 64, 32)])
def test_brute_force_small_alternative_formats(split):
    """The ablation's alternatives (MXFP6 as E2M3, MXFP8 as E5M2) through the
    same independent quantiser and exact triple loop."""
    K = sum(split)
    _brute_force_case(4, 3, K, split, seed=2 * K + split[1], fmts=(O.E2M1, O.E2M3, O.E5M2))


def test_all_fp8_e5m2_split_equals_plain_mxfp8_gemm_via_torch_decode():
    rng = np.random.default_rng(19)
    K = 128
    a, w, *_ = _quant_pair(rng, 6, 5, K, (0, 0, K), (O.E2M1, O.E3M2, O.E5M2))
    y = O.gemm_mixed(a, w)

    def torch_dq(t):
        vals = torch.from_numpy(np.ascontiguousarray(t.q8)).view(torch.float8_e5m2).double().numpy()
        return vals * np.exp2(t.sc.astype(np.int64) - 127).repeat(32, 1)

    np.testing.assert_allclose(y, torch_dq(a) @ torch_dq(w).T, rtol=1e-13, atol=0)


def test_all_fp6_e2m3_split_matches_closed_form_lookup_gemm():
    """E2M3 magnitudes from their closed form (bias 1): m/8 for exponent
    field 0, (1 + m/8) * 2^(E-1) otherwise; codes unpacked from the 24-byte
    little-endian stream by hand."""
    rng = np.random.default_rng(20)
    K = 64
    a, w, *_ = _quant_pair(rng, 4, 3, K, (0, K, 0), (O.E2M1, O.E2M3, O.E4M3))
    mag = [(m / 8 if E == 0 else (1 + m / 8) * 2.0 ** (E - 1)) for E in range(4) for m in range(8)]

    def dq(t):
        out = np.zeros((t.rows, K))
        for r in range(t.rows):
            bits = int.from_bytes(bytes(t.q6[r]), "little")
            for i in range(K):
                c = (bits >> (6 * i)) & 63
                out[r, i] = (-1 if c & 32 else 1) * mag[c & 31] * 2.0 ** (int(t.sc[r, i // 32]) - 127)
        return out

    np.testing.assert_allclose(O.gemm_mixed(a, w), dq(a) @ dq(w).T, rtol=1e-13, atol=0)


def test_group_formats_touch_only_their_group():
    rng = np.random.default_rng(21)
    split = (64, 64, 64)
    K = sum(split)
    x = _rand_bf16(rng, (5, K), 1.0)
    perm = rng.permutation(K).astype(np.int32)
    d = O.quantize_mixed(x, perm, split)
    v = O.quantize_mixed(x, perm, split, (O.E2M1, O.E2M3, O.E5M2))
    assert np.array_equal(d.q4, v.q4) and np.array_equal(d.sc[:, :2], v.sc[:, :2])
    # E2M3 has emax 2 (E3M2 4), E5M2 15 (E4M3 8): the scale bytes move by the difference
    # unless the clamp at -127 or the all-zero rule applies
    assert np.all(v.sc[:, 2:4].astype(int) - d.sc[:, 2:4] == 2)
    assert np.all(d.sc[:, 4:6].astype(int) - v.sc[:, 4:6] == 7)
    with pytest.raises(ValueError):
        O.quantize_mixed(x, perm, split, (O.E2M1, O.E4M3, O.E4M3))
    with pytest.raises(ValueError):
        O.gemm_mixed(d, v)


def test_average_bits_formula():
    # MicroMix stores (4 p4 + 6 p6 + 8 p8)/K bits per element plus 8/32 for the scale
    assert O.average_bits((3072, 768, 256)) == pytest.approx(4.625 + 0.25)
    assert O.average_bits((0, 0, 4096)) == 8.25
