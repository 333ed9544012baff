"""Pins for the oracle's MX element formats and its element encoder.

Each check ties the oracle to something other than itself: the constants the
paper prints (Appendix B, Table "tab:microscaling"), the closed-form value
sets of the OCP formats, torch's own float8 types (a library decode and RNE
cast), hand-worked blocks, and a brute-force nearest-value encoder written
independently here.
"""

import math
import os

import numpy as np
import pytest
import torch

from oracle import mx_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_formats():
    rows = []
    for line in open(os.path.join(GOLDEN, "mx_formats.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, eb, mb, bias, maxn = line.split()
        rows.append((name, int(eb), int(mb), int(bias), float(maxn)))
    return rows


@pytest.mark.parametrize("row", _golden_formats(), ids=lambda r: r[0])
def test_format_constants_match_paper_table(row):
    name, eb, mb, bias, maxn = row
    f = O.FORMATS[name]
    assert (f.ebits, f.mbits, f.bias) == (eb, mb, bias)
    assert f.max_normal == maxn


def test_emax_is_top_binade():
    # reading R1: emax = floor(log2(max normal))
    assert {n: f.emax for n, f in O.FORMATS.items()} == {
        "E2M1": 2, "E3M2": 4, "E2M3": 2, "E4M3": 8, "E5M2": 15}


def test_value_sets_closed_form():
    assert sorted(set(abs(v) for v in map(O.E2M1.decode, O.E2M1.finite_codes()))) == [
        0, 0.5, 1, 1.5, 2, 3, 4, 6]
    counts = {n: len(f.finite_codes()) for n, f in O.FORMATS.items()}
    assert counts == {"E2M1": 16, "E3M2": 64, "E2M3": 64, "E4M3": 254, "E5M2": 248}
    # smallest positive subnormal = 2^(emin - mbits)
    assert O.E3M2.decode(1) == 2.0 ** -4
    assert O.E2M3.decode(1) == 1 / 8
    assert O.E4M3.decode(1) == 2.0 ** -9
    assert O.E5M2.decode(1) == 2.0 ** -16
    # E2M3: step 1/8 below 2, then 1/4 on [2, 4) and 1/2 on [4, 8)
    pos = sorted(set(O.E2M3.decode(c) for c in range(32)))
    assert pos[:16] == [i / 8 for i in range(16)]
    assert pos[16:24] == [2 + i / 4 for i in range(8)]
    assert pos[24:] == [4 + i / 2 for i in range(8)]
    # E3M2 binade [1, 2) has step 1/4
    assert [O.E3M2.decode(c) for c in range(12, 16)] == [1.0, 1.25, 1.5, 1.75]


@pytest.mark.parametrize("name,tdt", [("E4M3", torch.float8_e4m3fn), ("E5M2", torch.float8_e5m2)])
def test_fp8_decode_matches_torch(name, tdt):
    f = O.FORMATS[name]
    codes = np.array(f.finite_codes(), dtype=np.uint8)
    ref = torch.from_numpy(codes).view(tdt).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.decode_codes(codes, f), ref)
    # signed zeros are kept apart
    assert math.copysign(1, O.decode_codes(np.array([0x80]), f)[0]) == -1


@pytest.mark.parametrize("name,tdt", [("E4M3", torch.float8_e4m3fn), ("E5M2", torch.float8_e5m2)])
def test_fp8_encode_matches_torch_rne_cast(name, tdt):
    f = O.FORMATS[name]
    rng = np.random.default_rng(7)
    # in-range values across every binade, plus exact midpoints
    v = rng.uniform(-1, 1, 20000) * np.exp2(rng.integers(-20, f.emax + 1, 20000))
    v = np.clip(v, -f.max_normal, f.max_normal)
    vals = np.array(sorted(set(f.decode(c) for c in f.finite_codes())))
    mids = (vals[:-1] + vals[1:]) / 2
    v = np.concatenate([v, mids, -mids])
    ours = O.encode_scaled(v, f)
    ref = torch.from_numpy(v).to(tdt).view(torch.uint8).numpy()
    np.testing.assert_array_equal(ours, ref)


def _brute_force_encode(v, f):
    """Nearest finite value by exhaustive search; ties go to the even code."""
    codes = [c for c in range(1 << (f.bits - 1)) if f.is_finite_code(c)]
    vals = [f.decode(c) for c in codes]
    out = []
    for x in np.asarray(v, dtype=np.float64):
        a = abs(x)
        best = None
        for c, val in zip(codes, vals):
            d = abs(a - val)
            if best is None or d < best[0] or (d == best[0] and c % 2 == 0):
                best = (d, c)
        c = best[1]
        if math.copysign(1.0, x) < 0:
            c |= 1 << (f.bits - 1)
        out.append(c)
    return np.array(out, dtype=np.uint8)


@pytest.mark.parametrize("name", list(O.FORMATS))
def test_rne_encoder_equals_brute_force(name):
    f = O.FORMATS[name]
    vals = np.array(sorted(set(abs(f.decode(c)) for c in f.finite_codes())))
    mids = (vals[:-1] + vals[1:]) / 2
    eps = np.ldexp(mids, -30)
    top = 2.0 ** (f.emax + 1)
    sat = np.linspace(f.max_normal, top * 0.999, 37)
    rng = np.random.default_rng(11)
    rand = rng.uniform(0, top, 300)
    sub = np.ldexp(rng.uniform(0, 1, 100), f.emin)
    v = np.concatenate([vals, mids, mids - eps, mids + eps, sat, rand, sub])
    v = np.concatenate([v, -v, [0.0, -0.0]])
    np.testing.assert_array_equal(O.encode_scaled(v, f), _brute_force_encode(v, f))


@pytest.mark.parametrize("name", list(O.FORMATS))
def test_exhaustive_round_trip(name):
    f = O.FORMATS[name]
    codes = np.array(f.finite_codes(), dtype=np.int64)
    back = O.encode_scaled(O.decode_codes(codes, f), f)
    np.testing.assert_array_equal(back, codes.astype(np.uint8))


def _hand_blocks():
    out = []
    for line in open(os.path.join(GOLDEN, "mx_blocks_hand.txt")):
        if line.startswith("#") or not line.strip():
            continue
        head, ins, codes = line.split("|")
        name, byte = head.split()
        xs = [float(t) for t in ins.split()]
        cs = [int(t, 16) for t in codes.split()]
        out.append((name, int(byte), xs, cs))
    return out


@pytest.mark.parametrize("case", _hand_blocks(), ids=lambda c: f"{c[0]}-{c[1]}-{len(c[2])}")
def test_hand_worked_blocks(case):
    name, byte, xs, cs = case
    f = O.FORMATS[name]
    x = np.zeros((1, 32))
    x[0, : len(xs)] = xs
    codes, e = O.quantize_blocks(x, f)
    assert int(e[0, 0]) + 127 == byte
    expect = np.zeros(32, dtype=np.uint8)
    expect[: len(cs)] = cs
    np.testing.assert_array_equal(codes[0], expect)


def test_bf16_helpers_match_torch():
    rng = np.random.default_rng(3)
    # float32 inputs, so that torch's conversion cannot double-round
    x = (rng.standard_normal(50000) * np.exp2(rng.integers(-130, 120, 50000))).astype(np.float32)
    x = x.astype(np.float64)
    ours = O.f64_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = O.bf16_bits_to_f64(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).double().numpy())
