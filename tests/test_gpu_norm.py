"""GPU parity of mm_rmsnorm_quantize_act (RMSNorm fused with the
reorder-and-quantize; App. D.2, Fig. "precision-mapping"; reading R14):
codes and scales byte-identical to the oracle's quantisation of its RMSNorm.

The row factor r = 1/sqrt(mean(x^2) + eps) is evaluated in float64 on both
sides but summed in different orders, so the two float64 values can differ in
the last places.  Both round r once to fp32; rows whose float64 factor lies
further than 4 K 2^-53 (relative) from an fp32 rounding midpoint get the same
fp32 factor on both sides and are compared byte for byte.  A row closer than
that (rare) is checked against the oracle's result with either neighbouring
fp32 factor, each evaluated exactly."""

import functools

import numpy as np
import pytest
import torch

from oracle import mx_oracle as O
from paper_2508_02343_amd import workloads as W
from tests.calib_cases import f32_bits
from tests.gpu_helpers import assert_codes_equal, assert_gemm_close, note, to_dev_bf16, to_dev_perm, y_to_f64
from tests import packed_layout as PL

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=None)
def _b():
    from paper_2508_02343_amd import binding

    return binding


def factor_candidates(r, K):
    """fp32 roundings of float64 row factors r, and for factors within
    4 K 2^-53 (relative) of an fp32 rounding midpoint the neighbour on the
    other side of that midpoint (else the same value)."""
    r = np.asarray(r, dtype=np.float64)
    r32 = r.astype(np.float32)
    up = np.nextafter(r32, np.float32(np.inf))
    dn = np.nextafter(r32, np.float32(0))
    mid_up = (r32.astype(np.float64) + up.astype(np.float64)) / 2
    mid_dn = (r32.astype(np.float64) + dn.astype(np.float64)) / 2
    tol = 4.0 * K * 2.0 ** -53 * r
    alt = np.where(np.abs(r - mid_up) <= tol, up, np.where(np.abs(r - mid_dn) <= tol, dn, r32))
    return r32, alt, alt != r32


def _factors(xb, eps):
    """fp32 row factors, and for rows near an fp32 midpoint the other candidate."""
    return factor_candidates(O.rmsnorm_row_factor(xb, eps), xb.shape[1])


def _run(xb, gb, eps, perm, split, formats=("E3M2", "E4M3"), ld_extra=0):
    x = to_dev_bf16(xb)
    if ld_extra:
        big = torch.zeros((x.shape[0], x.shape[1] + ld_extra), dtype=torch.bfloat16, device="cuda")
        big[:, : x.shape[1]] = x
        x = big[:, : xb.shape[1]]
    out = _b().rmsnorm_quantize_act(x, to_dev_bf16(gb), eps, to_dev_perm(perm), split, formats=formats)
    torch.cuda.synchronize()
    return out


def _check(xb, gb, eps, perm, split, formats=("E3M2", "E4M3"), ctx="", ld_extra=0):
    fm = (O.E2M1, O.FORMATS[formats[0]], O.FORMATS[formats[1]])
    r32, alt, amb = _factors(xb, eps)
    note(f"rmsnorm+quantize {ctx} rows={xb.shape[0]} K={xb.shape[1]} split={split} formats={formats} "
         f"eps={eps} near-midpoint rows={int(amb.sum())}")
    out = _run(xb, gb, eps, perm, split, formats, ld_extra)
    y = O.rmsnorm_apply(xb, gb, r32)
    if not amb.any():
        assert_codes_equal(out, O.quantize_mixed(y, perm, split, fm), ctx=ctx)
        return out, y
    ok = np.flatnonzero(~amb)
    if ok.size:
        assert_codes_equal(out, O.quantize_mixed(y[ok], perm, split, fm), rows=ok, ctx=ctx)
    got = PL.untile(out.raw_host(), out.rows, out.split)
    for i in np.flatnonzero(amb):
        matches = []
        for f in (r32[i], alt[i]):
            ref = O.quantize_mixed(O.rmsnorm_apply(xb[i : i + 1], gb, np.array([f], np.float32)), perm, split, fm)
            matches.append(all(np.array_equal(got[k][i], np.asarray(getattr(ref, k))[0])
                               for k in ("q4", "q6", "q8", "sc")))
        assert any(matches), f"{ctx}: row {i} matches neither fp32 factor"
    return out, y


def _gamma(K, seed):
    rng = np.random.default_rng([seed, 9])
    return f32_bits((1.0 + 0.25 * rng.standard_normal(K)).astype(np.float32))


RAGGED = [(96, 160, 96), (352, 0, 0), (0, 352, 0), (0, 0, 352), (32, 32, 288)]


@pytest.mark.parametrize("split", RAGGED)
@pytest.mark.parametrize("rows", [1, 37])
def test_ragged_shapes(split, rows):
    K = sum(split)
    rng = np.random.default_rng(rows * 100 + split[0])
    x = (rng.standard_normal((rows, K)) * np.exp2(rng.integers(-3, 4, (rows, K)))).astype(np.float32)
    _check(f32_bits(x), _gamma(K, rows), 1e-6, rng.permutation(K).astype(np.int32), split, ctx=str(split),
           ld_extra=24)


@pytest.mark.parametrize("K,split", [(32, (32, 0, 0)), (64, (32, 0, 32)), (512, (384, 64, 64))])
def test_narrow_rows_many_per_pass(K, split):
    # small K packs many rows into one pass (up to 256 row factors per pass)
    rng = np.random.default_rng(K)
    x = rng.standard_normal((700, K)).astype(np.float32)
    _check(f32_bits(x), _gamma(K, K), 1e-5, rng.permutation(K).astype(np.int32), split, ctx=f"K{K}")


@pytest.mark.parametrize("w,eps", [(W.LLAMA_ATTN, 1e-5), (W.QWEN_MLP_UP, 1e-6)])
def test_layer_widths(w, eps):
    # the hidden-state widths the norm feeds: 4096 (Llama-3.1-8B, eps 1e-5) and
    # 5120 (Qwen2.5-32B, eps 1e-6), with the workloads' outlier channels
    rows = 2048 if w is W.LLAMA_ATTN else 300
    _check(w.x_bits(rows), _gamma(w.K, 1), eps, w.perm(), w.split, ctx=w.name)


@pytest.mark.parametrize("rows", [3, 300])
def test_one_row_per_pass(rows):
    # 8192 < K <= 16384: one row per pass through the two-stage pipelined
    # kernel (K = 14336, the Llama-3-8B MLP width), ragged row counts
    K, split = 14336, (10752, 2688, 896)
    rng = np.random.default_rng(rows + 14)
    x = (rng.standard_normal((rows, K)) * np.exp(rng.normal(0, 1, K))).astype(np.float32)
    _check(f32_bits(x), _gamma(K, rows), 1e-5, rng.permutation(K).astype(np.int32), split, ctx=f"K14336 rows{rows}")


def test_wide_rows_one_per_workgroup():
    # K above one LDS stage: the one-row-per-workgroup kernel
    K, split = 28672, (20480, 4096, 4096)
    rng = np.random.default_rng(77)
    x = rng.standard_normal((5, K)).astype(np.float32)
    _check(f32_bits(x), _gamma(K, 77), 1e-5, rng.permutation(K).astype(np.int32), split, ctx="K28672")


@pytest.mark.parametrize("formats", [("E2M3", "E4M3"), ("E3M2", "E5M2"), ("E2M3", "E5M2")])
def test_alternative_formats(formats):
    rng = np.random.default_rng(88)
    K, split = 1024, (512, 256, 256)
    x = (rng.standard_normal((40, K)) * np.exp(rng.normal(0, 1, K))).astype(np.float32)
    _check(f32_bits(x), _gamma(K, 88), 1e-6, rng.permutation(K).astype(np.int32), split, formats, ctx="alt")


def test_edge_rows():
    K, split = 256, (128, 64, 64)
    rng = np.random.default_rng(99)
    x = rng.standard_normal((8, K)).astype(np.float32)
    x[0] = 0.0                                  # zero row: eps keeps r finite, codes all zero
    x[1] = 3.0                                  # constant row
    x[2] = rng.standard_normal(K) * 2.0 ** -130  # subnormal bf16 values (squares far below fp32 range)
    x[3] = rng.standard_normal(K) * 1e30         # large values
    x[4, ::2] = -0.0                            # signed zeros
    x[5, :] = 0.0
    x[5, 17] = -7.0                             # a single non-zero channel
    g = rng.standard_normal(K).astype(np.float32)
    g[::5] = 0.0                                # zero weights
    g[1::7] = -g[1::7]
    _check(f32_bits(x), f32_bits(g), 1e-6, rng.permutation(K).astype(np.int32), split, ctx="edges")


def test_fused_layer_end_to_end():
    """RMSNorm+quantise -> GEMM against the oracle's chain."""
    b = _b()
    M, K, N, split = 200, 2048, 320, (1536, 384, 128)
    rng = np.random.default_rng(123)
    xb = f32_bits((rng.standard_normal((M, K)) * np.exp(rng.normal(0, 1, K))).astype(np.float32))
    wb = f32_bits((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
    perm = rng.permutation(K).astype(np.int32)
    gb = _gamma(K, 123)
    qa, y = _check(xb, gb, 1e-5, perm, split, ctx="end to end")
    qw = b.quantize_weight(to_dev_bf16(wb), to_dev_perm(perm), split)
    out = b.gemm(qa, qw)
    torch.cuda.synchronize()
    ref = O.gemm_mixed(O.quantize_mixed(y, perm, split), O.quantize_mixed(wb, perm, split))
    assert_gemm_close(y_to_f64(out), ref, ctx="Y")


def test_plain_quantiser_of_the_normalised_input_agrees():
    """The fused call and mm_quantize_act on the normalised bf16 activation
    write the same bytes (the plain path is unchanged)."""
    b = _b()
    K, split = 1024, (640, 256, 128)
    rng = np.random.default_rng(5)
    xb = f32_bits(rng.standard_normal((64, K)).astype(np.float32))
    gb = _gamma(K, 5)
    perm = rng.permutation(K).astype(np.int32)
    r32, _, amb = _factors(xb, 1e-5)
    assert not amb.any()
    fused = _run(xb, gb, 1e-5, perm, split)
    plain = b.quantize_act(to_dev_bf16(O.rmsnorm_apply(xb, gb, r32)), to_dev_perm(perm), split)
    torch.cuda.synchronize()
    rf, rp = fused.raw_host(), plain.raw_host()
    for k in ("q4", "q6", "q8", "sc"):
        assert np.array_equal(rf[k], rp[k]), k
