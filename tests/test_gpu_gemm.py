"""GPU parity of the mixed-precision GEMM (mm_gemm) against the oracle's float64
product of the dequantised operands, within |gpu - ref| <= 2^-8 |ref| +
1e-3 rms(ref).  The quantised operands come from the HIP quantiser, whose
bytes are first checked against the oracle, so both sides multiply the same
codes."""

import functools

import numpy as np
import pytest
import torch

from oracle import mx_oracle as O
from paper_2508_02343_amd import workloads as W
from tests.gpu_helpers import assert_codes_equal, assert_gemm_close, note, to_dev_bf16, to_dev_perm, y_to_f64

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=None)
def _b():
    from paper_2508_02343_amd import binding

    return binding


def _gpu_pair(xb, wb, perm, split):
    b = _b()
    p = to_dev_perm(perm)
    a = b.quantize_act(to_dev_bf16(xb), p, split)
    w = b.quantize_weight(to_dev_bf16(wb), p, split)
    return a, w


def _check_full(xb, wb, perm, split, ctx):
    a, w = _gpu_pair(xb, wb, perm, split)
    y = _b().gemm(a, w)
    torch.cuda.synchronize()
    ra, rw = O.quantize_mixed(xb, perm, split), O.quantize_mixed(wb, perm, split)
    assert_codes_equal(a, ra, ctx=ctx + " A")
    assert_codes_equal(w, rw, ctx=ctx + " W")
    assert_gemm_close(y_to_f64(y), O.gemm_mixed(ra, rw), ctx=ctx)


def test_tiny_config():
    w = W.TINY
    note(w.name)
    _check_full(w.x_bits(), w.w_bits(), w.perm(), w.split, w.name)


def _rand_case(M, N, split, seed):
    K = sum(split)
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((M, K)).astype(np.float32)
    out = rng.choice(K, max(1, K // 64), replace=False)
    x[:, out] *= 25
    perm = np.concatenate([np.setdiff1d(np.arange(K), out), out]).astype(np.int32)
    wgt = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    return W.f32_to_bf16_bits(x), W.f32_to_bf16_bits(wgt), perm


@pytest.mark.parametrize("split", [(96, 160, 96), (352, 0, 0), (0, 352, 0), (0, 0, 352), (32, 32, 288),
                                   (128, 0, 224), (0, 64, 32)])
@pytest.mark.parametrize("M,N", [(1, 16), (5, 70), (17, 33), (37, 130), (100, 72), (300, 260)])
def test_ragged(M, N, split):
    note(f"ragged M={M} N={N} split={split}")
    xb, wb, perm = _rand_case(M, N, split, seed=M * 7 + N + split[0])
    _check_full(xb, wb, perm, split, f"M{M} N{N} {split}")


@pytest.mark.parametrize("M,N,split", [(1, 6001, (96, 160, 96)), (20, 6000, (256, 128, 128)),
                                       (50, 6000, (0, 0, 512)), (1, 12000, (256, 128, 128)),
                                       (20, 12000, (96, 160, 96)), (50, 12000, (256, 128, 128)),
                                       (8, 20008, (256, 128, 128)), (64, 20000, (0, 0, 512))])
def test_decode_strips(M, N, split):
    """Decode kernel (M <= 64) at the strip widths its launch picks: for one
    activation tile 16-row strips (N = 6001) or whole 32-row groups
    (N = 12000, 20008: a part-filled last group); for two or four activation
    tiles rows per workgroup that are not a multiple of 16 (24, 48 and 40 on
    256 CUs: part-filled last tiles, two or four tiles per workgroup), the
    last at a width that needs two workgroups per CU."""
    note(f"decode strips M={M} N={N} split={split}")
    xb, wb, perm = _rand_case(M, N, split, seed=M * 11 + N + split[0])
    _check_full(xb, wb, perm, split, f"M{M} N{N} {split}")


@pytest.mark.parametrize("M,N", [(4, 700), (24, 300)])
def test_decode_long_k(M, N):
    """Decode kernel on the MLP-down width (K = 14336, split 10752 / 2688 / 896:
    84, 21 and 7 steps): the eight wavefronts go 5 / 2 / 1 to the groups, so
    every group takes several batches of steps per wavefront."""
    split = (10752, 2688, 896)
    note(f"decode long K M={M} N={N}")
    xb, wb, perm = _rand_case(M, N, split, seed=M + N)
    _check_full(xb, wb, perm, split, f"M{M} N{N} {split}")


@pytest.mark.parametrize("split", [(96, 160, 96), (352, 0, 0), (0, 352, 0), (0, 0, 352), (128, 0, 224)])
@pytest.mark.parametrize("M,N", [(3000, 5400), (1000, 1000)])
def test_ragged_large(M, N, split):
    """Every output of shapes whose tile grids run the 256 x 256 tiles
    (12 x 22 tiles, at least one per CU) and the 256 x 128 tiles (4 x 8),
    both with ragged last tiles in M and N."""
    note(f"ragged large M={M} N={N} split={split}")
    xb, wb, perm = _rand_case(M, N, split, seed=M + N + split[1])
    _check_full(xb, wb, perm, split, f"M{M} N{N} {split}")


@pytest.mark.parametrize("M,N", [(3000, 5400), (1000, 1000)])
def test_ragged_large_alternative_formats(M, N):
    split, formats = (96, 160, 96), ("E2M3", "E5M2")
    note(f"ragged large formats {formats} M={M} N={N}")
    xb, wb, perm = _rand_case(M, N, split, seed=M + 2 * N)
    b = _b()
    p = to_dev_perm(perm)
    a = b.quantize_act(to_dev_bf16(xb), p, split, formats=formats)
    w = b.quantize_weight(to_dev_bf16(wb), p, split, formats=formats)
    y = b.gemm(a, w)
    torch.cuda.synchronize()
    fm = (O.E2M1, O.FORMATS[formats[0]], O.FORMATS[formats[1]])
    ra, rw = O.quantize_mixed(xb, perm, split, fm), O.quantize_mixed(wb, perm, split, fm)
    assert_codes_equal(a, ra, ctx="A")
    assert_codes_equal(w, rw, ctx="W")
    assert_gemm_close(y_to_f64(y), O.gemm_mixed(ra, rw), ctx=f"{formats} M{M} N{N}")


@pytest.mark.parametrize("w", W.decode_workloads(), ids=lambda w: w.name)
def test_decode_configs(w):
    """Full activation and full weight on the GPU; oracle on 256 sampled
    weight rows (output columns), all activation rows."""
    note(w.name)
    xb, wb, perm = w.x_bits(), w.w_bits(), w.perm()
    a, wq = _gpu_pair(xb, wb, perm, w.split)
    y = _b().gemm(a, wq)
    torch.cuda.synchronize()
    cols = np.unique(np.concatenate([[0, w.N - 1], np.random.default_rng(2).choice(w.N, 254, replace=False)]))
    ra, rw = O.quantize_mixed(xb, perm, w.split), O.quantize_mixed(wb[cols], perm, w.split)
    assert_codes_equal(a, ra, ctx=w.name + " A")
    assert_codes_equal(wq, rw, rows=cols, ctx=w.name + " W")
    assert_gemm_close(y_to_f64(y)[:, cols], O.gemm_mixed(ra, rw), ctx=w.name)


@pytest.mark.parametrize("w", W.PREFILL, ids=lambda w: w.name)
def test_prefill_configs_sampled(w):
    """Full-size quantisers and GEMM on the GPU; the oracle quantises 64
    sampled activation rows and 64 sampled weight rows (their codes and
    scales must match the GPU's bytes) and recomputes the 64 x 64 outputs
    they meet in."""
    note(w.name)
    xb, wb, perm = w.x_bits(), w.w_bits(), w.perm()
    a, wq = _gpu_pair(xb, wb, perm, w.split)
    y = _b().gemm(a, wq)
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([[0, w.M - 1], rng.choice(w.M, 62, replace=False)]))
    cols = np.unique(np.concatenate([[0, w.N - 1], rng.choice(w.N, 62, replace=False)]))
    ra, rw = O.quantize_mixed(xb[rows], perm, w.split), O.quantize_mixed(wb[cols], perm, w.split)
    assert_codes_equal(a, ra, rows=rows, ctx=w.name + " A")
    assert_codes_equal(wq, rw, rows=cols, ctx=w.name + " W")
    assert_gemm_close(y_to_f64(y[torch.from_numpy(rows).cuda()])[:, cols], O.gemm_mixed(ra, rw), ctx=w.name)


def test_one_activation_feeds_two_weights():
    """One quantised activation reused by two GEMMs with the same sigma."""
    note("shared activation")
    split = (256, 64, 64)
    xb, wb, perm = _rand_case(40, 96, split, seed=5)
    _, wb2, _ = _rand_case(40, 48, split, seed=6)
    b = _b()
    p = to_dev_perm(perm)
    a = b.quantize_act(to_dev_bf16(xb), p, split)
    y1 = b.gemm(a, b.quantize_weight(to_dev_bf16(wb), p, split))
    y2 = b.gemm(a, b.quantize_weight(to_dev_bf16(wb2), p, split))
    torch.cuda.synchronize()
    ra = O.quantize_mixed(xb, perm, split)
    assert_gemm_close(y_to_f64(y1), O.gemm_mixed(ra, O.quantize_mixed(wb, perm, split)), "y1")
    assert_gemm_close(y_to_f64(y2), O.gemm_mixed(ra, O.quantize_mixed(wb2, perm, split)), "y2")


@pytest.mark.parametrize("formats", [("E2M3", "E5M2"), ("E2M3", "E4M3"), ("E3M2", "E5M2")], ids="-".join)
@pytest.mark.parametrize("M,N", [(5, 70), (37, 130), (300, 260)])
def test_alternative_formats(M, N, formats):
    """The ablation's MXFP6 = E2M3 and MXFP8 = E5M2 variants through both
    GEMM kernels (decode for M <= 64, tiled above)."""
    split = (96, 160, 96)
    note(f"formats {formats} M={M} N={N}")
    xb, wb, perm = _rand_case(M, N, split, seed=M * 11 + N)
    b = _b()
    p = to_dev_perm(perm)
    a = b.quantize_act(to_dev_bf16(xb), p, split, formats=formats)
    w = b.quantize_weight(to_dev_bf16(wb), p, split, formats=formats)
    y = b.gemm(a, w)
    torch.cuda.synchronize()
    fm = (O.E2M1, O.FORMATS[formats[0]], O.FORMATS[formats[1]])
    ra, rw = O.quantize_mixed(xb, perm, split, fm), O.quantize_mixed(wb, perm, split, fm)
    ctx = f"{formats} M{M} N{N}"
    assert_codes_equal(a, ra, ctx=ctx + " A")
    assert_codes_equal(w, rw, ctx=ctx + " W")
    assert_gemm_close(y_to_f64(y), O.gemm_mixed(ra, rw), ctx=ctx)


def test_mixed_formats_are_rejected():
    xb, wb, perm = _rand_case(8, 16, (96, 160, 96), seed=3)
    b = _b()
    p = to_dev_perm(perm)
    a = b.quantize_act(to_dev_bf16(xb), p, (96, 160, 96), formats=("E2M3", "E4M3"))
    w = b.quantize_weight(to_dev_bf16(wb), p, (96, 160, 96))
    with pytest.raises(b.MMError, match="MM_ERR_FORMAT"):
        b.gemm(a, w)


@pytest.mark.parametrize("M", [8, 300])
def test_stacked_qkv_equals_separate_gemms(M):
    """Q, K and V share the activation's sigma and split, so their weights can
    be stacked along N (Llama-3-8B: 4096 + 1024 + 1024 rows), quantised once and
    multiplied in one launch; each column slice of that product equals,
    bit for bit, the separate GEMM of the same quantised activation (every
    output element sums the same K blocks in the same order)."""
    b = _b()
    K, split, parts = 4096, (3072, 768, 256), (4096, 1024, 1024)
    rng = np.random.default_rng(M)
    xb = W.LLAMA_ATTN.x_bits(M)
    perm = W.LLAMA_ATTN.perm()
    ws = [W.f32_to_bf16_bits((rng.standard_normal((n, K)) * 0.02).astype(np.float32)) for n in parts]
    note(f"stacked QKV M={M}")
    p = to_dev_perm(perm)
    a = b.quantize_act(to_dev_bf16(xb), p, split)
    stacked = b.gemm(a, b.quantize_weight(to_dev_bf16(np.concatenate(ws)), p, split))
    sep = [b.gemm(a, b.quantize_weight(to_dev_bf16(wk), p, split)) for wk in ws]
    torch.cuda.synchronize()
    col = 0
    for n, y in zip(parts, sep):
        assert torch.equal(stacked[:, col:col + n], y), (M, col)
        col += n
    ref = O.gemm_mixed(O.quantize_mixed(xb, perm, split), O.quantize_mixed(ws[1], perm, split))
    assert_gemm_close(y_to_f64(sep[1]), ref, ctx="K slice")
