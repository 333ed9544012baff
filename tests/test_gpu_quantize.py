"""GPU parity of the fused reorder-and-quantize kernel: every code and scale
byte must equal the oracle's (mm_quantize_act and mm_quantize_weight)."""

import functools

import numpy as np
import pytest
import torch

from oracle import mx_oracle as O
from paper_2508_02343_amd import workloads as W
from tests.gpu_helpers import assert_codes_equal, note, to_dev_bf16, to_dev_perm

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=None)
def _b():
    from paper_2508_02343_amd import binding

    return binding


def _run(bits, perm, split, weight=False, ld_extra=0):
    b = _b()
    x = to_dev_bf16(bits)
    if ld_extra:
        big = torch.zeros((x.shape[0], x.shape[1] + ld_extra), dtype=torch.bfloat16, device="cuda")
        big[:, : x.shape[1]] = x
        x = big[:, : bits.shape[1]]
    fn = b.quantize_weight if weight else b.quantize_act
    out = fn(x, to_dev_perm(perm), split)
    torch.cuda.synchronize()
    return out


def test_tiny_config_activation_and_weight():
    w = W.TINY
    note(w.name)
    xb, wb, perm = w.x_bits(), w.w_bits(), w.perm()
    assert_codes_equal(_run(xb, perm, w.split), O.quantize_mixed(xb, perm, w.split), ctx="tiny X")
    assert_codes_equal(_run(wb, perm, w.split, weight=True), O.quantize_mixed(wb, perm, w.split), ctx="tiny W")


RAGGED_SPLITS = [(96, 160, 96), (352, 0, 0), (0, 352, 0), (0, 0, 352), (32, 32, 288), (0, 96, 256),
                 (256, 64, 32)]


@pytest.mark.parametrize("split", RAGGED_SPLITS)
@pytest.mark.parametrize("rows", [1, 37])
def test_ragged_shapes(split, rows):
    K = sum(split)
    note(f"ragged rows={rows} split={split}")
    rng = np.random.default_rng(rows * 1000 + split[0])
    x = (rng.standard_normal((rows, K)) * np.exp2(rng.integers(-3, 4, (rows, K)))).astype(np.float32)
    bits = W.f32_to_bf16_bits(x)
    perm = rng.permutation(K).astype(np.int32)
    assert_codes_equal(_run(bits, perm, split, ld_extra=24), O.quantize_mixed(bits, perm, split), ctx=str(split))


def _edge_rows(rng, K):
    """Rows built to hit rounding ties, saturation, signed zeros, bf16
    subnormals and the E8M0 clamp in every group."""
    rows = []
    # 1. random finite bf16 patterns: every exponent, so big amax with tiny elements
    r = rng.integers(0, 1 << 16, K, dtype=np.uint32).astype(np.uint16)
    exp = (r >> 7) & 0xFF
    r[exp == 0xFF] &= 0x807F  # no Inf / NaN
    rows.append(r)
    # 2. narrow exponent range: few-mantissa-bit values sit exactly on grid midpoints
    for e0 in (120, 127, 133):
        e = rng.integers(e0, e0 + 3, K).astype(np.uint16)
        m = (rng.integers(0, 8, K) << 4).astype(np.uint16)  # 3 mantissa bits
        s = rng.integers(0, 2, K).astype(np.uint16) << 15
        rows.append(s | (e << 7) | m)
    # 3. zeros and negative zeros, whole blocks of them
    z = np.zeros(K, np.uint16)
    z[::2] = 0x8000
    rows.append(z)
    # 4. bf16 subnormals only (scale exponent clamps to -127)
    rows.append((rng.integers(1, 128, K) | (rng.integers(0, 2, K) << 15)).astype(np.uint16))
    # 5. largest finite values and tiny normal values mixed
    big = np.full(K, 0x7F7F, np.uint16)
    big[1::3] = 0x0080
    big[2::5] = 0xFF7F
    rows.append(big)
    # 6. a block's max on a binade edge (amax = 2^k exactly) with near-max members
    edge = np.full(K, 0x3F80, np.uint16)  # 1.0
    edge[1::4] = 0x3FFF  # just below 2.0
    edge[2::4] = 0xBF7F
    rows.append(edge)
    return np.stack(rows)


@pytest.mark.parametrize("split", [(128, 96, 64), (32, 0, 256), (0, 288, 0)])
def test_edge_blocks(split):
    K = sum(split)
    note(f"edge blocks split={split}")
    rng = np.random.default_rng(17 + split[1])
    bits = _edge_rows(rng, K)
    for perm in (np.arange(K, dtype=np.int32), rng.permutation(K).astype(np.int32)):
        assert_codes_equal(_run(bits, perm, split), O.quantize_mixed(bits, perm, split), ctx=f"edge {split}")


def test_repeatable_bytes():
    w = W.TINY
    note("determinism")
    xb, perm = w.x_bits(), w.perm()
    a, b = _run(xb, perm, w.split).raw_host(), _run(xb, perm, w.split).raw_host()
    for k in a:
        assert np.array_equal(a[k], b[k])


FULL = [W.LLAMA_ATTN, W.LLAMA_MLP_DOWN, W.QWEN_MLP_UP]


@pytest.mark.parametrize("w", FULL, ids=lambda w: w.name)
def test_full_size_activation_sampled_rows(w):
    """The whole activation is quantised at its real size, in the launch the
    benchmark times; the oracle checks a sample of rows (rows are independent)."""
    note(f"full-size activation {w.name}")
    xb, perm = w.x_bits(), w.perm()
    got = _run(xb, perm, w.split)
    rows = np.unique(np.concatenate([[0, w.M - 1], np.random.default_rng(0).choice(w.M, 62, replace=False)]))
    ref = O.quantize_mixed(xb[rows], perm, w.split)
    assert_codes_equal(got, ref, rows=rows, ctx=w.name)


def test_full_size_weight_sampled_rows():
    w = W.QWEN_MLP_UP
    note(f"full-size weight {w.name}")
    wb, perm = w.w_bits(), w.perm()
    got = _run(wb, perm, w.split, weight=True)
    rows = np.unique(np.concatenate([[0, w.N - 1], np.random.default_rng(1).choice(w.N, 62, replace=False)]))
    assert_codes_equal(got, O.quantize_mixed(wb[rows], perm, w.split), rows=rows, ctx=w.name + " W")


@pytest.mark.parametrize("rows,split", [(9, (64, 32, 32)), (40, (32, 96, 160)), (1, (96, 0, 64))])
def test_padding_is_written_as_zero(rows, split):
    """Blocks past a group's end inside its last step, and rows past `rows`
    up to the next multiple of 32, are zero codes and zero scale bytes, even
    over buffers that held garbage (the GEMM reads them)."""
    K = sum(split)
    note(f"padding rows={rows} split={split}")
    rng = np.random.default_rng(rows + K)
    bits = W.f32_to_bf16_bits(rng.standard_normal((rows, K)).astype(np.float32))
    perm = rng.permutation(K).astype(np.int32)
    b = _b()
    out = b.MXTensor.empty(rows, K, split)
    for t in (out.q4, out.q6, out.q8, out.sc):
        if t is not None:
            t.fill_(0xAB)
    b.quantize_act(to_dev_bf16(bits), to_dev_perm(perm), split, out=out)
    torch.cuda.synchronize()
    assert_codes_equal(out, O.quantize_mixed(bits, perm, split), ctx="padding")


@pytest.mark.parametrize("rows", [5, 33])
def test_wide_rows(rows):
    """Rows wider than a third of LDS (K = 28672, 56 KB of bf16) take the
    one-row-per-workgroup path; codes and scales still match the oracle."""
    split = (20480, 4096, 4096)
    K = sum(split)
    note(f"wide rows={rows} K={K}")
    rng = np.random.default_rng(K + rows)
    bits = W.f32_to_bf16_bits((rng.standard_normal((rows, K)) * np.exp2(rng.integers(-4, 5, (rows, K)))).astype(np.float32))
    perm = rng.permutation(K).astype(np.int32)
    got = _run(bits, perm, split)
    assert_codes_equal(got, O.quantize_mixed(bits, perm, split), ctx="wide rows")


# The ablation's alternatives (Table tab:ablation-study-mxfp6-mxfp8): MXFP6 as
# E2M3, MXFP8 as E5M2, alone and together.
ALT_FORMATS = [("E2M3", "E5M2"), ("E2M3", "E4M3"), ("E3M2", "E5M2")]


def _oracle_formats(formats):
    return (O.E2M1, O.FORMATS[formats[0]], O.FORMATS[formats[1]])


@pytest.mark.parametrize("formats", ALT_FORMATS, ids="-".join)
@pytest.mark.parametrize("split", [(96, 160, 96), (0, 352, 0), (0, 0, 352), (32, 32, 288)])
def test_alternative_formats_ragged(split, formats):
    K = sum(split)
    rows = 37
    note(f"formats {formats} split={split}")
    rng = np.random.default_rng(rows * 1000 + split[1] + 7 * split[2])
    x = (rng.standard_normal((rows, K)) * np.exp2(rng.integers(-3, 4, (rows, K)))).astype(np.float32)
    bits = W.f32_to_bf16_bits(x)
    perm = rng.permutation(K).astype(np.int32)
    b = _b()
    got = b.quantize_act(to_dev_bf16(bits), to_dev_perm(perm), split, formats=formats)
    torch.cuda.synchronize()
    assert_codes_equal(got, O.quantize_mixed(bits, perm, split, _oracle_formats(formats)), ctx=f"{formats} {split}")


@pytest.mark.parametrize("formats", ALT_FORMATS, ids="-".join)
def test_alternative_formats_edge_blocks(formats):
    """Ties, saturation at each format's top value (7.5 for E2M3, 57344 for
    E5M2), signed zeros, subnormal inputs and the E8M0 clamp."""
    split = (128, 96, 64)
    K = sum(split)
    note(f"edge blocks formats {formats}")
    rng = np.random.default_rng(29)
    bits = _edge_rows(rng, K)
    b = _b()
    for perm in (np.arange(K, dtype=np.int32), rng.permutation(K).astype(np.int32)):
        got = b.quantize_weight(to_dev_bf16(bits), to_dev_perm(perm), split, formats=formats)
        torch.cuda.synchronize()
        assert_codes_equal(got, O.quantize_mixed(bits, perm, split, _oracle_formats(formats)), ctx=f"edge {formats}")
