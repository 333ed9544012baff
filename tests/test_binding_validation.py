"""CPU checks of the binding's argument validation: a mismatched output
descriptor, permutation or result tensor is rejected with ValueError before
anything reaches the library (on the GPU it would be an out-of-bounds
access)."""

import pytest
import torch

from paper_2508_02343_amd import binding as b

SPLIT = (64, 32, 32)


def _mx(rows=40, K=128, split=SPLIT):
    return b.MXTensor.empty(rows, K, split, device="cpu")


def test_matching_descriptor_passes():
    t = _mx()
    b._check_mx(t, 40, 128, SPLIT, torch.device("cpu"), "t")


@pytest.mark.parametrize("rows,K,split", [(41, 128, SPLIT), (40, 160, (96, 32, 32)), (40, 128, (96, 0, 32))])
def test_descriptor_shape_or_split_mismatch(rows, K, split):
    with pytest.raises(ValueError):
        b._check_mx(_mx(), rows, K, split, torch.device("cpu"), "out")


def test_short_buffer_rejected():
    t = _mx()
    t.q4 = t.q4[:-1]
    with pytest.raises(ValueError, match="q4"):
        b._check_mx(t, 40, 128, SPLIT, torch.device("cpu"), "out")


def test_host_input_rejected():
    x = torch.zeros(40, 128, dtype=torch.bfloat16)
    perm = torch.arange(128, dtype=torch.int32)
    with pytest.raises(ValueError, match="device"):
        b.quantize_act(x, perm, SPLIT, out=_mx())


@pytest.mark.parametrize("shape", [(40, 64), (39, 48), (40, 48, 1)])
def test_gemm_result_shape_rejected(shape):
    a, w = _mx(40), _mx(48)
    y = torch.empty(shape, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="y must be"):
        b.gemm(a, w, y=y)


def test_gemm_result_dtype_and_stride_rejected():
    a, w = _mx(40), _mx(48)
    with pytest.raises(ValueError):
        b.gemm(a, w, y=torch.empty(40, 48, dtype=torch.float32))
    with pytest.raises(ValueError):
        b.gemm(a, w, y=torch.empty(48, 40, dtype=torch.bfloat16).t())
