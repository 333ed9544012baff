"""mm_calibrate_no_alloc (workspace in the library's static scratch) against
mm_calibrate (caller workspace) through the C ABI: sigma and the split must be
identical, on two calls in a row, the second with a smaller input, so the
second runs on what the first left in the scratch."""

import functools

import pytest
import torch

from paper_2508_02343_amd import workloads as W
from tests.gpu_helpers import note, to_dev_bf16

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=None)
def _b():
    from paper_2508_02343_amd import binding

    return binding


def _pair(rows, K, seed, formats):
    b = _b()
    x = to_dev_bf16(W.calibration_bits(rows, K, seed))
    perm_ref, split_ref = b.calibrate_async(x, formats)
    # outputs pre-filled with a value neither call can produce
    perm = torch.full((K,), -7, dtype=torch.int32, device=x.device)
    split = torch.full((3,), -7, dtype=torch.int32, device=x.device)
    b.calibrate_no_alloc_async(x, perm, split, formats)
    torch.cuda.synchronize()
    return perm, split, perm_ref, split_ref


@pytest.mark.parametrize("formats", [("E3M2", "E4M3"), ("E2M3", "E5M2")], ids="-".join)
def test_no_alloc_matches_workspace_call(formats):
    for rows, K, seed in ((8192, 5120, 11), (300, 1024, 12)):
        note(f"calibrate no-alloc rows={rows} K={K} {formats}")
        perm, split, perm_ref, split_ref = _pair(rows, K, seed, formats)
        assert torch.equal(split, split_ref), (rows, K, split.tolist(), split_ref.tolist())
        assert torch.equal(perm, perm_ref), (rows, K)
        p = perm.cpu()
        assert torch.equal(torch.sort(p).values, torch.arange(K, dtype=torch.int32))
        s = split.cpu().tolist()
        assert sum(s) == K and all(v % 32 == 0 and v >= 0 for v in s)


def test_no_alloc_largest_plan_and_nonfinite():
    """The widest K whose plan fits the scratch at a large row count, then an
    input holding Inf (split (-1, -1, -1), identity sigma) on a smaller one."""
    b = _b()
    note("calibrate no-alloc rows=4096 K=31488")
    perm, split, perm_ref, split_ref = _pair(4096, 31488, 13, ("E3M2", "E4M3"))
    assert torch.equal(split, split_ref) and torch.equal(perm, perm_ref)
    note("calibrate no-alloc Inf rows=64 K=256")
    x = to_dev_bf16(W.calibration_bits(64, 256, 14))
    x[5, 17] = float("inf")
    perm = torch.empty(256, dtype=torch.int32, device=x.device)
    split = torch.empty(3, dtype=torch.int32, device=x.device)
    b.calibrate_no_alloc_async(x, perm, split)
    torch.cuda.synchronize()
    assert split.cpu().tolist() == [-1, -1, -1]
    assert torch.equal(perm.cpu(), torch.arange(256, dtype=torch.int32))
