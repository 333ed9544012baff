"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
compare it with the oracle on the same seeded inputs."""

from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import mx_oracle as O


def note(msg: str) -> None:
    # name the case before each GPU step, so a failure points at it
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def to_dev_bf16(bits: np.ndarray) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).cuda()


def to_dev_perm(perm: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(perm, dtype=np.int32)).cuda()


def assert_codes_equal(gpu: dict, ref: O.MXTensor, rows=None, ctx: str = "") -> None:
    """Byte-exact comparison of q4/q6/q8/sc (optionally of selected rows)."""
    for name in ("q4", "q6", "q8", "sc"):
        g = gpu[name] if rows is None else gpu[name][rows]
        r = np.asarray(getattr(ref, name))
        assert g.shape == r.shape, (ctx, name, g.shape, r.shape)
        if not np.array_equal(g, r):
            bad = np.argwhere(g != r)
            i, j = bad[0]
            raise AssertionError(f"{ctx} {name}: {len(bad)} bytes differ; first at row {i} byte {j}: "
                                 f"gpu {g[i, j]:#04x} oracle {r[i, j]:#04x}")


def y_to_f64(y: torch.Tensor) -> np.ndarray:
    return y.float().cpu().numpy().astype(np.float64)


def assert_gemm_close(y_gpu: np.ndarray, y_ref: np.ndarray, ctx: str = "") -> None:
    """|gpu - ref| <= 2^-8 |ref| + 1e-3 rms(ref), elementwise."""
    tol = O.gemm_tolerance(y_ref)
    err = np.abs(y_gpu - y_ref)
    bad = err > tol
    if np.any(bad):
        i, j = np.argwhere(bad)[0]
        raise AssertionError(f"{ctx}: {bad.sum()} of {bad.size} outputs out of tolerance; first ({i},{j}) "
                             f"gpu {y_gpu[i, j]!r} ref {y_ref[i, j]!r} tol {tol[i, j]!r}")
