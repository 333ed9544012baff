"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
compare it with the oracle on the same seeded inputs."""

from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import mx_oracle as O
from tests import packed_layout as L


def note(msg: str) -> None:
    # name the case before each GPU step, so a failure points at it
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def to_dev_bf16(bits: np.ndarray) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).cuda()


def to_dev_perm(perm: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(perm, dtype=np.int32)).cuda()


def _first_diff(g, r, ctx, name):
    bad = np.argwhere(g != r)
    idx = tuple(bad[0])
    raise AssertionError(f"{ctx} {name}: {len(bad)} bytes differ; first at {idx}: "
                         f"gpu {g[idx]:#04x} oracle {r[idx]:#04x}")


def assert_codes_equal(t, ref: O.MXTensor, rows=None, ctx: str = "") -> None:
    """Byte-exact comparison of a binding MXTensor's buffers with the oracle.

    rows=None: ref covers all rows; every byte of the four packed buffers,
    padding included, must equal the oracle's codes and scales laid out per
    the header.  Otherwise ref covers only the listed rows, which are
    compared after unpacking the GPU's buffers to row-major form.
    """
    raw = t.raw_host()
    if rows is None:
        want = L.tile(ref.q4, ref.q6, ref.q8, ref.sc, t.rows, t.split)
        for name in ("q4", "q6", "q8", "sc"):
            g, r = raw[name], want[name]
            assert g.shape == r.shape, (ctx, name, g.shape, r.shape)
            if not np.array_equal(g, r):
                _first_diff(g, r, ctx, name)
        return
    got = L.untile(raw, t.rows, t.split)
    for name in ("q4", "q6", "q8", "sc"):
        g = got[name][rows]
        r = np.asarray(getattr(ref, name))
        assert g.shape == r.shape, (ctx, name, g.shape, r.shape)
        if not np.array_equal(g, r):
            _first_diff(g, r, ctx, name)


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
