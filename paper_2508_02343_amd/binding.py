"""Thin ctypes binding of libmicromix.so (include/micromix.h).

Argument marshalling only: every step of the path runs in the HIP kernels of
the library.  torch supplies device memory and the stream.  If the library
is missing the import of this module fails loudly; there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmicromix.so")

MM_OK = 0
ABI_VERSION = 6  # MM_ABI_VERSION of include/micromix.h this binding follows
STATUS_NAMES = {0: "MM_OK", 1: "MM_ERR_NULL", 2: "MM_ERR_SHAPE", 3: "MM_ERR_SPLIT", 4: "MM_ERR_ALIGN",
                5: "MM_ERR_FORMAT", 6: "MM_ERR_DEVICE", 7: "MM_ERR_WORKSPACE",
                8: "MM_ERR_VALUE"}


class MMSplit(ctypes.Structure):
    _fields_ = [("p4", ctypes.c_int32), ("p6", ctypes.c_int32), ("p8", ctypes.c_int32)]


class MMFormats(ctypes.Structure):
    _fields_ = [("fp6", ctypes.c_int32), ("fp8", ctypes.c_int32)]


# element formats of the 6-bit and 8-bit groups: name -> mm_fp6_format / mm_fp8_format
FP6_FORMATS = {"E3M2": 0, "E2M3": 1}
FP8_FORMATS = {"E4M3": 0, "E5M2": 1}
DEFAULT_FORMATS = ("E3M2", "E4M3")


class MMTensor(ctypes.Structure):
    _fields_ = [
        ("rows", ctypes.c_int64),
        ("K", ctypes.c_int64),
        ("split", MMSplit),
        ("formats", MMFormats),
        ("q4", ctypes.c_void_p),
        ("q6", ctypes.c_void_p),
        ("q8", ctypes.c_void_p),
        ("sc", ctypes.c_void_p),
    ]


class MMSizes(ctypes.Structure):
    _fields_ = [("q4", ctypes.c_int64), ("q6", ctypes.c_int64), ("q8", ctypes.c_int64), ("sc", ctypes.c_int64)]


def _load(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it first (python -m paper_2508_02343_amd.build_lib)")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    T = ctypes.POINTER(MMTensor)
    lib.mm_quantize_act.argtypes = [P, I64, P, T, P]
    lib.mm_quantize_weight.argtypes = [P, I64, P, T, P]
    lib.mm_gemm.argtypes = [T, T, P, I64, P]
    lib.mm_rmsnorm_quantize_act.argtypes = [P, I64, P, ctypes.c_float, P, T, P]
    for f in (lib.mm_quantize_act, lib.mm_quantize_weight, lib.mm_gemm, lib.mm_rmsnorm_quantize_act):
        f.restype = ctypes.c_int
    lib.mm_status_str.argtypes = [ctypes.c_int]
    lib.mm_status_str.restype = ctypes.c_char_p
    lib.mm_last_error.argtypes = []
    lib.mm_last_error.restype = ctypes.c_char_p
    lib.mm_abi_version.argtypes = []
    lib.mm_abi_version.restype = ctypes.c_int
    lib.mm_mx_layout_sizes.argtypes = [I64, I64, MMSplit, ctypes.POINTER(MMSizes)]
    lib.mm_mx_layout_sizes.restype = ctypes.c_int
    lib.mm_calibrate_workspace_size.argtypes = [I64, I64, ctypes.POINTER(I64)]
    lib.mm_calibrate_workspace_size.restype = ctypes.c_int
    lib.mm_calibrate.argtypes = [P, I64, I64, I64, MMFormats, P, I64, P, P, P]
    lib.mm_calibrate.restype = ctypes.c_int
    lib.mm_calibrate_no_alloc.argtypes = [P, I64, I64, I64, MMFormats, P, P, P]
    lib.mm_calibrate_no_alloc.restype = ctypes.c_int
    if lib.mm_abi_version() != ABI_VERSION:
        raise ImportError(f"{path}: ABI version {lib.mm_abi_version()}, this binding needs {ABI_VERSION}")
    return lib


lib = _load()


class MMError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def _check(status: int) -> None:
    if status != MM_OK:
        raise MMError(status, lib.mm_last_error().decode())


def _round16(v: int) -> int:
    return (v + 15) // 16 * 16


def layout_sizes(rows: int, K: int, split) -> dict:
    """mm_mx_layout_sizes: byte count of each buffer of a quantised tensor."""
    sz = MMSizes()
    _check(lib.mm_mx_layout_sizes(rows, K, MMSplit(*(int(p) for p in split)), ctypes.byref(sz)))
    return {"q4": sz.q4, "q6": sz.q6, "q8": sz.q8, "sc": sz.sc}


def _stream_ptr(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


@dataclass
class MXTensor:
    """Quantised operand in device memory: three code buffers and scales,
    each a flat uint8 tensor in the packed layout of include/micromix.h
    (an empty group has no buffer)."""

    rows: int
    K: int
    split: tuple[int, int, int]
    q4: torch.Tensor | None
    q6: torch.Tensor | None
    q8: torch.Tensor | None
    sc: torch.Tensor
    formats: tuple[str, str] = DEFAULT_FORMATS  # element formats of the 6-bit and 8-bit groups

    @classmethod
    def empty(cls, rows: int, K: int, split, device="cuda", formats=DEFAULT_FORMATS) -> "MXTensor":
        split = tuple(int(p) for p in split)
        sz = layout_sizes(rows, K, split)

        def buf(nbytes):
            if nbytes == 0:
                return None
            return torch.empty(nbytes, dtype=torch.uint8, device=device)

        return cls(rows, K, split, buf(sz["q4"]), buf(sz["q6"]), buf(sz["q8"]), buf(sz["sc"]), tuple(formats))

    def descriptor(self) -> MMTensor:
        d = MMTensor()
        d.rows, d.K = self.rows, self.K
        d.split = MMSplit(*self.split)
        # unknown names map to -1, which the library rejects (MM_ERR_FORMAT)
        d.formats = MMFormats(FP6_FORMATS.get(self.formats[0], -1), FP8_FORMATS.get(self.formats[1], -1))
        for name in ("q4", "q6", "q8", "sc"):
            t = getattr(self, name)
            setattr(d, name, t.data_ptr() if t is not None else None)
        return d

    def raw_host(self) -> dict:
        """The four buffers' bytes as numpy arrays (empty for an absent group)."""
        import numpy as np

        return {k: (getattr(self, k).cpu().numpy() if getattr(self, k) is not None else np.zeros(0, np.uint8))
                for k in ("q4", "q6", "q8", "sc")}


def _check_mx(t: MXTensor, rows: int, K: int, split, device, name: str) -> None:
    """An MXTensor whose buffers hold the packed layout of (rows, K, split)
    on `device` (the library reads and writes exactly those bytes)."""
    if t.rows != rows or t.K != K or tuple(int(p) for p in t.split) != tuple(int(p) for p in split):
        raise ValueError(f"{name} is [{t.rows}, {t.K}] split {tuple(t.split)}, expected [{rows}, {K}] split "
                         f"{tuple(split)}")
    sz = layout_sizes(rows, K, split)
    for b in ("q4", "q6", "q8", "sc"):
        buf = getattr(t, b)
        n = 0 if buf is None else buf.numel() * buf.element_size()
        if n < sz[b]:
            raise ValueError(f"{name}.{b} holds {n} bytes, the layout needs {sz[b]}")
        if buf is not None and (buf.device != device or not buf.is_contiguous()):
            raise ValueError(f"{name}.{b} must be contiguous and on {device}")


def _quantize(fn, x: torch.Tensor, perm: torch.Tensor, split, out: MXTensor | None, stream, formats) -> MXTensor:
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1 or not x.is_cuda:
        raise ValueError("x must be a 2-D row-major bfloat16 device tensor")
    rows, K = x.shape
    if perm.dtype != torch.int32 or not perm.is_contiguous() or perm.numel() != K or perm.device != x.device:
        raise ValueError("perm must be a contiguous int32 tensor of K elements on x's device")
    split = tuple(int(p) for p in split)
    if out is None:
        out = MXTensor.empty(rows, K, split, device=x.device, formats=formats)
    else:
        _check_mx(out, rows, K, split, x.device, "out")
    d = out.descriptor()
    _check(fn(ctypes.c_void_p(x.data_ptr()), x.stride(0), ctypes.c_void_p(perm.data_ptr()), ctypes.byref(d),
              _stream_ptr(stream)))
    return out


def quantize_act(x: torch.Tensor, perm: torch.Tensor, split, out: MXTensor | None = None, stream=None,
                 formats=DEFAULT_FORMATS) -> MXTensor:
    """mm_quantize_act: fused reorder-and-quantize of bf16 activations
    (formats: of the 6-bit and 8-bit groups, used when out is None)."""
    return _quantize(lib.mm_quantize_act, x, perm, split, out, stream, formats)


def rmsnorm_quantize_act(x: torch.Tensor, gamma: torch.Tensor, eps: float, perm: torch.Tensor, split,
                         out: MXTensor | None = None, stream=None, formats=DEFAULT_FORMATS) -> MXTensor:
    """mm_rmsnorm_quantize_act: RMSNorm (bf16 weight gamma [K], 16-byte
    aligned, eps) fused with the reorder-and-quantize of bf16 activations."""
    if gamma.dtype != torch.bfloat16 or gamma.dim() != 1 or not gamma.is_contiguous() or gamma.numel() != x.shape[-1]:
        raise ValueError("gamma must be a contiguous bfloat16 tensor [K]")
    g = ctypes.c_void_p(gamma.data_ptr())

    def fn(xp, ld, pp, d, st):
        return lib.mm_rmsnorm_quantize_act(xp, ld, g, ctypes.c_float(eps), pp, d, st)

    return _quantize(fn, x, perm, split, out, stream, formats)


def quantize_weight(w: torch.Tensor, perm: torch.Tensor, split, out: MXTensor | None = None,
                    stream=None, formats=DEFAULT_FORMATS) -> MXTensor:
    """mm_quantize_weight: offline reorder-and-quantize of a bf16 weight [N, K]
    (formats as for quantize_act)."""
    return _quantize(lib.mm_quantize_weight, w, perm, split, out, stream, formats)


def gemm(a: MXTensor, w: MXTensor, y: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """mm_gemm: Y[M, N] = A W^T in bf16 (one fp32 accumulator over all groups)."""
    dev = a.sc.device
    _check_mx(a, a.rows, a.K, a.split, dev, "a")
    _check_mx(w, w.rows, w.K, w.split, dev, "w")
    if y is None:
        ldy = _round16(w.rows) if w.rows % 8 else w.rows
        y = torch.empty((a.rows, ldy), dtype=torch.bfloat16, device=dev)[:, : w.rows]
    elif (y.dtype != torch.bfloat16 or y.dim() != 2 or tuple(y.shape) != (a.rows, w.rows) or y.stride(1) != 1
          or y.device != dev):
        raise ValueError(f"y must be a bfloat16 [{a.rows}, {w.rows}] tensor with unit column stride on {dev}")
    da, dw = a.descriptor(), w.descriptor()
    _check(lib.mm_gemm(ctypes.byref(da), ctypes.byref(dw), ctypes.c_void_p(y.data_ptr()), y.stride(0),
                       _stream_ptr(stream)))
    return y


def calibrate_workspace_size(rows: int, K: int) -> int:
    """mm_calibrate_workspace_size: device bytes mm_calibrate needs."""
    n = ctypes.c_int64()
    _check(lib.mm_calibrate_workspace_size(rows, K, ctypes.byref(n)))
    return n.value


def calibrate_async(x: torch.Tensor, formats=DEFAULT_FORMATS, workspace: torch.Tensor | None = None,
                    perm: torch.Tensor | None = None, split: torch.Tensor | None = None, stream=None):
    """mm_calibrate: enqueue the offline channel assignment of bf16 calibration
    activations x [L, K]; returns the device tensors (perm int32 [K],
    split int32 [3]) it writes."""
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bfloat16 tensor")
    rows, K = x.shape
    if workspace is None:
        workspace = torch.empty(calibrate_workspace_size(rows, K), dtype=torch.uint8, device=x.device)
    if perm is None:
        perm = torch.empty(K, dtype=torch.int32, device=x.device)
    if split is None:
        split = torch.empty(3, dtype=torch.int32, device=x.device)
    fm = MMFormats(FP6_FORMATS.get(formats[0], -1), FP8_FORMATS.get(formats[1], -1))
    _check(lib.mm_calibrate(ctypes.c_void_p(x.data_ptr()), rows, K, x.stride(0), fm,
                            ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                            ctypes.c_void_p(perm.data_ptr()), ctypes.c_void_p(split.data_ptr()), _stream_ptr(stream)))
    return perm, split


def calibrate_no_alloc_async(x: torch.Tensor, perm: torch.Tensor, split: torch.Tensor, formats=DEFAULT_FORMATS,
                             stream=None):
    """mm_calibrate_no_alloc: mm_calibrate on the library's static scratch;
    the caller supplies the outputs (perm int32 [K], split int32 [3]) and no
    device memory is allocated anywhere in the call."""
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D row-major bfloat16 tensor")
    rows, K = x.shape
    if perm.dtype != torch.int32 or perm.numel() != K or not perm.is_contiguous() or perm.device != x.device:
        raise ValueError("perm must be a contiguous int32 tensor of K elements on x's device")
    if split.dtype != torch.int32 or split.numel() != 3 or not split.is_contiguous() or split.device != x.device:
        raise ValueError("split must be a contiguous int32 tensor of 3 elements on x's device")
    fm = MMFormats(FP6_FORMATS.get(formats[0], -1), FP8_FORMATS.get(formats[1], -1))
    _check(lib.mm_calibrate_no_alloc(ctypes.c_void_p(x.data_ptr()), rows, K, x.stride(0), fm,
                                     ctypes.c_void_p(perm.data_ptr()), ctypes.c_void_p(split.data_ptr()),
                                     _stream_ptr(stream)))
    return perm, split


def calibrate(x: torch.Tensor, formats=DEFAULT_FORMATS, stream=None):
    """mm_calibrate, then wait for it: (sigma as a device int32 tensor, split
    as a host tuple).  Raises ValueError if x holds Inf or NaN."""
    perm, split = calibrate_async(x, formats, stream=stream)
    p = tuple(int(v) for v in split.cpu().tolist())
    if p[0] < 0:
        raise ValueError("calibration input holds Inf or NaN")
    return perm, p
