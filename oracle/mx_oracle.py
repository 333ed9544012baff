"""Plain CPU oracle for MicroMix's hot path (arXiv 2508.02343).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code with the HIP kernels.

Everything is written for readability, in float64 numpy, following the
paper's definitions in the order the paper gives them:

* Microscaling block quantisation (Sec. 2.1, the MX quantisation equation):
  a block of k = 32 elements shares one power-of-two scale
  s = 2^(floor(log2 max|X_i|) - b) stored as E8M0, and every element is
  Q(X_j) = round(X_j / s), round = nearest representable MX value.
* Element formats and their constants (Appendix B, Table "tab:microscaling"):
  E2M1 (MXFP4), E3M2 / E2M3 (MXFP6), E4M3 / E5M2 (MXFP8).
* Channel permutation and three-way split (Sec. 3.1, "Reducing quantization
  error through permutation" and "Offline channel assignment strategy"):
  X' = sigma(X) gathers channels, G4 = X'[:, :p4], G6 = X'[:, p4:p4+p6],
  G8 = X'[:, p4+p6:]; weights are permuted with the same sigma and get the
  same bit-widths (Sec. 3.2, "Quantization kernel").
* The quantised linear layer Y = X W ~ Q(X) Q(W) s_X s_W (Sec. 2.1, eq. 1),
  computed here as the exact float64 product of the dequantised operands,
  with a single accumulation over all three partitions (Sec. 3.2, "GEMM
  kernel": FP32 partial sums into a BFloat16 result).

Readings where the paper is silent or ambiguous (each one is listed with its
justification in the design notes of the repository):

R1  b is read as the element format's largest binade exponent emax
    (E2M1 2, E3M2 4, E2M3 2, E4M3 8, E5M2 15), the OCP MX rule.  With the
    table's exponent bias instead, the top binade of E2M1/E3M2/E2M3/E4M3
    would never be used.
R2  round() is round-to-nearest, ties to the even code.
R3  |X/s| above the largest normal saturates to +-max normal.
R4  an all-zero block gets scale exponent -127 (E8M0 byte 0x00).
R5  the scale exponent is clamped to the E8M0 range [-127, 127].
R6  the code keeps the sign of the input, so -0.0 and negative values that
    round to zero give the negative-zero code.
R7  sigma is a gather: X'[:, j] = X[:, sigma[j]].
R8  the third group is X'[:, p4+p6 : K] (the printed upper bound p8*I is
    read as the end of the row).
R9  blocks run along K inside one row, never straddling a partition.
R10 input X and W are bfloat16 bit patterns; Y = X W^T with W stored [N, K].
R11 p4, p6, p8 are channel counts, multiples of 32, zero allowed.
R12 storage: FP4 two codes per byte (even element in the low nibble); FP6
    four codes per three bytes as a little-endian bit stream (code i at bits
    6i..6i+5 of its 24-byte block); FP8 one code per byte; one E8M0 byte per
    block, row-major, in X' block order.
R13 calibration: a channel's statistic against the thresholds T(4), T(6) is
    its mean |X| over the calibration rows (the key sigma sorts by), so every
    group is a contiguous slice of sigma; max|X| in Ebar_INT8 = max|X| / 254 is
    taken over the whole calibration tensor; the counts are rounded down to
    multiples of 32 (channels move to the next wider group, never to a
    narrower one); T(6) uses the constants of the MXFP6 variant in use.
R14 the normalisation fused with the reorder-and-quantize is RMSNorm (the
    norm of the Llama and Qwen models the paper evaluates), evaluated as bf16
    frameworks do: the row factor r = 1/sqrt(mean(x^2) + eps) in float64,
    rounded once to fp32; x * r as an fp32 product rounded to bf16; that
    times the bf16 weight gamma as an fp32 product rounded to bf16 again.
    The quantiser then sees these bf16 values.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

BLOCK = 32  # k, the MX scaling block size (Appendix B table)


# ---------------------------------------------------------------------------
# Element formats (Appendix B, Table "tab:microscaling")
# ---------------------------------------------------------------------------


@dataclass(frozen=True)
class MXFormat:
    name: str
    ebits: int  # exponent field width
    mbits: int  # mantissa field width
    bias: int  # exponent bias (Appendix B table, column b)
    # True for E4M3 (OCP "FN" flavour): only S.1111.111 is NaN, no infinities.
    # False with ebits>=5 means IEEE-like: the all-ones exponent is Inf/NaN.
    # Formats of 4 or 6 bits have no special values at all.
    fn_nan_only: bool

    @property
    def bits(self) -> int:
        return 1 + self.ebits + self.mbits

    @property
    def emin(self) -> int:
        # exponent of the smallest normal binade (also of the subnormals)
        return 1 - self.bias

    def is_finite_code(self, code: int) -> bool:
        mag = code & ((1 << (self.bits - 1)) - 1)
        e = mag >> self.mbits
        m = mag & ((1 << self.mbits) - 1)
        top = (1 << self.ebits) - 1
        if self.bits < 8:
            return True
        if self.fn_nan_only:
            return not (e == top and m == (1 << self.mbits) - 1)
        return e != top

    def decode(self, code: int) -> float:
        """Exact value of one element code (sign | exponent | mantissa)."""
        if not self.is_finite_code(code):
            raise ValueError(f"{self.name}: code {code:#x} is not finite")
        sign = -1.0 if (code >> (self.bits - 1)) & 1 else 1.0
        mag = code & ((1 << (self.bits - 1)) - 1)
        e = mag >> self.mbits
        m = mag & ((1 << self.mbits) - 1)
        if e == 0:  # subnormal: 2^emin * m / 2^mbits
            v = math.ldexp(m, self.emin - self.mbits)
        else:  # normal: 2^(e-bias) * (1 + m / 2^mbits)
            v = math.ldexp((1 << self.mbits) + m, e - self.bias - self.mbits)
        return sign * v

    def finite_codes(self) -> list[int]:
        return [c for c in range(1 << self.bits) if self.is_finite_code(c)]

    @property
    def max_normal(self) -> float:
        return max(self.decode(c) for c in self.finite_codes())

    @property
    def emax(self) -> int:
        # exponent of the largest binade that holds finite values (reading R1)
        return math.frexp(self.max_normal)[1] - 1

    def positive_values(self) -> np.ndarray:
        """Values of the non-negative codes, indexed by code magnitude."""
        n = 1 << (self.bits - 1)
        vals = [self.decode(c) if self.is_finite_code(c) else np.nan for c in range(n)]
        return np.array(vals, dtype=np.float64)


E2M1 = MXFormat("E2M1", 2, 1, 1, False)
E3M2 = MXFormat("E3M2", 3, 2, 3, False)
E2M3 = MXFormat("E2M3", 2, 3, 1, False)
E4M3 = MXFormat("E4M3", 4, 3, 7, True)
E5M2 = MXFormat("E5M2", 5, 2, 15, False)

FORMATS = {f.name: f for f in (E2M1, E3M2, E2M3, E4M3, E5M2)}

# The formats MicroMix uses for its three groups (Sec. 4.1 "Quantization").
PARTITION_FORMATS = (E2M1, E3M2, E4M3)
# The alternatives its ablation compares (Table "tab:ablation-study-mxfp6-mxfp8"):
# MXFP6 as E2M3 instead of E3M2, MXFP8 as E5M2 instead of E4M3.
GROUP_FORMAT_CHOICES = ((E2M1,), (E3M2, E2M3), (E4M3, E5M2))


def check_formats(formats) -> tuple:
    formats = tuple(formats)
    if len(formats) != 3 or any(f not in choices for f, choices in zip(formats, GROUP_FORMAT_CHOICES)):
        raise ValueError("formats must be (E2M1, E3M2 | E2M3, E4M3 | E5M2)")
    return formats


# ---------------------------------------------------------------------------
# bfloat16 <-> float64 (inputs are bf16 bit patterns; output is bf16)
# ---------------------------------------------------------------------------


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns (the top half of an fp32 word)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 to the nearest bf16, ties to even (finite inputs).

    Done in two exact steps so that no double rounding can occur: the bf16
    grid at x's binade has quantum 2^(E-7); rint(x / q) * q is exact in
    float64, and the result is representable in fp32 exactly.
    """
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    _, ex = np.frexp(a)
    E = np.maximum(ex - 1, -126)  # bf16 normals start at 2^-126
    q = np.ldexp(1.0, E - 7)
    r = np.rint(a / q) * q
    r = np.copysign(r, x)
    return (r.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


# ---------------------------------------------------------------------------
# MX block quantisation (Sec. 2.1, MX quantisation equation)
# ---------------------------------------------------------------------------


def block_scale_exponent(amax: np.ndarray, fmt: MXFormat) -> np.ndarray:
    """Shared-scale exponent e with s = 2^e = 2^(floor(log2 amax) - emax).

    Readings R1 (emax), R4 (zero block -> -127) and R5 (clamp to E8M0).
    floor(log2 amax) is taken from frexp, which is exact.
    """
    amax = np.asarray(amax, dtype=np.float64)
    _, ex = np.frexp(amax)  # amax = m * 2^ex with m in [0.5, 1)
    e = (ex.astype(np.int64) - 1) - fmt.emax
    e = np.clip(e, -127, 127)
    return np.where(amax == 0.0, -127, e).astype(np.int64)


def round_to_format(v: np.ndarray, fmt: MXFormat) -> np.ndarray:
    """Nearest representable magnitude of |v| in fmt (readings R2, R3).

    In the binade of |v| the grid spacing is 2^(E - mbits), E = max(floor(
    log2|v|), emin); rint() of |v| over that spacing is exact in float64 and
    rounds ties to even, then the result saturates at the max normal.
    """
    a = np.abs(np.asarray(v, dtype=np.float64))
    _, ex = np.frexp(a)
    E = np.maximum(ex.astype(np.int64) - 1, fmt.emin)
    q = np.ldexp(1.0, E - fmt.mbits)
    r = np.rint(a / q) * q
    return np.minimum(r, fmt.max_normal)


def encode_scaled(v: np.ndarray, fmt: MXFormat) -> np.ndarray:
    """Element codes of already-scaled values v = X / s (reading R6 for sign)."""
    v = np.asarray(v, dtype=np.float64)
    mag = round_to_format(v, fmt)
    table = fmt.positive_values()
    order = np.where(np.isfinite(table))[0]
    vals = table[order]  # increasing with the code magnitude
    idx = np.searchsorted(vals, mag)
    if not np.all(vals[np.minimum(idx, len(vals) - 1)] == mag):
        raise AssertionError("rounded value is not on the format grid")
    code = order[idx].astype(np.int64)
    sign = np.signbit(v).astype(np.int64) << (fmt.bits - 1)
    return (code | sign).astype(np.uint8)


def decode_codes(codes: np.ndarray, fmt: MXFormat) -> np.ndarray:
    """Vectorised decode of element codes to float64."""
    lut = np.array(
        [fmt.decode(c) if fmt.is_finite_code(c) else np.nan for c in range(1 << fmt.bits)],
        dtype=np.float64,
    )
    return lut[np.asarray(codes, dtype=np.int64)]


def quantize_blocks(x: np.ndarray, fmt: MXFormat):
    """MX-quantise the rows of x (float64 [R, n*32]) block by block.

    Returns (codes uint8 [R, n*32], scale exponents int64 [R, n]).
    """
    x = np.asarray(x, dtype=np.float64)
    R, C = x.shape
    assert C % BLOCK == 0
    xb = x.reshape(R, C // BLOCK, BLOCK)
    amax = np.max(np.abs(xb), axis=2) if C else np.zeros((R, 0))
    e = block_scale_exponent(amax, fmt)
    v = np.ldexp(xb, -e[:, :, None])  # X / s, exact (power-of-two scale)
    codes = encode_scaled(v, fmt).reshape(R, C)
    return codes, e


def dequantize_blocks(codes: np.ndarray, e: np.ndarray, fmt: MXFormat) -> np.ndarray:
    """s * x_i for every element (Appendix B: the original value is s x_i)."""
    R, C = codes.shape
    vals = decode_codes(codes, fmt).reshape(R, C // BLOCK, BLOCK)
    return np.ldexp(vals, np.asarray(e)[:, :, None]).reshape(R, C)


# ---------------------------------------------------------------------------
# Packing (reading R12)
# ---------------------------------------------------------------------------


def pack_fp4(codes: np.ndarray) -> np.ndarray:
    c = np.asarray(codes, dtype=np.uint8)
    return (c[:, 0::2] & 0xF) | ((c[:, 1::2] & 0xF) << 4)


def unpack_fp4(packed: np.ndarray, n: int) -> np.ndarray:
    p = np.asarray(packed, dtype=np.uint8)[:, : n // 2]
    out = np.empty((p.shape[0], n), dtype=np.uint8)
    out[:, 0::2] = p & 0xF
    out[:, 1::2] = p >> 4
    return out


def pack_fp6(codes: np.ndarray) -> np.ndarray:
    c = np.asarray(codes, dtype=np.uint32)
    R, n = c.shape
    g = c.reshape(R, n // 4, 4)
    word = g[:, :, 0] | (g[:, :, 1] << 6) | (g[:, :, 2] << 12) | (g[:, :, 3] << 18)
    out = np.empty((R, n // 4, 3), dtype=np.uint8)
    out[:, :, 0] = word & 0xFF
    out[:, :, 1] = (word >> 8) & 0xFF
    out[:, :, 2] = (word >> 16) & 0xFF
    return out.reshape(R, 3 * n // 4)


def unpack_fp6(packed: np.ndarray, n: int) -> np.ndarray:
    p = np.asarray(packed, dtype=np.uint32)[:, : 3 * n // 4]
    R = p.shape[0]
    t = p.reshape(R, n // 4, 3)
    word = t[:, :, 0] | (t[:, :, 1] << 8) | (t[:, :, 2] << 16)
    out = np.empty((R, n // 4, 4), dtype=np.uint8)
    for i in range(4):
        out[:, :, i] = (word >> (6 * i)) & 0x3F
    return out.reshape(R, n)


# ---------------------------------------------------------------------------
# Reorder + three-partition quantisation (Sec. 3.1 and Sec. 3.2)
# ---------------------------------------------------------------------------


def check_split(K: int, split) -> tuple[int, int, int]:
    p4, p6, p8 = (int(p) for p in split)
    if min(p4, p6, p8) < 0 or any(p % BLOCK for p in (p4, p6, p8)) or p4 + p6 + p8 != K:
        raise ValueError(f"bad split {split} for K={K}")
    return p4, p6, p8


def check_perm(perm: np.ndarray, K: int) -> np.ndarray:
    perm = np.asarray(perm, dtype=np.int64)
    if perm.shape != (K,) or not np.array_equal(np.sort(perm), np.arange(K)):
        raise ValueError("perm is not a permutation of [0, K)")
    return perm


@dataclass
class MXTensor:
    """One quantised operand: rows x K in X' (permuted) channel order."""

    q4: np.ndarray  # uint8 [rows, p4/2]
    q6: np.ndarray  # uint8 [rows, 3*p6/4]
    q8: np.ndarray  # uint8 [rows, p8]
    sc: np.ndarray  # uint8 [rows, K/32], E8M0 bytes (exponent + 127)
    split: tuple[int, int, int]
    formats: tuple = PARTITION_FORMATS  # element format of each group

    @property
    def rows(self) -> int:
        return self.sc.shape[0]

    @property
    def K(self) -> int:
        return sum(self.split)


def reorder(x: np.ndarray, perm: np.ndarray) -> np.ndarray:
    """X'[:, j] = X[:, sigma[j]] (reading R7)."""
    return np.asarray(x)[:, np.asarray(perm, dtype=np.int64)]


def quantize_mixed(x_bf16_bits: np.ndarray, perm: np.ndarray, split, formats=PARTITION_FORMATS) -> MXTensor:
    """Reorder, split into G4/G6/G8 and MX-quantise each group.

    x_bf16_bits: uint16 [rows, K] bf16 patterns (finite).  Used unchanged for
    activations (online) and weights (offline, same sigma and split).
    formats: element format of each group, (E2M1, E3M2, E4M3) by default;
    the 6-bit group may use E2M3 and the 8-bit group E5M2 instead.
    """
    f4, f6, f8 = check_formats(formats)
    bits = np.asarray(x_bf16_bits, dtype=np.uint16)
    rows, K = bits.shape
    p4, p6, p8 = check_split(K, split)
    perm = check_perm(perm, K)
    x = bf16_bits_to_f64(bits)
    if not np.all(np.isfinite(x)):
        raise ValueError("input holds Inf or NaN")
    xp = reorder(x, perm)
    g4, g6, g8 = xp[:, :p4], xp[:, p4 : p4 + p6], xp[:, p4 + p6 :]
    c4, e4 = quantize_blocks(g4, f4)
    c6, e6 = quantize_blocks(g6, f6)
    c8, e8 = quantize_blocks(g8, f8)
    e = np.concatenate([e4, e6, e8], axis=1) if K else np.zeros((rows, 0), np.int64)
    return MXTensor(
        q4=pack_fp4(c4),
        q6=pack_fp6(c6),
        q8=c8.astype(np.uint8),
        sc=(e + 127).astype(np.uint8),
        split=(p4, p6, p8),
        formats=(f4, f6, f8),
    )


def element_codes(t: MXTensor):
    """Unpacked codes of the three groups (for inspection and tests)."""
    p4, p6, p8 = t.split
    return unpack_fp4(t.q4, p4), unpack_fp6(t.q6, p6), np.asarray(t.q8)[:, :p8]


def dequantize_mixed(t: MXTensor) -> np.ndarray:
    """Float64 [rows, K] values s * x_i of all three groups, X' order."""
    p4, p6, p8 = t.split
    c4, c6, c8 = element_codes(t)
    e = np.asarray(t.sc, dtype=np.int64)[:, : t.K // BLOCK] - 127
    b4, b6 = p4 // BLOCK, (p4 + p6) // BLOCK
    f4, f6, f8 = t.formats
    parts = [
        dequantize_blocks(c4, e[:, :b4], f4),
        dequantize_blocks(c6, e[:, b4:b6], f6),
        dequantize_blocks(c8, e[:, b6:], f8),
    ]
    return np.concatenate(parts, axis=1)


# ---------------------------------------------------------------------------
# Mixed-precision GEMM (Sec. 2.1 eq. 1, Sec. 3.2 "GEMM kernel")
# ---------------------------------------------------------------------------


def gemm_mixed(a: MXTensor, w: MXTensor) -> np.ndarray:
    """Y[m, n] = sum over all three partitions of dq(A)[m, :] . dq(W)[n, :].

    Float64.  Every product of two dequantised values is exact in float64,
    so the only error is float64 summation order (about K * 2^-53 relative).
    """
    if a.split != w.split:
        raise ValueError("activation and weight must share the split")
    if tuple(a.formats) != tuple(w.formats):
        raise ValueError("activation and weight must share the group formats")
    return dequantize_mixed(a) @ dequantize_mixed(w).T


def gemm_tolerance(y_ref: np.ndarray) -> np.ndarray:
    """Elementwise bound |y - y_ref| <= 2^-8 |y_ref| + 1e-3 rms(y_ref)."""
    y_ref = np.asarray(y_ref, dtype=np.float64)
    rms = math.sqrt(float(np.mean(y_ref * y_ref))) if y_ref.size else 0.0
    return np.ldexp(np.abs(y_ref), -8) + 1e-3 * rms


def average_bits(split) -> float:
    """Average storage bits per element incl. the 8-bit scale per 32 (App. C)."""
    p4, p6, p8 = split
    K = p4 + p6 + p8
    return (4 * p4 + 6 * p6 + 8 * p8) / K + 8 / BLOCK


# ---------------------------------------------------------------------------
# Offline calibration (Sec. 3.1 "Offline Channel Assignment Strategy";
# Def. 1 eq. quantization-threshold; Appendix "Derivations" eq. last)
# ---------------------------------------------------------------------------


def quantization_threshold(fmt: MXFormat, amax_tensor: float) -> float:
    """T(n) = 2^b * 2^(n-1) / q_max * Ebar_INT8 with Ebar_INT8 = max|X| / 254
    (the INT8 per-tensor error bound), b the format's exponent bias and q_max
    its largest value (Table "tab:microscaling")."""
    return 2.0 ** fmt.bias * 2.0 ** (fmt.bits - 1) / fmt.max_normal * (amax_tensor / 254.0)


def channel_abs_mean(x_bf16_bits: np.ndarray) -> np.ndarray:
    """M_j = (1/L) sum_i |X_ij| over the L calibration rows, float64."""
    x = bf16_bits_to_f64(np.asarray(x_bf16_bits, dtype=np.uint16))
    return np.abs(x).sum(axis=0) / x.shape[0]


def calibrate(x_bf16_bits: np.ndarray, formats=PARTITION_FORMATS):
    """(sigma, split) from calibration activations X [L, K] (bf16 patterns).

    sigma: int32 [K], the stable ascending argsort of the channel absolute
    means M.  split: the group sizes from the thresholds T(4) (E2M1) and T(6)
    (the MXFP6 format of `formats`) against M under reading R13:
    p4 = 32 floor(n4/32), p4 + p6 = 32 floor((n4 + n6)/32), p8 the rest.
    """
    f4, f6, _ = check_formats(formats)
    bits = np.asarray(x_bf16_bits, dtype=np.uint16)
    if bits.ndim != 2:
        raise ValueError("X must be [L, K]")
    L, K = bits.shape
    if L == 0 or K == 0 or K % BLOCK:
        raise ValueError("need rows > 0 and K a positive multiple of 32")
    x = bf16_bits_to_f64(bits)
    if not np.all(np.isfinite(x)):
        raise ValueError("input holds Inf or NaN")
    M = np.abs(x).sum(axis=0) / L
    sigma = np.argsort(M, kind="stable").astype(np.int32)
    t = float(np.abs(x).max())
    T4, T6 = quantization_threshold(f4, t), quantization_threshold(f6, t)
    n4 = int(np.count_nonzero(M <= T4))
    n6 = int(np.count_nonzero((M > T4) & (M <= T6)))
    p4 = n4 // BLOCK * BLOCK
    p46 = (n4 + n6) // BLOCK * BLOCK
    return sigma, (p4, p46 - p4, K - p46)


# ---------------------------------------------------------------------------
# RMSNorm fused before the reorder-and-quantize (App. D.2, Fig.
# "precision-mapping": the reorder-and-quantize runs inside the layer's
# normalisation; reading R14)
# ---------------------------------------------------------------------------


def rmsnorm_bf16(x_bf16_bits: np.ndarray, gamma_bf16_bits: np.ndarray, eps: float) -> np.ndarray:
    """bf16 bit patterns of RMSNorm(X)[i, j] = gamma_j * X_ij / sqrt(mean_j X_ij^2 + eps),
    with the roundings of reading R14."""
    r32 = rmsnorm_row_factor(x_bf16_bits, eps).astype(np.float32)  # one rounding, to nearest even
    return rmsnorm_apply(x_bf16_bits, gamma_bf16_bits, r32)


def rmsnorm_row_factor(x_bf16_bits: np.ndarray, eps: float) -> np.ndarray:
    """The float64 row factors r = 1/sqrt(mean(x^2) + eps), before their
    rounding to fp32."""
    x = bf16_bits_to_f64(np.asarray(x_bf16_bits, dtype=np.uint16))
    if x.ndim != 2:
        raise ValueError("X must be [L, K]")
    ms = (x * x).sum(axis=1) / x.shape[1]  # every square of a bf16 value is exact in float64
    return 1.0 / np.sqrt(ms + float(np.float32(eps)))


def rmsnorm_apply(x_bf16_bits: np.ndarray, gamma_bf16_bits: np.ndarray, r32: np.ndarray) -> np.ndarray:
    """bf16(gamma_j * bf16(x_ij * r_i)) for given fp32 row factors r: both
    products in fp32 (exact inputs), each rounded to nearest even."""
    x = bf16_bits_to_f64(np.asarray(x_bf16_bits, dtype=np.uint16))
    g = bf16_bits_to_f64(np.asarray(gamma_bf16_bits, dtype=np.uint16))
    r32 = np.asarray(r32, dtype=np.float32)
    if x.ndim != 2 or g.shape != (x.shape[1],) or r32.shape != (x.shape[0],):
        raise ValueError("X must be [L, K], gamma [K] and r [L]")
    t = x.astype(np.float32) * r32[:, None]
    y1 = f64_to_bf16_bits(t.astype(np.float64))
    u = bf16_bits_to_f64(y1).astype(np.float32) * g.astype(np.float32)[None, :]
    return f64_to_bf16_bits(u.astype(np.float64))
