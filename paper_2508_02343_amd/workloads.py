"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and lays them out: it holds none of
the quantisation or GEMM arithmetic, so both the HIP path and the CPU oracle
can take their inputs from it.

The paper quantises real Llama-3.1-8B / Qwen2.5 activations (Sec. 3.1,
Fig. "p4-p6-p8-llama"; Sec. 4.3, Table "ablation:each-part-time").  Those are
not available, so each configuration below stands in for them with the same
layer shape, a heavy-tailed channel-outlier structure (a few channels scaled
up, as in Fig. "motivation1", where outlier channels end up last after the
reordering) and a split of roughly 5 bits per element with p4 > 50 %
(Sec. 3.1 "FP4 dominance"; App. D.2 "5-5.6 bits").

The permutation puts every regular channel first, in a seeded random order
(what sorting the channel mean |X| of i.i.d. channels yields), and the
outlier channels last.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite float32 values to bf16 (nearest, ties to even)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


@dataclass(frozen=True)
class Workload:
    name: str
    M: int
    K: int
    N: int
    split: tuple[int, int, int]
    seed: int
    x_dist: str = "normal"  # "normal" or "student_t3"
    outlier_frac: float = 0.01
    n_outliers: int | None = None  # overrides outlier_frac when given
    outlier_scale: float = 30.0
    w_std: float = 0.02
    identity_regular_order: bool = False  # regular channels kept in index order
    description: str = field(default="", compare=False)

    @property
    def outliers(self) -> int:
        if self.n_outliers is not None:
            return self.n_outliers
        return int(round(self.outlier_frac * self.K))

    # -- generators --------------------------------------------------------

    def _outlier_channels(self) -> np.ndarray:
        rng = np.random.default_rng([self.seed, 0])
        return np.sort(rng.choice(self.K, size=self.outliers, replace=False))

    def x_bits(self, rows: int | None = None) -> np.ndarray:
        """Activation X as bf16 bits, uint16 [M, K] (or the first `rows`)."""
        M = self.M if rows is None else rows
        rng = np.random.default_rng([self.seed, 0])
        out_ch = np.sort(rng.choice(self.K, size=self.outliers, replace=False))
        if self.x_dist == "normal":
            x = rng.standard_normal((M, self.K), dtype=np.float32)
        elif self.x_dist == "student_t3":
            x = rng.standard_t(3, size=(M, self.K)).astype(np.float32)
        else:
            raise ValueError(self.x_dist)
        x[:, out_ch] *= np.float32(self.outlier_scale)
        return f32_to_bf16_bits(x)

    def w_bits(self, rows: int | None = None) -> np.ndarray:
        """Weight W as bf16 bits, uint16 [N, K] (or the first `rows`)."""
        N = self.N if rows is None else rows
        rng = np.random.default_rng([self.seed, 1])
        w = rng.standard_normal((N, self.K), dtype=np.float32)
        w *= np.float32(self.w_std)
        return f32_to_bf16_bits(w)

    def perm(self) -> np.ndarray:
        """int32 [K] gather permutation: regular channels first, outliers last."""
        out_ch = self._outlier_channels()
        is_out = np.zeros(self.K, dtype=bool)
        is_out[out_ch] = True
        regular = np.nonzero(~is_out)[0]
        rng = np.random.default_rng([self.seed, 2])
        if not self.identity_regular_order:
            regular = rng.permutation(regular)
            out_ch = rng.permutation(out_ch)
        return np.concatenate([regular, out_ch]).astype(np.int32)

    def with_shape(self, M: int | None = None, N: int | None = None, name: str | None = None):
        kw = dict(self.__dict__)
        if M is not None:
            kw["M"] = M
        if N is not None:
            kw["N"] = N
        if name is not None:
            kw["name"] = name
        return Workload(**kw)


def calibration_bits(rows: int, K: int, seed: int, channel_sigma: float = 1.0) -> np.ndarray:
    """Calibration activations, bf16 bits uint16 [rows, K]: token values
    N(0, 1) times a per-channel scale exp(N(0, channel_sigma)).  With the
    default spread the thresholds assign about 53 / 37 / 10 % of the channels
    to the 4 / 6 / 8-bit groups (about 5.4 bits per element), the range the
    paper reports for Llama and Qwen layers, and the split hardly moves with
    the number of rows."""
    rng = np.random.default_rng([seed, 7])
    scale = np.exp(rng.normal(0.0, channel_sigma, K)).astype(np.float32)
    x = rng.standard_normal((rows, K), dtype=np.float32) * scale
    return f32_to_bf16_bits(x)


def _split(K: int, f4: float, f6: float) -> tuple[int, int, int]:
    p4 = int(round(K * f4 / 32)) * 32
    p6 = int(round(K * f6 / 32)) * 32
    return p4, p6, K - p4 - p6


# The five configurations.  Sizes follow Llama-3-8B (hidden 4096, MLP 14336)
# and Qwen2.5-32B (hidden 5120, MLP 27648) linear layers.
TINY = Workload(
    "tiny_16x512x512", 16, 512, 512, (384, 64, 64), seed=0,
    n_outliers=4, outlier_scale=20.0, identity_regular_order=True,
    description="tiny layer, 4 outlier channels x20",
)
LLAMA_ATTN = Workload(
    "llama8b_attn_2048x4096x4096", 2048, 4096, 4096, (3072, 768, 256), seed=1,
    description="Llama-3-8B attention projection, prefill 2048 tokens",
)
LLAMA_MLP_UP = Workload(
    "llama8b_mlp_up_4096x4096x14336", 4096, 4096, 14336, _split(4096, 0.75, 0.1875), seed=2,
    description="Llama-3-8B gate/up projection, prefill 4096 tokens",
)
LLAMA_MLP_DOWN = Workload(
    "llama8b_mlp_down_4096x14336x4096", 4096, 14336, 4096, _split(14336, 0.75, 0.1875), seed=2,
    description="Llama-3-8B down projection, prefill 4096 tokens",
)
QWEN_MLP_UP = Workload(
    "qwen32b_mlp_up_8192x5120x27648", 8192, 5120, 27648, (3584, 1024, 512), seed=3,
    x_dist="student_t3", outlier_frac=0.005, outlier_scale=50.0, w_std=0.015,
    description="Qwen2.5-32B MLP up projection, Student-t(3) activations",
)

DECODE_SPLITS = {"fp4": (4096, 0, 0), "fp8": (0, 0, 4096), "mix": (2048, 1024, 1024)}


def decode_workloads() -> list[Workload]:
    out = []
    for M in (1, 8, 32):
        for N in (4096, 14336):
            for tag, sp in DECODE_SPLITS.items():
                out.append(Workload(f"decode_m{M}_n{N}_{tag}", M, 4096, N, sp, seed=4))
    return out


PREFILL = [LLAMA_ATTN, LLAMA_MLP_UP, LLAMA_MLP_DOWN, QWEN_MLP_UP]
ALL = [TINY] + PREFILL + decode_workloads()
BY_NAME = {w.name: w for w in ALL}
