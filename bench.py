"""Benchmark of the MicroMix hot path on one MI355X.

A step is one pass of the online path over one batch: fused reorder-and-
quantize of the bf16 activation (mm_quantize_act) followed by the mixed
MXFP4/6/8 GEMM (mm_gemm) against an offline-quantised weight.  Weight
quantisation (mm_quantize_weight) runs once per weight and is timed apart.

Prints one JSON line: whole-step throughput in TFLOP/s (2 M N K per step),
the GEMM's roofline against the MFMA peak of its bit mix, the quantiser's HBM
bandwidth, the CPU oracle timed on the host as a baseline, and (outside the
step) the offline calibration's HBM bandwidth on a calibration set of the
layer's width.

Inputs are seeded synthetic tensors resident in HBM before the timed region;
several buffer sets are rotated so the working set exceeds the 256 MB
Infinity Cache.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published dense peaks (TFLOP/s) and HBM bandwidth (GB/s).
PEAK_FP4_FP6 = 10100.0
PEAK_FP8 = 5000.0
PEAK_HBM = 8000.0


def mix_peak_tflops(split) -> float:
    """MFMA peak for the bit mix: FP4 and FP6 run at the FP4 rate, FP8 at half."""
    p4, p6, p8 = split
    K = p4 + p6 + p8
    t = (p4 + p6) / K / PEAK_FP4_FP6 + p8 / K / PEAK_FP8
    return 1.0 / t


def quant_bytes(rows: int, K: int, split) -> int:
    """Algorithmic bytes of one quantiser launch: bf16 read, codes and scales
    written, sigma read once."""
    p4, p6, p8 = split
    return rows * K * 2 + rows * (p4 // 2 + 3 * p6 // 4 + p8) + rows * K // 32 + 4 * K


DIRECT_MAX_M = 64  # mm_gemm takes the HBM-bound decode kernel up to this many activation rows


def gemm_bytes(M: int, N: int, K: int, split) -> int:
    """Algorithmic bytes of one GEMM launch: packed A and W (codes + scales)
    read once, bf16 Y written once."""
    p4, p6, p8 = split
    row = p4 // 2 + 3 * p6 // 4 + p8 + K // 32
    return M * row + N * row + M * N * 2


# sources each GEMM kernel is compiled from (a committed counter summary is
# used only while they are unchanged)
GEMM_SOURCES = {"tiled": ("gemm_tiled.hip", "gemm_common.hpp", "mx_device.hpp", "kernels.hpp"),
                "direct": ("gemm_direct.hip", "gemm_common.hpp", "mx_device.hpp", "kernels.hpp")}
CALIB_BYTES = 256 << 20  # plain copy used to calibrate the FETCH_SIZE / WRITE_SIZE counters


def gemm_source_hash(kind: str = "tiled") -> str:
    import hashlib

    h = hashlib.sha256()
    for f in GEMM_SOURCES[kind]:
        with open(os.path.join(ROOT, "paper_2508_02343_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _profile_entry(fname: str, workload: str):
    """A workload's entry of a committed rocprofv3 counter summary, or None
    when the summary is missing or was taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", fname)
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    entry = rec.get(workload)
    if not entry:
        return None
    from paper_2508_02343_amd import workloads as W

    kind = "direct" if W.BY_NAME[workload].M <= DIRECT_MAX_M else "tiled"
    if entry.get("source_hash") != gemm_source_hash(kind):
        return None
    return entry


def measured_traffic(workload: str):
    """HBM bytes per GEMM launch (rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE,
    scaled by a plain copy's counts), or None."""
    e = _profile_entry("gemm_traffic.json", workload)
    return None if e is None else e.get("hbm_bytes_per_launch")


def measured_mfma_util(workload: str):
    """Fraction of the GEMM's active cycles its matrix cores were busy
    (rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES over GRBM_GUI_ACTIVE per SIMD),
    with the clock the counters imply, or None."""
    e = _profile_entry("gemm_mfma.json", workload)
    return None if e is None else {"mfma_busy": e.get("mfma_busy"), "clock_GHz": e.get("clock_GHz")}


def cpu_threads() -> tuple[int, int]:
    """(threads used, os.cpu_count()): the host's cores, at most the 16 a
    one-GPU share of a GPU host gets."""
    n = os.cpu_count() or 1
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        avail = n
    return max(1, min(avail, 16)), n


def cpu_baseline(w, seconds: float) -> dict:
    """The oracle (float64 numpy) on a bounded sample of the workload, its
    BLAS pool set to the host's threads: the quantiser on a slice of the
    activation rows (GB/s over the same algorithmic bytes the GPU kernel is
    charged) and the GEMM of that slice with the full, pre-quantised weight
    (GFLOPS); value is the whole step (quantise + GEMM) in the metric's unit."""
    from oracle import mx_oracle as O

    threads, ncpu = cpu_threads()
    try:
        from threadpoolctl import threadpool_limits
    except ImportError:  # pragma: no cover
        threadpool_limits = None
    rows = min(w.M, 256)
    xb, wb, perm = w.x_bits(rows), w.w_bits(), w.perm()

    def run():
        wq = O.quantize_mixed(wb, perm, w.split)

        def loop(fn, budget):
            fn()  # one untimed call first (allocator and BLAS warm-up)
            n, t0 = 0, time.perf_counter()
            while True:
                out = fn()
                n += 1
                el = time.perf_counter() - t0
                if el >= budget:
                    return out, n, el

        a, nq, tq = loop(lambda: O.quantize_mixed(xb, perm, w.split), seconds / 3)
        _, ng, tg = loop(lambda: O.gemm_mixed(a, wq), 2 * seconds / 3)
        return nq, tq, ng, tg

    if threadpool_limits is not None:
        with threadpool_limits(limits=threads):
            nq, tq, ng, tg = run()
    else:  # pragma: no cover
        nq, tq, ng, tg = run()
    q_s, g_s = tq / nq, tg / ng
    flops = 2.0 * rows * w.N * w.K
    return {"value": flops / (q_s + g_s) / 1e12, "unit": "TFLOP/s", "cores": threads, "os_cpu_count": ncpu,
            "kind": "oracle",
            "quantize_GBps": round(quant_bytes(rows, w.K, w.split) / q_s / 1e9, 4),
            "gemm_GFLOPS": round(flops / g_s / 1e9, 3),
            "sample": f"{rows} of {w.M} activation rows x full weight [{w.N},{w.K}]: quantise {nq} times in "
                      f"{tq:.1f} s, GEMM {ng} times in {tg:.1f} s (weight quantised once, untimed); "
                      f"BLAS threads {threads}"}


def measure_calibration(B, W, w, stream, dev, rows: int, min_set_mb: float, reps: int = 10) -> dict:
    """mm_calibrate over `rows` calibration tokens of the layer's width K
    (offline, not part of the step): whole-call time (a graph of `reps`
    calls, HIP events around its replays), and HBM bandwidth over the bytes it must move (X read once,
    sigma and the split written)."""
    import torch

    xb = W.calibration_bits(rows, w.K, 1)
    x0 = torch.from_numpy(xb.view(np.int16)).view(torch.bfloat16).to(dev)
    del xb
    nset = max(1, int(np.ceil(min_set_mb * 1e6 / (rows * w.K * 2))))
    xs = [x0] + [x0.clone() for _ in range(nset - 1)]
    ws = torch.empty(B.calibrate_workspace_size(rows, w.K), dtype=torch.uint8, device=dev)
    perm = torch.empty(w.K, dtype=torch.int32, device=dev)
    split = torch.empty(3, dtype=torch.int32, device=dev)
    for i in range(2):
        B.calibrate_async(xs[i % nset], workspace=ws, perm=perm, split=split, stream=stream)
    torch.cuda.synchronize()
    # its launches captured as a graph of `reps` calls (no host time between them)
    ms = launch_stats(stream, lambda i, s: B.calibrate_async(xs[i % nset], workspace=ws, perm=perm, split=split,
                                                             stream=s), reps, mean_only=True)
    nbytes = rows * w.K * 2 + w.K * 4 + 12
    gbps = nbytes / (ms * 1e-3) / 1e9
    return {"kernel": "offline calibration (mm_calibrate, 4 launches)", "rows": rows, "K": w.K, "ms": round(ms, 5),
            "achieved": round(gbps, 1), "peak": PEAK_HBM, "unit": "GB/s", "frac": round(gbps / PEAK_HBM, 4),
            "bytes_per_call": nbytes, "split": split.cpu().tolist()}


class Operands:
    """One workload's device buffers: bf16 activations, their packed
    quantised form, the packed (offline-quantised) weight and the bf16
    output, in several sets rotated so that what each kernel touches over a
    rotation (the quantiser: activations and their codes; the GEMM: codes,
    weight and output) exceeds min_set_mb, well past the 256 MB Infinity
    Cache: every launch reads its inputs from HBM."""

    def __init__(self, B, w, dev, stream, min_set_mb: float):
        import torch

        self.B, self.w, self.stream = B, w, stream
        xb, wb, perm_np = w.x_bits(), w.w_bits(), w.perm()
        self.perm = torch.from_numpy(perm_np).to(dev)
        x0, w0 = to_dev_bf16(xb, dev), to_dev_bf16(wb, dev)
        del xb, wb
        p4, p6, p8 = w.split
        row = p4 // 2 + 3 * p6 // 4 + p8 + w.K // 32
        quant_set = w.M * w.K * 2 + w.M * row
        gemm_set = w.M * row + w.N * row + w.M * w.N * 2
        # (a decode step's activation is a few KB, read from cache whatever
        # the rotation: there the GEMM's weight stream sets the count)
        touched = min(quant_set, gemm_set) if w.M > DIRECT_MAX_M else gemm_set
        self.nbuf = n = max(1, int(np.ceil(min_set_mb * 1e6 / touched)))
        self.X = [x0] + [x0.clone() for _ in range(n - 1)]
        self.XQ = [B.MXTensor.empty(w.M, w.K, w.split, device=dev) for _ in range(n)]
        self.WQ = [B.MXTensor.empty(w.N, w.K, w.split, device=dev) for _ in range(n)]
        self.Y = [torch.empty((w.M, w.N), dtype=torch.bfloat16, device=dev) for _ in range(n)]
        # offline weight quantisation (once per weight), timed on its own
        self.wq_ms = launch_stats(stream, lambda i, s: B.quantize_weight(w0, self.perm, w.split, out=self.WQ[i],
                                                                         stream=s), n, mean_only=True)
        for k in range(n):
            B.quantize_act(self.X[k], self.perm, w.split, out=self.XQ[k], stream=stream)
        torch.cuda.synchronize()

    def quant(self, i, stream=None):
        k = i % self.nbuf
        self.B.quantize_act(self.X[k], self.perm, self.w.split, out=self.XQ[k], stream=stream or self.stream)

    def gemm(self, i, stream=None):
        k = i % self.nbuf
        self.B.gemm(self.XQ[k], self.WQ[k], y=self.Y[k], stream=stream or self.stream)

    def step(self, i, stream=None):
        self.quant(i, stream)
        self.gemm(i, stream)


def capture_steps(ops, n: int, stream):
    """A HIP graph of steps 0 .. n-1 (the launches only; the Python and
    ctypes cost of issuing 2 n kernels one by one is paid once, at capture)."""
    return graph_of(ops.step, n, stream)


def to_dev_bf16(bits, dev):
    import torch

    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)


def graph_of(fn, n: int, stream):
    """A HIP graph of fn(0, s) .. fn(n-1, s), s the capture stream (the
    launches only: no host time between them when it is replayed)."""
    import torch

    side = torch.cuda.Stream()
    side.wait_stream(stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        cs = torch.cuda.current_stream()
        for i in range(n):
            fn(i, cs)
    torch.cuda.synchronize()
    return graph


def replay_ms(graph, stream, reps: int) -> list:
    """Durations of `reps` replays of a graph, from HIP events recorded on
    the stream it is replayed on."""
    import torch

    out = []
    with torch.cuda.stream(stream):
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            graph.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            out.append(e0.elapsed_time(e1))
    return out


def launch_stats(stream, fn, n: int, mean_only: bool = False, reps: int = 5):
    """Launch durations of fn(i, s), i = 0..n-1, s the stream to launch on:
    the n launches are captured as one HIP graph, so host issue time (ctypes,
    Python) never leaves the GPU idle between them, and the graph is
    replayed `reps` times after one untimed replay.  mean: all replays'
    time over reps * n launches; median: the median of the replays' per-launch
    means.  Returns (mean ms, median ms), or the mean alone."""
    graph = graph_of(fn, n, stream)
    replay_ms(graph, stream, 1)
    t = replay_ms(graph, stream, reps)
    del graph
    mean = sum(t) / (reps * n)
    if mean_only:
        return mean
    return mean, float(np.median(t)) / n


def norm_stats(B, W, ops, dev, stream, n: int, quant_ms: float) -> dict:
    """The quantiser with the layer's RMSNorm fused in front (weight ~ 1 +
    N(0, 0.25^2), eps 1e-5), against the unfused pair it replaces: torch's
    bf16 RMSNorm kernel (reads and writes the activation) then the plain
    quantiser."""
    import torch

    w = ops.w
    g_np = (1.0 + 0.25 * np.random.default_rng([w.seed, 9]).standard_normal(w.K)).astype(np.float32)
    gamma = to_dev_bf16(W.f32_to_bf16_bits(g_np), dev)
    fused_ms, fused_med = launch_stats(
        stream, lambda i, s: B.rmsnorm_quantize_act(ops.X[i % ops.nbuf], gamma, 1e-5, ops.perm, w.split,
                                                    out=ops.XQ[i % ops.nbuf], stream=s), n)
    # torch's norm is timed as a captured graph of 20 calls (its Python
    # dispatch per call is slower than the kernel itself)
    reps = 20
    xs = [ops.X[i % ops.nbuf] for i in range(reps)]
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        for x in xs[:3]:
            torch.nn.functional.rms_norm(x, (w.K,), weight=gamma, eps=1e-5)
    stream.wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        outs = [torch.nn.functional.rms_norm(x, (w.K,), weight=gamma, eps=1e-5) for x in xs]
    norm_ms = float(np.mean(replay_ms(graph, stream, max(3, n // reps)))) / reps
    del graph, outs
    qbytes = quant_bytes(w.M, w.K, w.split) + 2 * w.K
    return {"kernel": "RMSNorm fused with reorder-and-quantize", "ms": round(fused_ms, 5),
            "median_ms": round(fused_med, 5), "achieved": round(qbytes / (fused_ms * 1e-3) / 1e9, 1),
            "peak": PEAK_HBM, "unit": "GB/s", "frac": round(qbytes / (fused_ms * 1e-3) / 1e9 / PEAK_HBM, 4),
            "vs_plain_quantizer": round(fused_ms / quant_ms, 3),
            "unfused_pair_ms": round(norm_ms + quant_ms, 5), "torch_rms_norm_ms": round(norm_ms, 5)}


def gemm_roofline(w, mean_ms: float, median_ms: float) -> dict:
    """The GEMM against its roofline: the bit mix's MFMA peak for prefill
    shapes, HBM for the decode kernel (M <= 64)."""
    flops = 2.0 * w.M * w.N * w.K
    if w.M > DIRECT_MAX_M:
        ach = flops / (mean_ms * 1e-3) / 1e12
        peak = mix_peak_tflops(w.split)
        r = {"bound": "mfma", "kernel": "mixed MX GEMM", "achieved": round(ach, 2), "peak": round(peak, 1),
             "unit": "TFLOP/s", "frac": round(ach / peak, 4),
             "median_frac": round(flops / (median_ms * 1e-3) / 1e12 / peak, 4),
             "mfma_util": measured_mfma_util(w.name)}
    else:
        nbytes = gemm_bytes(w.M, w.N, w.K, w.split)
        ach = nbytes / (mean_ms * 1e-3) / 1e9
        r = {"bound": "hbm", "kernel": "mixed MX GEMM (decode)", "achieved": round(ach, 1), "peak": PEAK_HBM,
             "unit": "GB/s", "frac": round(ach / PEAK_HBM, 4),
             "median_frac": round(nbytes / (median_ms * 1e-3) / 1e9 / PEAK_HBM, 4)}
    r.update({"traffic": measured_traffic(w.name), "ms": round(mean_ms, 5), "median_ms": round(median_ms, 5),
              "source_hash": gemm_source_hash("direct" if w.M <= DIRECT_MAX_M else "tiled")})
    return r


def quant_roofline(w, mean_ms: float, median_ms: float) -> dict:
    qbytes = quant_bytes(w.M, w.K, w.split)
    gbps = qbytes / (mean_ms * 1e-3) / 1e9
    return {"kernel": "reorder-and-quantize (activation)", "ms": round(mean_ms, 5), "median_ms": round(median_ms, 5),
            "achieved": round(gbps, 1), "peak": PEAK_HBM, "unit": "GB/s", "frac": round(gbps / PEAK_HBM, 4),
            "bytes_per_launch": qbytes}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama8b_attn_2048x4096x4096")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-qkv", action="store_true",
                    help="skip the stacked-vs-separate Q/K/V GEMM comparison (attention shape)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the per-configuration table of the other prefill shapes")
    ap.add_argument("--min-working-set-mb", type=float, default=768.0)
    ap.add_argument("--calibration-rows", type=int, default=32768,
                    help="calibration tokens for the offline mm_calibrate timing (0 skips it)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE {world})", file=sys.stderr)
        return 2
    n_time = max(args.steps, 50)  # per-kernel statistics over at least 50 launches

    import torch

    from paper_2508_02343_amd import binding as B
    from paper_2508_02343_amd import workloads as W

    w = W.BY_NAME[args.workload]
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    # a plain device copy of known size: under rocprofv3 --pmc its FETCH_SIZE /
    # WRITE_SIZE give the scale factor for the GEMM's counters
    calib = torch.empty(CALIB_BYTES, dtype=torch.uint8, device=dev)
    calib_dst = torch.empty_like(calib)
    calib_dst.copy_(calib)
    del calib, calib_dst

    ops = Operands(B, w, dev, stream, args.min_working_set_mb)
    for i in range(args.warmup):
        ops.step(i)
    torch.cuda.synchronize()
    # the same K steps issued one by one (host launch cost included) ...
    t0 = time.perf_counter()
    for i in range(args.steps):
        ops.step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    eager_ms = (t1 - t0) * 1e3 / args.steps
    ref_y = [y.clone() for y in ops.Y]
    # ... and as one replay of a captured graph of exactly K steps, the timed
    # figure; every replay's outputs must equal the eager ones bit for bit
    graph = capture_steps(ops, args.steps, stream)
    graph.replay()
    torch.cuda.synchronize()
    graph_ok = all(torch.equal(a, b) for a, b in zip(ops.Y, ref_y))
    t0 = time.perf_counter()
    graph.replay()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    graph_ok = graph_ok and all(torch.equal(a, b) for a, b in zip(ops.Y, ref_y))
    if not graph_ok:
        raise RuntimeError("graph replay of the steps differs from their eager launches")
    del graph, ref_y

    # each kernel alone, back to back over the same rotated buffers
    quant_ms, quant_med = launch_stats(stream, ops.quant, n_time)
    gemm_ms, gemm_med = launch_stats(stream, ops.gemm, n_time)
    # the same quantiser with the layer's RMSNorm fused in front
    norm = norm_stats(B, W, ops, dev, stream, n_time, quant_ms)

    qkv = None
    if w.name == "llama8b_attn_2048x4096x4096" and not args.no_qkv:
        # Q, K and V projections of Llama-3-8B (4096 + 1024 + 1024 outputs) on one
        # quantised activation: the weights stacked along N in one GEMM, against
        # three GEMMs (weights resident: the same for both)
        rng = np.random.default_rng([w.seed, 5])
        parts = (4096, 1024, 1024)
        wl = [W.f32_to_bf16_bits((rng.standard_normal((n, w.K)) * 0.02).astype(np.float32)) for n in parts]
        wst = B.quantize_weight(to_dev_bf16(np.concatenate(wl), dev), ops.perm, w.split, stream=stream)
        wsep = [B.quantize_weight(to_dev_bf16(x, dev), ops.perm, w.split, stream=stream) for x in wl]
        yst = torch.empty((w.M, sum(parts)), dtype=torch.bfloat16, device=dev)
        ysep = [torch.empty((w.M, n), dtype=torch.bfloat16, device=dev) for n in parts]
        st_ms = launch_stats(stream, lambda i, s: B.gemm(ops.XQ[i % ops.nbuf], wst, y=yst, stream=s), n_time,
                             mean_only=True)

        def three(i, s):
            for k in range(3):
                B.gemm(ops.XQ[i % ops.nbuf], wsep[k], y=ysep[k], stream=s)

        sep_ms = launch_stats(stream, three, n_time, mean_only=True)
        qflops = 2.0 * w.M * w.K * sum(parts)
        qkv = {"N": list(parts), "stacked_ms": round(st_ms, 5), "separate_ms": round(sep_ms, 5),
               "stacked_TFLOPs": round(qflops / (st_ms * 1e-3) / 1e12, 1),
               "separate_TFLOPs": round(qflops / (sep_ms * 1e-3) / 1e12, 1)}
        del wst, wsep, yst, ysep

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    flops = 2.0 * w.M * w.N * w.K
    value = flops / (ms_per_step * 1e-3) / 1e12
    quant = quant_roofline(w, quant_ms, quant_med)
    wq_gbps = quant_bytes(w.N, w.K, w.split) / (ops.wq_ms * 1e-3) / 1e9

    def config_row(wl, q_mean, q_med, g_mean, g_med, nrm):
        g = gemm_roofline(wl, g_mean, g_med)
        q = quant_roofline(wl, q_mean, q_med)
        return {"workload": wl.name, "M": wl.M, "K": wl.K, "N": wl.N, "split": list(wl.split),
                "gemm": {k: g[k] for k in ("ms", "median_ms", "achieved", "peak", "unit", "frac", "median_frac",
                                           "mfma_util", "traffic") if k in g},
                "quantizer": {k: q[k] for k in ("ms", "median_ms", "achieved", "unit", "frac")},
                "quant_to_gemm_time": round(q_med / g_med, 4),
                "quant_share_of_kernel_time": round(q_med / (q_med + g_med), 4),
                "rmsnorm_quantizer": {k: nrm[k] for k in ("ms", "frac", "vs_plain_quantizer", "unfused_pair_ms")}}

    sweep = None
    if not args.no_sweep and w.M > DIRECT_MAX_M:
        # the other prefill shapes, each kernel timed the same way
        sweep = []
        for wl in W.PREFILL:
            if wl.name == w.name:
                sweep.append(config_row(wl, quant_ms, quant_med, gemm_ms, gemm_med, norm))
                continue
            o2 = Operands(B, wl, dev, stream, args.min_working_set_mb)
            for i in range(args.warmup):
                o2.step(i)
            q2 = launch_stats(stream, o2.quant, n_time)
            g2 = launch_stats(stream, o2.gemm, n_time)
            sweep.append(config_row(wl, *q2, *g2, norm_stats(B, W, o2, dev, stream, n_time, q2[0])))
            del o2
            torch.cuda.empty_cache()

    out = {
        "metric": "mixed MX GEMM TFLOPS (+quantizer GB/s) on Llama-8B/Qwen-32B layer shapes",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "mxfp4/mxfp6/mxfp8 (e2m1/e3m2/e4m3), fp32 accumulate, bf16 in/out",
        "data": "synthetic",
        "config": {"workload": w.name, "M": w.M, "K": w.K, "N": w.N, "split": list(w.split),
                   "x_dist": w.x_dist, "rotated_buffer_sets": ops.nbuf},
        "roofline": gemm_roofline(w, gemm_ms, gemm_med),
        "quantizer": quant,
        "rmsnorm_quantizer": norm,
        "gemm_ms": round(gemm_ms, 5),
        "quant_share_of_kernel_time": round(quant_med / (quant_med + gemm_med), 4),
        "prefill_configs": sweep,
        "shared_activation_qkv": qkv,
        "weight_quantize": {"ms": round(ops.wq_ms, 5), "GB/s": round(wq_gbps, 1)},
        "timing": f"ms_per_step: one replay of a HIP graph of the {args.steps} steps (outputs checked equal to "
                  f"their eager launches), wall clock between synchronizations; per-kernel ms: a HIP graph of "
                  f"{n_time} launches replayed 5 times (HIP events around each replay), mean over all launches; "
                  f"median_ms: median of the replays' per-launch means",
        "ms_per_step_eager": round(eager_ms, 5),
    }
    if args.calibration_rows > 0:
        out["calibration"] = measure_calibration(B, W, w, stream, dev, args.calibration_rows,
                                                 args.min_working_set_mb)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
