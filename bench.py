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


GEMM_SOURCES = ("gemm_tiled.hip", "gemm_direct.hip", "gemm_common.hpp", "mx_device.hpp", "kernels.hpp", "api.cpp")
CALIB_BYTES = 256 << 20  # plain copy used to calibrate the FETCH_SIZE / WRITE_SIZE counters


def gemm_source_hash() -> str:
    import hashlib

    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2508_02343_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per GEMM launch from the committed rocprofv3 counter summary,
    or None when the summary is missing or was taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", "gemm_traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    entry = rec.get(workload)
    if not entry or entry.get("source_hash") != gemm_source_hash():
        return None
    return entry.get("hbm_bytes_per_launch")


def cpu_baseline(w, seconds: float) -> dict:
    """The oracle (float64 numpy) on a bounded sample: quantise a slice of the
    activation rows and multiply it with the (pre-quantised) weight."""
    from oracle import mx_oracle as O

    try:
        from threadpoolctl import threadpool_info

        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    rows = min(w.M, 256)
    xb, wb, perm = w.x_bits(rows), w.w_bits(), w.perm()
    wq = O.quantize_mixed(wb, perm, w.split)
    n_iter, t0 = 0, time.perf_counter()
    while True:
        a = O.quantize_mixed(xb, perm, w.split)
        O.gemm_mixed(a, wq)
        n_iter += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    tflops = 2.0 * rows * w.N * w.K * n_iter / el / 1e12
    return {"value": tflops, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{rows} of {w.M} activation rows x full weight [{w.N},{w.K}], quantise + GEMM, "
                      f"{n_iter} iterations in {el:.1f} s"}


def measure_calibration(B, W, w, stream, dev, rows: int, min_set_mb: float, reps: int = 10) -> dict:
    """mm_calibrate over `rows` calibration tokens of the layer's width K
    (offline, not part of the step): whole-call time with HIP events on the
    launch stream, and HBM bandwidth over the bytes it must move (X read once,
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
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(reps):
        B.calibrate_async(xs[i % nset], workspace=ws, perm=perm, split=split, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = rows * w.K * 2 + w.K * 4 + 12
    gbps = nbytes / (ms * 1e-3) / 1e9
    return {"kernel": "offline calibration (mm_calibrate, 4 launches)", "rows": rows, "K": w.K, "ms": round(ms, 5),
            "achieved": round(gbps, 1), "peak": PEAK_HBM, "unit": "GB/s", "frac": round(gbps / PEAK_HBM, 4),
            "bytes_per_call": nbytes, "split": split.cpu().tolist()}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama8b_attn_2048x4096x4096")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--min-working-set-mb", type=float, default=768.0)
    ap.add_argument("--calibration-rows", type=int, default=32768,
                    help="calibration tokens for the offline mm_calibrate timing (0 skips it)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE {world})", file=sys.stderr)
        return 2

    import torch

    from paper_2508_02343_amd import binding as B
    from paper_2508_02343_amd import workloads as W

    w = W.BY_NAME[args.workload]
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    xb, wb, perm_np = w.x_bits(), w.w_bits(), w.perm()
    to_bf16 = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
    x0, w0 = to_bf16(xb), to_bf16(wb)
    perm = torch.from_numpy(perm_np).to(dev)

    p4, p6, p8 = w.split
    set_bytes = (w.M * w.K * 2 + w.M * (p4 // 2 + 3 * p6 // 4 + p8 + w.K // 32)
                 + w.N * (p4 // 2 + 3 * p6 // 4 + p8 + w.K // 32) + w.M * w.N * 2)
    nbuf = max(1, int(np.ceil(args.min_working_set_mb * 1e6 / set_bytes)))
    X = [x0.clone() for _ in range(nbuf)]
    XQ = [B.MXTensor.empty(w.M, w.K, w.split, device=dev) for _ in range(nbuf)]
    WQ = [B.MXTensor.empty(w.N, w.K, w.split, device=dev) for _ in range(nbuf)]
    Y = [torch.empty((w.M, w.N), dtype=torch.bfloat16, device=dev) for _ in range(nbuf)]
    del x0

    stream = torch.cuda.current_stream()
    # a plain device copy of known size: under rocprofv3 --pmc its FETCH_SIZE /
    # WRITE_SIZE give the scale factor for the GEMM's counters
    calib = torch.empty(CALIB_BYTES, dtype=torch.uint8, device=dev)
    calib_dst = torch.empty_like(calib)
    calib_dst.copy_(calib)
    del calib, calib_dst
    # offline weight quantisation (once per weight), timed on its own
    ew0, ew1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ew0.record(stream)
    for k in range(nbuf):
        B.quantize_weight(w0, perm, w.split, out=WQ[k], stream=stream)
    ew1.record(stream)
    torch.cuda.synchronize()
    wq_ms = ew0.elapsed_time(ew1) / nbuf
    del w0

    def step(i):
        k = i % nbuf
        B.quantize_act(X[k], perm, w.split, out=XQ[k], stream=stream)
        B.gemm(XQ[k], WQ[k], y=Y[k], stream=stream)

    def timed(fn, n):
        """Average duration of n back-to-back launches, HIP events on the
        stream the kernels run on."""
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(n):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    # per-kernel average launch durations: each kernel alone, back to back over
    # the same rotated buffers (no event between launches)
    quant_ms = timed(lambda i: B.quantize_act(X[i % nbuf], perm, w.split, out=XQ[i % nbuf], stream=stream),
                     args.steps)
    gemm_ms = timed(lambda i: B.gemm(XQ[i % nbuf], WQ[i % nbuf], y=Y[i % nbuf], stream=stream), args.steps)
    # the same quantiser with the layer's RMSNorm fused in front (weight ~ 1 + N(0, 0.25^2), eps 1e-5)
    g_np = (1.0 + 0.25 * np.random.default_rng([w.seed, 9]).standard_normal(w.K)).astype(np.float32)
    gamma = to_bf16(W.f32_to_bf16_bits(g_np))
    norm_ms = timed(lambda i: B.rmsnorm_quantize_act(X[i % nbuf], gamma, 1e-5, perm, w.split, out=XQ[i % nbuf],
                                                     stream=stream), args.steps)

    qkv = None
    if w.name == "llama8b_attn_2048x4096x4096":
        # Q, K and V projections of Llama-3-8B (4096 + 1024 + 1024 outputs) on one
        # quantised activation: the weights stacked along N in one GEMM, against
        # three GEMMs (weights resident: the same for both)
        rng = np.random.default_rng([w.seed, 5])
        parts = (4096, 1024, 1024)
        wl = [W.f32_to_bf16_bits((rng.standard_normal((n, w.K)) * 0.02).astype(np.float32)) for n in parts]
        wst = B.quantize_weight(to_bf16(np.concatenate(wl)), perm, w.split, stream=stream)
        wsep = [B.quantize_weight(to_bf16(x), perm, w.split, stream=stream) for x in wl]
        yst = torch.empty((w.M, sum(parts)), dtype=torch.bfloat16, device=dev)
        ysep = [torch.empty((w.M, n), dtype=torch.bfloat16, device=dev) for n in parts]
        st_ms = timed(lambda i: B.gemm(XQ[i % nbuf], wst, y=yst, stream=stream), args.steps)

        def three(i):
            for k in range(3):
                B.gemm(XQ[i % nbuf], wsep[k], y=ysep[k], stream=stream)

        sep_ms = timed(three, args.steps)
        qflops = 2.0 * w.M * w.K * sum(parts)
        qkv = {"N": list(parts), "stacked_ms": round(st_ms, 5), "separate_ms": round(sep_ms, 5),
               "stacked_TFLOPs": round(qflops / (st_ms * 1e-3) / 1e12, 1),
               "separate_TFLOPs": round(qflops / (sep_ms * 1e-3) / 1e12, 1)}

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    flops = 2.0 * w.M * w.N * w.K
    value = flops / (ms_per_step * 1e-3) / 1e12
    gemm_tflops = flops / (gemm_ms * 1e-3) / 1e12
    peak = mix_peak_tflops(w.split)
    qbytes = quant_bytes(w.M, w.K, w.split)
    quant_gbps = qbytes / (quant_ms * 1e-3) / 1e9
    wq_gbps = quant_bytes(w.N, w.K, w.split) / (wq_ms * 1e-3) / 1e9

    if w.M > DIRECT_MAX_M:  # prefill: the block-scaled MFMA peak for the bit mix
        roofline = {"bound": "mfma", "kernel": "mixed MX GEMM", "achieved": round(gemm_tflops, 2),
                    "peak": round(peak, 1), "unit": "TFLOP/s", "frac": round(gemm_tflops / peak, 4),
                    "traffic": measured_traffic(w.name), "source_hash": gemm_source_hash()}
    else:  # decode: HBM bandwidth over the packed weight (and the small A / Y terms)
        gbps = gemm_bytes(w.M, w.N, w.K, w.split) / (gemm_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "kernel": "mixed MX GEMM (decode)", "achieved": round(gbps, 1),
                    "peak": PEAK_HBM, "unit": "GB/s", "frac": round(gbps / PEAK_HBM, 4),
                    "traffic": measured_traffic(w.name), "source_hash": gemm_source_hash()}
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
                   "x_dist": w.x_dist, "rotated_buffer_sets": nbuf},
        "roofline": roofline,
        "quantizer": {"kernel": "reorder-and-quantize (activation)", "ms": round(quant_ms, 5),
                      "achieved": round(quant_gbps, 1), "peak": PEAK_HBM, "unit": "GB/s",
                      "frac": round(quant_gbps / PEAK_HBM, 4), "bytes_per_launch": qbytes},
        "rmsnorm_quantizer": {"kernel": "RMSNorm fused with reorder-and-quantize", "ms": round(norm_ms, 5),
                              "achieved": round((qbytes + 2 * w.K) / (norm_ms * 1e-3) / 1e9, 1), "peak": PEAK_HBM,
                              "unit": "GB/s", "frac": round((qbytes + 2 * w.K) / (norm_ms * 1e-3) / 1e9 / PEAK_HBM, 4),
                              "vs_plain_quantizer": round(norm_ms / quant_ms, 3)},
        "gemm_ms": round(gemm_ms, 5),
        "shared_activation_qkv": qkv,
        "quant_share_of_kernel_time": round(quant_ms / (quant_ms + gemm_ms), 4),
        "weight_quantize": {"ms": round(wq_ms, 5), "GB/s": round(wq_gbps, 1)},
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
