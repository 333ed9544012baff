"""Build libmicromix.so (gfx950) in place with hipcc.

Usage: python -m paper_2508_02343_amd.build_lib   (or call build()).

Each source is compiled to an object of its own (in parallel), then linked.
The prefill GEMM is compiled at -O2: at -O3 the extra code motion leaves the
register allocator moving its 256 accumulators between the K loops of the
three groups and spilling to scratch; at -O2 each loop keeps them in place.
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libmicromix.so")
SOURCES = ["api.cpp", "quantize.hip", "gemm_direct.hip", "gemm_tiled.hip", "calibrate.hip"]
OPT = {"gemm_tiled.hip": "-O2"}  # default -O3
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Werror",
    "-Wno-unused-function",
    # never let the compiler form packed fp32 ops (v_pk_*_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _run(cmd: list[str], verbose: bool) -> None:
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


def build(verbose: bool = False) -> str:
    inc = os.path.join(HERE, "..", "include")
    with tempfile.TemporaryDirectory(prefix="mm_build_") as tmpd:
        objs = [os.path.join(tmpd, s + ".o") for s in SOURCES]
        cmds = [[HIPCC, *FLAGS, OPT.get(s, "-O3"), "-I", inc, "-c", "-o", o, os.path.join(CSRC, s)]
                for s, o in zip(SOURCES, objs)]
        with ThreadPoolExecutor(max_workers=len(cmds)) as ex:
            for f in [ex.submit(_run, c, verbose) for c in cmds]:
                f.result()
        tmp = LIB + ".tmp"
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
