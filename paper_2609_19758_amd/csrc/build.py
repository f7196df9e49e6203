"""Build libfpsketch.so (gfx950 HIP kernels + C-ABI host library) in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
OUT = os.path.join(PKG, "libfpsketch.so")
# Diagnostic build: the same kernels with the stream pass's per-work-group timeline recorded
# (bench.py --wg-timeline reads it).  The binding never loads it for the probe path.
OUT_TIMELINE = os.path.join(PKG, "libfpsketch_timeline.so")
SOURCES = ["fpsk_stream.hip", "fpsk_kernels.hip", "fpsk_host.hip"]

# gfx950 only; packed FP32 instructions disabled (hipcc forms them from plain float code).
# Matrix-core accumulators in ordinary VGPRs: with the compiler's default the loop-carried
# accumulators of the bucket-space product were copied between VGPRs and AGPRs on every k-step
# and the 64 x 64 product tile took 192 registers (2 waves per SIMD) instead of 98.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-mllvm", "-amdgpu-mfma-vgpr-form",
         "-Wall", "-Wno-unused-function", f"-I{os.path.join(ROOT, 'include')}"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False, timeline: bool = False) -> str:
    out = OUT_TIMELINE if timeline else OUT
    tmp = out + ".tmp"
    extra = ["-DFPSK_WG_TIMELINE"] if timeline else []
    cmd = [hipcc(), *FLAGS, *extra, "-o", tmp, *[os.path.join(HERE, s) for s in SOURCES]]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode}")
    if verbose and res.stderr.strip():
        sys.stderr.write(res.stderr)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True, timeline="--timeline" in sys.argv[1:]))
