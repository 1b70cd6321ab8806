"""Build ``libgift.so`` (HIP, gfx950) in-tree with hipcc.

``python -m paper_2607_07494_amd.build`` compiles every source under
``csrc/`` for gfx950 and links the shared library next to this file.  The
flags matter for the codec's exactness: ``-ffp-contract=off`` keeps the
scale multiply, the dequantize multiply-add chain and the residual update as
separate IEEE operations, and packed FP32 instructions are disabled.
"""

from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libgift.so")
ARCH = "gfx950"

CALIB_SOURCE = "calib.hip"
CALIB_LIB = os.path.join(PKG, "libgift_calib.so")

SOURCES = ["gift_api.cpp", "k_tile.hip", "k_reduce.hip", "k_factor.hip", "k_syrk.hip", "k_update.hip", "k_stream.hip",
           "k_lowrank.hip", "k_chol.hip", "k_mx.hip"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libgift.so)")


def compile_flags():
    return [
        f"--offload-arch={ARCH}",
        "-O3",
        "-std=c++17",
        "-fPIC",
        "-ffp-contract=off",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
        "-I", os.path.join(ROOT, "include"),
        "-I", CSRC,
    ]


# Sources whose compiler resource report is kept (kernel-resource-usage
# remarks), for the spill check below.
RESOURCE_REPORT = {"k_lowrank.hip"}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [hipcc(), "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj] + compile_flags()
    if src in RESOURCE_REPORT:
        cmd.append("-Rpass-analysis=kernel-resource-usage")
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}\n{res.stderr}")
    if src in RESOURCE_REPORT:
        with open(obj + ".resources.txt", "w") as fh:
            fh.write(res.stderr)
    return obj


def two_wave_scratch():
    """{kernel: scratch bytes per lane} of the two-waves-per-SIMD update
    variants (lr_update_kernel_o2, lr_sweep_kernel), from the compiler's
    resource report."""
    import re
    path = os.path.join(BUILD, "k_lowrank.hip.o.resources.txt")
    out, name = {}, None
    for line in open(path):
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name and ("lr_update_kernel_o2" in name or "lr_sweep_kernel" in name):
            out[name] = int(m.group(1))
    return out


def check_two_wave_spills(verbose: bool = False):
    """The two-wave update variants exist to hold two waves per SIMD with no
    scratch; a toolchain or code change that makes one spill would slow the
    rank-128 encode without changing its results, so the build fails."""
    scratch = two_wave_scratch()
    if not scratch:
        raise RuntimeError("no resource report for the two-wave update kernels")
    bad = {k: v for k, v in scratch.items() if v > 0}
    if bad:
        raise RuntimeError("two-wave update kernels spill to scratch: " +
                           ", ".join(f"{k} ({v} B/lane)" for k, v in sorted(bad.items())))
    if verbose:
        print(f"{len(scratch)} two-wave update kernels, no scratch")


def _link(objs, out):
    tmp = out + ".tmp"
    cmd = [hipcc(), "-shared", f"--offload-arch={ARCH}", "-fPIC", "-o", tmp] + objs
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    """Compile all sources and link ``libgift.so`` (and the benchmark's peak
    calibration kernels, ``libgift_calib.so``); returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    workers = min(len(SOURCES) + 1, max(1, (os.cpu_count() or 2) // 2), 8)
    with concurrent.futures.ThreadPoolExecutor(workers) as pool:
        objs = list(pool.map(_compile, SOURCES + [CALIB_SOURCE]))
    _link(objs[:-1], LIB)
    _link(objs[-1:], CALIB_LIB)
    check_two_wave_spills(verbose)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
