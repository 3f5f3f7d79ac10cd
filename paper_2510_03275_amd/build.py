"""Builds libsdq.so (HIP kernels + C ABI) in-tree for gfx950 with hipcc.

    python paper_2510_03275_amd/build.py        # or __graft_entry__.build()

Every call recompiles all sources.  Device code is built with packed-fp32
instructions disabled and with floating-point contraction off in the encoder
(its sources also say so with a pragma), and without fast-math; the fp64 GEMM
and the prefill expansion keep their matrix-core accumulators in VGPRs.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libsdq.so")
ARCH = os.environ.get("SDQ_OFFLOAD_ARCH", "gfx950")

SOURCES = ["sdq_api.cpp", "encoder.hip", "linear_decode.hip", "linear_prefill.hip", "expand_prefill.hip",
           "moments.hip", "compensation.hip", "linear_noalloc.hip"]

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fno-gpu-flush-denormals-to-zero", "-Wall", "-Wno-unused-function",
]
PER_FILE = {
    "encoder.hip": ["-ffp-contract=off"],
    "sdq_api.cpp": ["-ffp-contract=off"],
    # fp64 GEMM: keep the MFMA accumulators in VGPRs (left to its heuristics the
    # compiler carries them across the k loop in VGPRs but runs the MFMAs on
    # AGPR copies, 64 moves and a pipeline drain per k step).
    "compensation.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "expand_prefill.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    # the 2-16-row contractions: without it the integer accumulators rotate
    # through AGPR copies, 40 moves per 64-code chunk at 5-8 rows
    "linear_decode.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src + ".o")
    lang = ["-x", "hip"]
    cmd = [_hipcc(), *lang, *COMMON, *PER_FILE.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


SYNTH_SRCS = [os.path.join(os.path.dirname(HERE), "synth", "csrc", f) for f in ("synth_gen.hip", "read_probe.hip")]
SYNTH_LIB = os.path.join(os.path.dirname(HERE), "synth", "libsdqsynth.so")


def _build_synth() -> str:
    """The input generator's device twin and the bench's streaming-read probe: a
    library of its own (no method code)."""
    tmp = SYNTH_LIB + ".tmp"
    cmd = [_hipcc(), "-x", "hip", *COMMON, "-shared", *SYNTH_SRCS, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"synth build failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, SYNTH_LIB)
    return SYNTH_LIB


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES) + 1, 8)) as ex:
        synth_job = ex.submit(_build_synth)
        objs = list(ex.map(_compile, SOURCES))
        synth_job.result()
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
