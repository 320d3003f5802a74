"""Build libprq.so (and the test-only libprq_probe.so) in-tree for gfx950.

    python -m paper_2609_22106_amd.build          # or build() from Python

Device code: hipcc --offload-arch=gfx950 -O3, packed-FP32 instruction
selection disabled.  Host C++ (the offline prepare and the ABI layer): g++
with -ffp-contract=off so every float/double operation rounds as written.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libprq.so")
PROBE_LIB = os.path.join(PKG, "libprq_probe.so")

ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-mcode-object-version=5",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-munsafe-fp-atomics", "-Wall", "-Wno-unused-function",
]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-Wall",
              "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include"]

DEVICE_SOURCES = ["act_quant.hip", "pack.hip", "gemm_tile.hip", "gemm_stream.hip", "gemm_decode.hip",
                  "gemm_streamk.hip",
                  "evaluate.hip", "noalloc.hip"]
HOST_SOURCES = ["prepare.cpp", "abi.cpp"]
PROBE_SOURCES = ["probe.hip"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}")
    return r.stdout


def _compile_all(tmp, verbose):
    inc = [f"-I{INCLUDE}", f"-I{CSRC}"]
    objs = []
    for src in DEVICE_SOURCES:
        obj = os.path.join(tmp, src + ".o")
        _run([HIPCC, *HIP_FLAGS, *inc, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
        if verbose:
            print("built", src, flush=True)
    for src in HOST_SOURCES:
        obj = os.path.join(tmp, src + ".o")
        _run(["g++", *HOST_FLAGS, *inc, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
        if verbose:
            print("built", src, flush=True)
    return objs


def build(verbose=False):
    """Compile every HIP and host source and link the two shared libraries."""
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    with tempfile.TemporaryDirectory(prefix="prq_build_") as tmp:
        objs = _compile_all(tmp, verbose)
        out = os.path.join(tmp, "libprq.so")
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", out, *objs, "-lpthread"])
        shutil.move(out, LIB)
        # kernels for the tuning entry points (evaluate.hip and noalloc.hip call
        # into the host library and stay out)
        pobjs = [o for o in objs if o.endswith(".hip.o") and not o.endswith("evaluate.hip.o")
                 and not o.endswith("noalloc.hip.o")]
        for src in PROBE_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            _run([HIPCC, *HIP_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-c", os.path.join(CSRC, src),
                  "-o", obj])
            pobjs.append(obj)
        pout = os.path.join(tmp, "libprq_probe.so")
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", pout, *pobjs])
        shutil.move(pout, PROBE_LIB)
    if verbose:
        print("wrote", LIB, "and", PROBE_LIB, flush=True)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
