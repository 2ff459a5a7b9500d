"""Build libks.so (HIP kernels for gfx950 + the C-ABI host code) in-tree.

Run as ``python -m paper_2606_28565_amd.build``.  hipcc cross-compiles for
gfx950 without a GPU present."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libks.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Device code: gfx950 only; packed-fp32 VALU forms are kept out of the
# generated code on purpose.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                # MFMA results stay in ordinary VGPRs: the epilogues are VALU
                # work, and accumulator-register round trips cost a VALU op each
                "-mllvm", "-amdgpu-mfma-vgpr-form",
                "-Wall", "-Wno-unused-function"]
# host-only translation units: plain C++ against the HIP runtime API
HOST_FLAGS = ["-x", "c++", "-O2", "-std=c++17", "-fPIC", "-Wall",
              "-I", os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(HIPCC))), "include")]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{err}")
    if err.strip():
        print(err, file=sys.stderr)


def build(verbose: bool = False) -> str:
    objs = []
    tmp = os.path.join(PKG, "_obj")
    os.makedirs(tmp, exist_ok=True)
    kern = os.path.join(tmp, "ks_kernels.o")
    api = os.path.join(tmp, "ks_api.o")
    common = ["-I", INCLUDE, "-I", CSRC]
    expand = os.path.join(tmp, "ks_expand.o")
    _run([HIPCC, *DEVICE_FLAGS, *common, "-c", os.path.join(CSRC, "ks_kernels.hip"), "-o", kern])
    _run([HIPCC, *DEVICE_FLAGS, *common, "-c", os.path.join(CSRC, "ks_expand.hip"), "-o", expand])
    static = os.path.join(tmp, "ks_static.o")
    _run([HIPCC, *DEVICE_FLAGS, *common, "-c", os.path.join(CSRC, "ks_static.hip"), "-o", static])
    _run([HIPCC, *HOST_FLAGS, *common, "-D__HIP_PLATFORM_AMD__", "-c",
          os.path.join(CSRC, "ks_api.cpp"), "-o", api])
    simo = os.path.join(tmp, "ks_sim.o")
    _run([HIPCC, *HOST_FLAGS, *common, "-D__HIP_PLATFORM_AMD__", "-c",
          os.path.join(CSRC, "ks_sim.cpp"), "-o", simo])
    objs = [kern, expand, static, api, simo]
    tmp_lib = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp_lib])
    os.replace(tmp_lib, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
