"""Builds libgdn_tailreplay.so (HIP, gfx950) in-tree.

``python -m paper_2608_30310_amd.build``.  Cross-compiles on a machine without
a GPU; the shared library lands next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libgdn_tailreplay.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)
SOURCES = ["gdn_plan.cpp", "gdn_gemm.cpp", "gdn_api.hip", "gdn_block.hip"]
ROCM_LIB = "/opt/rocm/lib"
ARCH = "gfx950"


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP toolchain is required")
    return path


def build(verbose: bool = False) -> str:
    tmp = LIB_PATH + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
           # packed fp32 instructions stay off on this target
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           # MFMA results in ordinary VGPRs: the scan feeds them to VALU work
           # every step, and accumulator-register copies would serialise it
           "-mllvm", "-amdgpu-mfma-vgpr-form",
           "-Wall", "-I", INCLUDE, "-I", CSRC, "-o", tmp]
    cmd += [os.path.join(CSRC, s) for s in SOURCES]
    # the layer block's projections run through hipBLASLt
    cmd += ["-L", ROCM_LIB, "-Wl,-rpath," + ROCM_LIB, "-lhipblaslt"]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = [l for l in (res.stdout + res.stderr).splitlines() if noise not in l]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
