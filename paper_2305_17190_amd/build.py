"""Build step for the HIP library libpam.so (gfx950 only).

    python -m paper_2305_17190_amd.build

compiles csrc/*.hip and csrc/*.cpp with hipcc into paper_2305_17190_amd/libpam.so.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libpam.so")

# Device code: gfx950 only; float32 denormals flushed (the GEMM relies on the
# accumulate treating denormal encodings as zero); no packed-fp32 VALU ops.
DEVICE_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fgpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the PAM library needs ROCm's hipcc")
    return path


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


def build(verbose: bool = False, extra_flags=()) -> str:
    tmp = f"{LIB}.{os.getpid()}.tmp"   # per process: concurrent builds never see a partial file
    cmd = [hipcc(), *DEVICE_FLAGS, *extra_flags, "-fPIC", "-shared", "-I", INCLUDE, "-I", CSRC,
           *sources(), "-o", tmp, "-lhsa-runtime64"]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed to build libpam.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
