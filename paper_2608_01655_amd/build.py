"""Build the gfx950 planner library (libprefixplace.so) in-tree with hipcc."""

from __future__ import annotations

import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libprefixplace.so")
BUILD_DIR = os.path.join(PKG, "_build")

ARCH = "gfx950"
# Packed-FP32 selection is disabled for all device code (no packed f32 math
# is used here; this keeps the compiler from forming it).  No contraction of
# a * b + c into one rounding: the real-valued path rounds every product and
# sum as written.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-ffp-contract=off"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I", INCLUDE, "-I", CSRC]


def hipcc() -> str:
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found; the ROCm toolchain is required")
    return exe


def _run(cmd):
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" +
                           proc.stdout + proc.stderr)
    return proc


def build(verbose: bool = False) -> str:
    """Compile every HIP source for gfx950 and link the shared library."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    cc = hipcc()
    objs = []
    for src, device in (("pp_kernels.hip", True), ("pp_host.cpp", False)):
        obj = os.path.join(BUILD_DIR, src + ".o")
        cmd = [cc, f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS, "-c",
               os.path.join(CSRC, src), "-o", obj]
        if not device:
            cmd.insert(1, "-x")
            cmd.insert(2, "hip")
        p = _run(cmd)
        if verbose and (p.stdout or p.stderr):
            print(p.stdout + p.stderr)
        objs.append(obj)
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


def isa(kernel_src: str = "pp_kernels.hip") -> str:
    """gfx950 assembly of a source file (for inspection)."""
    out = os.path.join(BUILD_DIR, kernel_src + ".s")
    os.makedirs(BUILD_DIR, exist_ok=True)
    _run([hipcc(), f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS,
          "--cuda-device-only", "-S", os.path.join(CSRC, kernel_src), "-o", out])
    return out


if __name__ == "__main__":
    print(build(verbose=True))
