"""Build libmalt.so (HIP, gfx950) in-tree with hipcc, and the matrix-core
calibration library libmalt_calib.so beside it.

Usage: python -m paper_2608_05088_amd.build [-v]
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "lib", "libmalt.so")
CALIB = os.path.join(PKG, "calib")
CALIB_LIB = os.path.join(PKG, "lib", "libmalt_calib.so")
SOURCES = ["malt_api.hip", "elementwise.hip", "ns_sym.hip", "ns_update.hip", "small_ns.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm toolchain required to build libmalt)")


def build_cmd(out: str = LIB) -> list:
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
            # Packed-fp32 VALU forms are disabled for all device code.
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
            "-I", os.path.join(ROOT, "include"), "-I", CSRC,
            *[os.path.join(CSRC, s) for s in SOURCES],
            "-o", out]


def calib_cmd(out: str = CALIB_LIB) -> list:
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", os.path.join(CALIB, "mfma_ceiling.hip"), "-o", out]


def _compile(cmd: list, lib: str, what: str, verbose: bool) -> None:
    tmp = cmd[-1]
    if verbose:
        print(" ".join(cmd), flush=True)
    proc = subprocess.run(cmd, cwd=os.path.dirname(lib), stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass does not know the packed-fp32 feature; that note is harmless.
    out = "\n".join(l for l in proc.stdout.splitlines() if "packed-fp32-ops" not in l)
    if proc.returncode != 0:
        raise RuntimeError(f"{what} build failed ({proc.returncode}):\n{out}")
    if verbose and out.strip():
        print(out)
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Compile every HIP source of the package into libmalt.so, and the
    matrix-core calibration into libmalt_calib.so (always rebuilds)."""
    os.makedirs(os.path.dirname(LIB), exist_ok=True)
    _compile(build_cmd(LIB + ".tmp"), LIB, "libmalt", verbose)
    _compile(calib_cmd(CALIB_LIB + ".tmp"), CALIB_LIB, "libmalt_calib", verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
