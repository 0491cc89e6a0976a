"""Build the HIP library ``libforge.so`` (gfx950 only) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libforge.so")
SOURCES = [os.path.join(CSRC, f) for f in ("forge_kernels.hip", "forge_dx.hip", "forge_scratch.hip",
                                           "forge_api.cpp")]
HEADERS = [os.path.join(CSRC, "forge_internal.h"), os.path.join(CSRC, "forge_device.h"),
           os.path.join(INCLUDE, "forge.h")]

CEILING_SRC = os.path.join(CSRC, "hbm_ceiling.hip")
CEILING_BIN = os.path.join(HERE, "hbm_ceiling")   # measured HBM ceilings (bench context)

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-fvisibility=hidden",
    "-ffp-contract=off",                      # fused multiply-adds only where written
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def build(verbose: bool = False) -> str:
    """Compile every source into ``paper_2606_22932_amd/libforge.so`` (always rebuilds)."""
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *FLAGS, "-I", INCLUDE, "-I", CSRC, *SOURCES, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libforge.so")
    if verbose:
        sys.stderr.write(res.stderr)
    os.replace(tmp, LIB)
    build_ceiling(verbose)
    return LIB


def build_ceiling(verbose: bool = False) -> str:
    """Compile the stand-alone HBM ceiling probe ``paper_2606_22932_amd/hbm_ceiling``."""
    tmp = CEILING_BIN + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-Wall", CEILING_SRC, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building hbm_ceiling")
    if verbose:
        sys.stderr.write(res.stderr)
    os.replace(tmp, CEILING_BIN)
    return CEILING_BIN


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(f) > t for f in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose=True))
