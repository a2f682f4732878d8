"""Build libwino.so in-tree for gfx950 with hipcc.

Usage: python -m paper_1903_01521_amd.build [--check]
"""
from __future__ import annotations

import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libwino.so")
SOURCES = [os.path.join(CSRC, "wino_kernels.hip"), os.path.join(CSRC, "wino_api.cpp")]
HEADERS = [os.path.join(CSRC, f) for f in ("wino_transforms.h", "wino_internal.h")] + [
    os.path.join(ROOT, "include", "wino.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 VALU ops are kept out of every kernel: plain fp32 FMA/add/mul only.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-I", os.path.join(ROOT, "include")]


def build(verbose: bool = False) -> str:
    """Compile every HIP source into libwino.so (always recompiles)."""
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + COMMON + DEVICE_FLAGS + ["-shared", "-o", tmp] + SOURCES
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


def device_asm() -> str:
    """gfx950 assembly of the kernels (for inspection and the packed-op check)."""
    cmd = [HIPCC] + COMMON + DEVICE_FLAGS + ["--cuda-device-only", "-S", "-o", "-", SOURCES[0]]
    return subprocess.check_output(cmd, text=True)


def resource_usage() -> str:
    """Per-kernel VGPR/AGPR/spill/occupancy report from the compiler."""
    cmd = [HIPCC] + COMMON + DEVICE_FLAGS + ["--cuda-device-only", "-c", "-o", os.devnull,
                                             "-Rpass-analysis=kernel-resource-usage", SOURCES[0]]
    p = subprocess.run(cmd, capture_output=True, text=True, check=True)
    return p.stderr


def check_no_packed_fp32(asm: str | None = None) -> None:
    asm = device_asm() if asm is None else asm
    bad = re.findall(r"\bv_pk_(?:fma|mul|add)_f32\b", asm)
    if bad:
        raise RuntimeError(f"packed fp32 instructions in device code: {sorted(set(bad))}")


if __name__ == "__main__":
    print(build(verbose=True))
    if "--check" in sys.argv:
        check_no_packed_fp32()
        print(resource_usage())
