"""Builds the HIP library libredash.so for gfx950, in-tree.

The library holds every kernel and the C ABI declared in include/redash.h.
Run ``python -m paper_2506_14489_amd.build`` (or call ``build()``).
"""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libredash.so")
SOURCES = [os.path.join(CSRC, "redash.hip"), os.path.join(CSRC, "linear.hip"), os.path.join(CSRC, "aes_rate.hip"),
           os.path.join(CSRC, "plan.cpp")]
HEADERS = [os.path.join(CSRC, f) for f in ("aes_tables.hpp", "aes_bitslice.hpp", "device.hpp", "plan.hpp")] + [
    os.path.join(ROOT, "include", "redash.h")
]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # no packed-FP32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-function",
]


def build(verbose: bool = False) -> str:
    """Compile every source into libredash.so (always recompiles)."""
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = [HIPCC, *FLAGS, "-I", os.path.join(ROOT, "include"), "-o", tmp, *SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        sys.stderr.write(proc.stdout + proc.stderr)
        raise RuntimeError(f"hipcc failed with exit code {proc.returncode}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
