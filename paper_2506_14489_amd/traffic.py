"""Measured HBM traffic (and vector instruction count) of the evaluation
kernel, from hardware counters.

The figures were taken with two rocprofv3 counter passes over
``bench.py`` (``--pmc FETCH_SIZE``, then ``--pmc WRITE_SIZE``; KiB per
dispatch) and scaled by what the same counters read for a plain
device-to-device copy of known size (``bench.py --copy-calibration 1024``:
a 1 GiB copy reads FETCH_SIZE = 524,300 KiB and WRITE_SIZE = 1,048,576 KiB,
so FETCH_SIZE is scaled by 2 and WRITE_SIZE by 1).

A figure is only valid for the kernel it was taken on: ``traffic_bytes``
returns None as soon as any source file that defines the evaluation kernel
differs from the one the counters were read on (a SHA-256 over those
sources, in a fixed order; the linear-layer source and the C header, which
the kernel does not depend on beyond the plan, are not part of it).
"""

from __future__ import annotations

import hashlib
import os

from . import build as _build

# 1 GiB device-to-device copy: counter reading -> bytes moved
FETCH_FACTOR = 1048576 / 524300
WRITE_FACTOR = 1048576 / 1048576

# workload name -> counters per k_eval dispatch (KiB) and the source hash
MEASURED = {
    "batched": {
        "kernel": "k_eval",
        "fetch_kib": 12965419.0,  # mean of four dispatches: 12,964,332 .. 12,966,117
        "write_kib": 1404928.0,  # four dispatches, equal
        "valu_insts": 4382490490,  # SQ_INSTS_VALU per dispatch (wave instructions; two dispatches, equal)
        "sources_sha256": "b3f36e4997a0ab6a67ffa26bf5807a1bb3cc0c5851e32c83f009608848f52bd3",
    },
}


# the files that define k_eval: its source, the device helpers, the plan and the AES tables
EVAL_SOURCES = ("redash.hip", "device.hpp", "plan.cpp", "plan.hpp", "aes_tables.hpp")


def sources_sha256() -> str:
    """SHA-256 over the evaluation kernel's source files (name and contents)."""
    h = hashlib.sha256()
    paths = [p for p in _build.SOURCES + _build.HEADERS if os.path.basename(p) in EVAL_SOURCES]
    for path in sorted(paths, key=os.path.basename):
        h.update(os.path.basename(path).encode())
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def valu_instructions(workload: str):
    """Vector ALU wave instructions per k_eval launch on ``workload``
    (SQ_INSTS_VALU), or None as for traffic_bytes."""
    rec = MEASURED.get(workload)
    if rec is None or rec["sources_sha256"] != sources_sha256() or "valu_insts" not in rec:
        return None
    return rec["valu_insts"]


def traffic_bytes(workload: str):
    """HBM bytes (reads + writes) per k_eval launch on ``workload``, or None
    if no counters were taken on it or the kernel sources changed since."""
    rec = MEASURED.get(workload)
    if rec is None or rec["sources_sha256"] != sources_sha256():
        return None
    return (rec["fetch_kib"] * FETCH_FACTOR + rec["write_kib"] * WRITE_FACTOR) * 1024.0
