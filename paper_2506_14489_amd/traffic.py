"""Measured HBM traffic of the evaluation kernel, from hardware counters.

The figures were taken with two rocprofv3 counter passes over
``bench.py`` (``--pmc FETCH_SIZE``, then ``--pmc WRITE_SIZE``; KiB per
dispatch) and scaled by what the same counters read for a plain
device-to-device copy of known size (``bench.py --copy-calibration 1024``:
a 1 GiB copy reads FETCH_SIZE = 524,300 KiB and WRITE_SIZE = 1,048,576 KiB,
so FETCH_SIZE is scaled by 2 and WRITE_SIZE by 1).

A figure is only valid for the kernel it was taken on: ``traffic_bytes``
returns None as soon as any source file of the library differs from the one
the counters were read on (a SHA-256 over the sources, in a fixed order).
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
        "fetch_kib": 15211545.7,  # mean of two dispatches: 15,210,247 and 15,212,844
        "write_kib": 5049479.0,  # mean of 5,049,628 and 5,049,330
        "sources_sha256": "eb8e0b936b0cb705748016c5e4da501de551fc4e19b98a8568b5201710d774a1",
    },
}


def sources_sha256() -> str:
    """SHA-256 over the library's source files (name and contents)."""
    h = hashlib.sha256()
    for path in sorted(_build.SOURCES + _build.HEADERS, key=os.path.basename):
        h.update(os.path.basename(path).encode())
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_bytes(workload: str):
    """HBM bytes (reads + writes) per k_eval launch on ``workload``, or None
    if no counters were taken on it or the kernel sources changed since."""
    rec = MEASURED.get(workload)
    if rec is None or rec["sources_sha256"] != sources_sha256():
        return None
    return (rec["fetch_kib"] * FETCH_FACTOR + rec["write_kib"] * WRITE_FACTOR) * 1024.0
