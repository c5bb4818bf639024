"""Host code under the address and undefined-behaviour sanitizers.

* tests/oracle_check.c drives the C oracle end to end (garble with and
  without tables, encode, evaluate, decode, trace, hash and PRG helpers with
  extreme arguments) on eight small bases and checks every decode.
* tests/plan_check.cpp checks every per-modulus constant of the library's
  host plan (plan.cpp) over the operand range the kernels use it on, for
  every modulus the library accepts, and runs the evaluator's target-major
  schedule on values for many bases.
* tests/aes_bitslice_check.cpp checks the bitsliced AES (S-box circuit,
  rounds, transpose) against GF(2^8) arithmetic and a byte-level AES.

Both are built with gcc/g++ (host code only; no GPU code is built here).
"""

from __future__ import annotations

import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g", "-O1"]


def _run(cmd_build, exe, tmp_path):
    r = subprocess.run(cmd_build, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    return r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_check")
    out = _run(["gcc", "-std=gnu11", *SAN, os.path.join(HERE, "oracle_check.c"),
                os.path.join(ROOT, "oracle", "gc_oracle.c"), "-o", exe], exe, tmp_path)
    assert "oracle check: 0 failures" in out


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the HIP headers")
def test_plan_constants_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_check")
    out = _run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                os.path.join(HERE, "plan_check.cpp"),
                os.path.join(ROOT, "paper_2506_14489_amd", "csrc", "plan.cpp"), "-o", exe], exe, tmp_path)
    assert " 0 failures" in out
    # every accepted modulus: 54 primes and 6 powers of two up to 255; all but
    # 4, 16 and 41..61 take the evaluator's fast path
    assert "accepted 60 moduli, 52 on the fast path" in out, out
    assert "generic: 4 16 41 47 53 59 61\n" in out, out


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the HIP headers")
def test_bitsliced_aes_under_sanitizers(tmp_path):
    exe = str(tmp_path / "aes_bitslice_check")
    out = _run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                os.path.join(HERE, "aes_bitslice_check.cpp"), "-o", exe], exe, tmp_path)
    assert "aes bitslice check: 0 failures" in out, out
