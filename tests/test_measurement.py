"""Host-side checks of the work model that the benchmark reports against:
per-gadget gate lists, AES blocks and byte counts agree with the oracle's
gate list and sizes, the recorded HBM counters are only reported for the
kernel they were read on, and bench.py refuses more than one GPU."""

import os
import subprocess
import sys

import pytest

from oracle import oracle as O
from oracle import rns
from paper_2506_14489_amd import cost, traffic
from paper_2506_14489_amd import workloads as WL

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

BASES = [
    ([2, 3, 5, 7, 11], [4]),
    ([2, 3, 5, 7, 11, 13, 17, 19], [7]),
    ([2, 3, 5, 7, 11, 13, 17, 19, 23, 29], [8, 9]),
    ([2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37], [11]),
    ([2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37], [10, 11]),
    ([2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37], [9]),
    ([2, 5, 7, 97, 251], [1, 2]),
]


@pytest.mark.parametrize("base,S", BASES)
def test_gate_list_matches_oracle(base, S):
    """The (q, m) pairs the work model iterates over are the oracle's gates."""
    want = [(base[g.src], base[g.dst]) for g in rns.gate_list(base, S)]
    assert cost.gates(base, S) == want
    p = O.make_params(base, S, 1, 0)
    assert len(want) == O.sizes(p, 1)["gates"]


@pytest.mark.parametrize("base,S", BASES)
def test_label_sizes_match_oracle(base, S):
    for m in base:
        assert cost.lam(m) == O.lam(m)
        assert cost.words(m) == O.words(m)


@pytest.mark.parametrize("base,S", BASES)
def test_table_bytes_match_oracle_sizes(base, S):
    """Stored rows: (q-1) W_m words per gate and gadget (row reduction, Sec. 2.3)."""
    n = 37
    sz = O.sizes(O.make_params(base, S, n, 0), n)
    assert cost.table_bytes_per_gadget(base, S) * n == 4 * sz["table_words"]
    assert 2 * sum(4 * cost.words(m) for m in base) * n == 2 * 4 * sz["label_words"]


@pytest.mark.parametrize("base,S", BASES)
def test_expected_row_bytes(base, S):
    """A gate reads its row unless the digit label's colour is 0 (probability
    1/q), so the expected read is (q-1)/q of a row."""
    expect = 0.0
    for g in rns.gate_list(base, S):
        q, m = base[g.src], base[g.dst]
        expect += sum(4 * O.words(m) for c in range(1, q)) / q
    labels = 2 * sum(4 * O.words(m) for m in base)
    assert cost.bytes_per_gadget(base, S) == pytest.approx(labels + expect, rel=1e-12)


def test_batched_figures():
    """Per-gadget figures of the 16x64x56x56 workload over the first 12 primes, s = 37."""
    w = WL.by_name("batched")
    assert w.n == 16 * 64 * 56 * 56
    assert len(cost.gates(w.moduli, w.scale_idx)) == 77
    assert cost.aes_blocks_per_gadget(w.moduli, w.scale_idx) == 153
    assert cost.bytes_per_gadget(w.moduli, w.scale_idx) == pytest.approx(1825.2, abs=0.05)
    assert cost.table_bytes_per_gadget(w.moduli, w.scale_idx) == 19932


def test_aes_blocks_count_hash_calls():
    """Two AES blocks per gate, one when the output modulus is 2 (256 or 128
    pad bits); the oracle's hash of a q=3 label onto m=2 and onto m=5 agree
    with that split through their digit counts."""
    base, S = [2, 3, 5, 7, 11], [4]
    n_two = sum(1 for (_q, m) in cost.gates(base, S) if m == 2)
    assert cost.aes_blocks_per_gadget(base, S) == 2 * len(cost.gates(base, S)) - n_two
    assert len(O.hash_label(3, 2, [0] * O.lam(3), 7, 1)) == O.lam(2)
    assert len(O.hash_label(3, 5, [0] * O.lam(3), 7, 1)) == O.lam(5)


def test_op_model_constants():
    """T-table AES: 10 rounds of 16 lookups; a lookup is one index
    extraction and one XOR of vector ALU work and one 4-byte LDS read."""
    assert cost.AES_OPS_PER_BLOCK == 10 * 16 * 2 + 4 + 12
    assert cost.AES_LOOKUPS_PER_BLOCK == 160
    w = WL.by_name("batched")
    assert cost.lds_bytes_per_gadget(w.moduli, w.scale_idx) == 153 * 160 * 4
    # every gate of the base (2, 3, 37) scaled by 37: AES, fold, limb and residue terms
    assert cost.ops_per_gadget([2, 3, 37], [2]) == (
        (1 * cost.AES_OPS_PER_BLOCK + cost.words(37) + 1 + 3 * cost.words(2))
        + (2 * cost.AES_OPS_PER_BLOCK + cost.words(37) + 1 + cost.LIMB_OPS_PER_WORD * cost.words(3)
           + cost.OPS_PER_RESIDUE * cost.lam(3))
        + (2 * cost.AES_OPS_PER_BLOCK + cost.words(2) + 1 + cost.LIMB_OPS_PER_WORD * cost.words(3)
           + cost.OPS_PER_RESIDUE * cost.lam(3))
        + (2 * cost.AES_OPS_PER_BLOCK + cost.words(2) + 1 + cost.LIMB_OPS_PER_WORD * cost.words(37)
           + cost.OPS_PER_RESIDUE * cost.lam(37))
        + (2 * cost.AES_OPS_PER_BLOCK + cost.words(3) + 1 + cost.LIMB_OPS_PER_WORD * cost.words(37)
           + cost.OPS_PER_RESIDUE * cost.lam(37)))


def test_traffic_only_for_unchanged_sources(monkeypatch):
    rec = traffic.MEASURED["batched"]
    monkeypatch.setitem(rec, "sources_sha256", traffic.sources_sha256())
    b = traffic.traffic_bytes("batched")
    assert b == pytest.approx((rec["fetch_kib"] * traffic.FETCH_FACTOR + rec["write_kib"]) * 1024)
    monkeypatch.setitem(rec, "sources_sha256", "0" * 64)
    assert traffic.traffic_bytes("batched") is None
    assert traffic.traffic_bytes("no-such-workload") is None


def test_copy_calibration_factors():
    assert traffic.FETCH_FACTOR == pytest.approx(2.0, rel=1e-4)
    assert traffic.WRITE_FACTOR == 1.0


def test_bench_refuses_several_gpus():
    proc = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                          capture_output=True, text=True, timeout=120)
    assert proc.returncode == 2
    assert "one GPU" in proc.stderr
    assert proc.stdout == ""
