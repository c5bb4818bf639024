"""Pins of the value-level oracle (oracle/rns.py) against what the paper and
plain arithmetic fix: Table 1, the signed-encoding example of Sec. 2.4,
floor division by brute force, and Python's own divmod for MRS digits."""

import os
import random

import pytest

from oracle import rns

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1.txt")


def _vec(s):
    return [int(v) for v in s.split("/")]


def _table1_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            c = line.split()
            rows.append({
                "x": int(c[0]), "xs": int(c[1]), "phi_x": _vec(c[2]), "x_up": int(c[3]),
                "x_up_s": int(c[4]), "phi_x_up": _vec(c[5]), "y_prime": _vec(c[6]),
                "crt_y_prime": int(c[7]), "crt_y_prime_s": int(c[8]), "y": int(c[9]),
                "phi_y": _vec(c[10]), "phi_y_down": _vec(c[11]), "y_down": int(c[12]),
                "y_down_s": int(c[13]),
            })
    return rows


def test_table1_every_column():
    """Table 1 (Sec. 3.4): s = 3, base (2, 3), all of Z_6."""
    base, S = [2, 3], [1]
    P = rns.cardinality(base)
    half, down = rns.shift_constants(base, S)
    assert (half, down) == (3, 1)
    rows = _table1_rows()
    assert [r["x"] for r in rows] == list(range(6))
    for r in rows:
        x = r["x"]
        assert rns.signed_decode(x, P) == r["xs"]
        assert rns.rns(x, base) == r["phi_x"]
        x_up = (x + half) % P
        assert x_up == r["x_up"]
        assert rns.signed_decode(x_up, P) == r["x_up_s"]
        assert rns.rns(x_up, base) == r["phi_x_up"]
        # READING: the column "y' = [b(phi(x)), 0]" is b applied to phi(x_up).
        y_prime = rns.scale_residues(rns.rns(x_up, base), base, 1)
        assert y_prime == r["y_prime"]
        assert rns.crt(y_prime, base) == r["crt_y_prime"]
        assert rns.signed_decode(rns.crt(y_prime, base), P) == r["crt_y_prime_s"]
        # y: the base extension fills the missing residue.
        y_full = [y_prime[0], rns.be_missing_residue(y_prime, base)]
        assert rns.crt(y_full, base) == r["y"]
        assert y_full == r["phi_y"]
        y_down = (r["y"] - down) % P
        assert rns.rns(y_down, base) == r["phi_y_down"]
        assert y_down == r["y_down"]
        assert rns.signed_decode(y_down, P) == r["y_down_s"]
        # The whole gadget agrees with the table and with floor division.
        t = rns.gadget_trace(base, S, r["xs"])
        assert t["x_up"] == r["x_up"]
        assert t["out"] == r["phi_y"]
        assert t["y"] == r["y_down_s"] == r["xs"] // 3


def test_printed_missing_residue_formula_disagrees_with_table1():
    """The missing-residue formula as printed after Eq. (rns_to_mrs) gives
    [y]_2 = 0 for Table 1's first row, where the table has [1, 1]; the reading
    used by the oracle reproduces the table (see be_missing_residue)."""
    base = [2, 3]
    y_prime = [1, 0]
    assert rns.be_missing_residue_printed(y_prime, base) == 0
    assert rns.be_missing_residue(y_prime, base) == 1


@pytest.mark.parametrize("base", [[2, 3], [2, 3, 5], [2, 3, 5, 7], [3, 5, 7, 11], [2, 3, 5, 7, 11]])
def test_missing_residue_reading_brute_force(base):
    """For every y < P_{k-1}: the corrected formula returns y mod p_k."""
    Pk1 = rns.cardinality(base[:-1])
    for y in range(Pk1):
        y_prime = rns.rns(y, base[:-1]) + [0]
        assert rns.be_missing_residue(y_prime, base) == y % base[-1]


def test_be_recursion_digits_are_mrs_digits():
    """Eq. (rns_to_mrs) yields the associated MRS digits (checked with divmod)."""
    base = [2, 3, 5, 7, 11]
    P = rns.cardinality(base)
    for y in range(0, P, 7):
        digits, _ = rns.be_recursion(rns.rns(y, base), base)
        assert digits == rns.mrs_digits(y, base)


def test_signed_encoding_example():
    """Sec. 2.4: (0, 1, 2, -2, -1) -> (0, 1, 2, 3, 4) in Z_5."""
    assert [rns.signed_encode(x, 5) for x in (0, 1, 2, -2, -1)] == [0, 1, 2, 3, 4]
    assert [rns.signed_decode(v, 5) for v in range(5)] == [0, 1, 2, -2, -1]


def test_crt_and_mrs_round_trip():
    base = rns.first_primes(6)
    P = rns.cardinality(base)
    rng = random.Random(5)
    for _ in range(500):
        y = rng.randrange(P)
        assert rns.crt(rns.rns(y, base), base) == y
        assert rns.mrs_value(rns.mrs_digits(y, base), base) == y


def test_inverses():
    for m in rns.first_primes(12):
        for a in range(1, m):
            assert (a * rns.inv_mod(a, m)) % m == 1


def test_first_primes_cpm():
    assert rns.first_primes(5) == [2, 3, 5, 7, 11]
    assert rns.cardinality(rns.first_primes(5)) == 2310
    assert rns.cardinality(rns.first_primes(8)) == 9699690
    assert rns.cardinality(rns.first_primes(10)) == 6469693230
    assert rns.cardinality(rns.first_primes(12)) == 7420738134810


CASES = [
    ([2, 3], [1]),            # s = 3 (Table 1)
    ([2, 3, 5], [2]),         # s = 5
    ([2, 3, 5], [1, 2]),      # s = 15 (product of base moduli)
    ([2, 3, 5, 7], [2, 3]),   # s = 35
    ([2, 3, 5, 7], [1]),      # s = 3, scaling modulus not last
    ([2, 3, 5, 7, 11], [4]),  # s = 11
    ([2, 3, 5, 7, 11], [1, 3, 4]),  # s = 231
]


@pytest.mark.parametrize("base,S", CASES)
def test_gadget_is_floor_division_brute_force(base, S):
    """Sec. 3.2: y = floor(x/s) for every x of the signed range of Z_P."""
    P = rns.cardinality(base)
    s = rns.cardinality([base[i] for i in S])
    for x in range(-(P // 2), P // 2):
        assert rns.plain_scale(x, base, S) == x // s, (x, base, S)


def test_gadget_floor_division_large_base_sampled():
    base = rns.first_primes(12)
    P = rns.cardinality(base)
    rng = random.Random(3)
    for S in ([11], [10, 11], [9, 10, 11], [5]):
        s = rns.cardinality([base[i] for i in S])
        xs = [rng.randrange(-(P // 2), P // 2) for _ in range(200)]
        xs += [-(P // 2), P // 2 - 1, 0, -1, s - 1, -s, s, -s - 1]
        for x in xs:
            assert rns.plain_scale(x, base, S) == x // s


def test_shift_constants_reading():
    """Sec. 3.4 shifts by P/2 and P/(2s).  READING where they are not integers:
    ShiftUp by U = floor(P/2), ShiftDown by floor(U/s).  Where they are
    integers nothing changes (Table 1: up 3, down 1)."""
    assert rns.shift_constants([2, 3], [1]) == (3, 1)
    assert rns.rounding_offset([2, 3], [1]) == 0
    assert rns.shift_constants([3, 5, 7], [2]) == (52, 7)   # P = 105 odd
    assert rns.rounding_offset([3, 5, 7], [2]) == 3
    Q = 167 * 173
    assert rns.shift_constants([32, 167, 173], [0]) == (16 * Q, (16 * Q) // 32)
    assert rns.rounding_offset([32, 167, 173], [0]) == 16  # s/2: round half up
    for k in range(3, 13):
        base = rns.first_primes(k)
        for S in ([k - 1], [k - 2, k - 1]):
            assert rns.rounding_offset(base, S) == 0


# Bases the paper's Sec. 4 uses or that stress the reading: a power-of-two
# modulus (scaled by, or among the remaining moduli) and odd P.
ROUNDING_CASES = [
    ([2, 3, 5], [0]),          # s = 2, 2 scaled by: U mod s = 1
    ([3, 4, 5], [1]),          # s = 4
    ([4, 5, 7], [0]),          # s = 4, 4 first
    ([5, 7, 8], [2]),          # s = 8
    ([3, 5, 8], [2]),          # s = 8
    ([3, 5, 7, 16], [3]),      # s = 16
    ([3, 5, 7, 16], [0]),      # s = 3, 16 among R
    ([3, 5, 7], [2]),          # P odd, s = 7
    ([3, 5, 7], [0, 1]),       # P odd, s = 15
    ([8, 11, 13], [0]),        # s = 8, 2^l with odd primes
]


@pytest.mark.parametrize("base,S", ROUNDING_CASES)
def test_gadget_rounding_brute_force(base, S):
    """Every x of the signed range [-floor(P/2), ceil(P/2) - 1] (Sec. 2.4):
    the residue-level gadget returns floor((x + r)/s), r = floor(P/2) mod s."""
    P = rns.cardinality(base)
    s = rns.cardinality([base[i] for i in S])
    r = (P // 2) % s
    assert r == rns.rounding_offset(base, S)
    for x in range(-(P // 2), P - P // 2):
        assert rns.plain_scale(x, base, S) == (x + r) // s, (x, base, S)


@pytest.mark.parametrize("base,S", ROUNDING_CASES)
def test_no_shift_gives_floor_on_the_whole_signed_range(base, S):
    """The alternative reading weighed against the kept one: a ShiftUp U that
    is a multiple of s (U = s floor(floor(P/2)/s), ShiftDown U/s) makes the
    gadget's floor((x_up)/s) - U/s exactly floor(x/s) -- but only where
    x + U stays in [0, P): the r = floor(P/2) mod s most negative inputs of
    the signed range wrap.  And no shift at all keeps the whole signed range
    in [0, P) except U = floor(P/2): so when r > 0 a gadget either rounds
    (the kept reading) or wraps r inputs."""
    P = rns.cardinality(base)
    s = rns.cardinality([base[i] for i in S])
    r = rns.rounding_offset(base, S)
    lo, hi = -(P // 2), P - P // 2 - 1
    assert [U for U in range(P) if lo + U >= 0 and hi + U < P] == [P // 2]
    U = s * ((P // 2) // s)
    bad = [x for x in range(lo, hi + 1) if ((x + U) % P) // s - U // s != x // s]
    assert bad == list(range(lo, lo + r))
    # the kept reading: exact on every x of the range, floor((x + r)/s)
    if r:
        assert any((x + r) // s != x // s for x in range(lo, hi + 1))


def test_round_half_up_for_half_offset():
    """With r = s/2 (a 2^l modulus scaled by, Sec. 4's bases) the gadget rounds
    x/s to the nearest integer, halves upward."""
    base, S = [5, 7, 8], [2]
    assert rns.rounding_offset(base, S) == 4
    for x in range(-140, 140):
        want = (2 * x + 8) // 16  # nearest, ties up
        assert rns.plain_scale(x, base, S) == want


def test_gate_counts():
    """Gates per instance: sum_{a=1}^{t} (k-a) for the division steps plus
    u(u-1)/2 + u t for the base extension."""
    for k in range(3, 13):
        base = rns.first_primes(k)
        for S in ([k - 1], [k - 2, k - 1]):
            t, u = len(S), k - len(S)
            G = len(rns.gate_list(base, S))
            assert G == sum(k - a for a in range(1, t + 1)) + u * (u - 1) // 2 + u * t


def test_be_cost_formula_reading():
    """Sec. 3.3 cost: sum_{i=1}^{k-1} sum_{j=i}^{k-1} p_j ciphertexts for the BE.
    READING: for one scaling modulus it equals the base-extension ciphertexts
    without row reduction when the remaining moduli are listed largest first
    (the gadget extracts digits from the smallest modulus first)."""
    for k in (3, 5, 8, 12):
        base = rns.first_primes(k)
        S = [k - 1]
        _, b = rns.ciphertext_counts(base, S, row_reduction=False)
        R = base[:-1]
        assert b == rns.be_cost_formula(list(reversed(R)))
    # the reference points quoted for the 8- and 12-prime bases
    assert rns.ciphertext_counts(rns.first_primes(8), [7], False)[1] == 161
    assert rns.ciphertext_counts(rns.first_primes(12), [11], False)[1] == 627


def test_division_step_ciphertexts():
    """Division by one base modulus p: (k-1) projection gates from Z_p, each
    with p-1 rows after row reduction."""
    base = rns.first_primes(12)
    a, _ = rns.ciphertext_counts(base, [11], row_reduction=True)
    assert a == 11 * 36
