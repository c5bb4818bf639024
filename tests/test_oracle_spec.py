"""Pins of the oracle's garbling hash and PRG, step by step.

The paper fixes the projection-gate algebra (Sec. 2.3) but no hash, PRG or
tweak layout, so the oracle's ``hash_label`` and ``prg_label`` follow a
construction of our own.  These tests pin every step of it against things
outside the oracle:

* sigma is checked to be a linear orthomorphism of GF(2)^128 (sigma and
  x -> sigma(x) xor x both bijective), the property the construction relies
  on (Guo, Katz, Wang and Yu, 2020), by the rank of its matrix;
* the fold lanes, sigma, the tweak words (gadget id in bits 96-127,
  4 tau + j in bits 0-63, also for tau >= 2^32 and where 4 tau wraps) and the
  Matyas-Meyer-Oseas feed-forward are recomputed on Python integers with
  libcrypto's AES (tests/rspec.py), value by value;
* the digit extraction is recomputed with Python big integers;
* the PRG counter C_h = stream 2^120 + 2 idx + h is recomputed the same way,
  for idx at and above 2^31, 2^32 and 2^63;
* the offsets and input zero-labels of a gadget far into the index range, and
  the hash of every gate of whole gadgets (tweak a G + g, gadget id = seed
  mod 2^32), are recomputed from those pieces;
* the known-answer files in tests/golden hold the oracle's values; each line
  is checked against libcrypto here.

Planted mistakes (sigma's halves swapped, the gadget id in the wrong lane, a
tweak without the factor 4, a PRG counter without the factor 2) are shown to
fail these checks.
"""

from __future__ import annotations

import os

import numpy as np
import pytest

from oracle import oracle as O
from oracle import rns

rspec = pytest.importorskip("rspec")

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module")
def aes():
    try:
        return rspec.LibCrypto()
    except OSError:
        pytest.skip("libcrypto not available")


def _int(limbs) -> int:
    return sum(int(v) << (32 * i) for i, v in enumerate(limbs))


# ---------------------------------------------------------------------------
# sigma and fold
# ---------------------------------------------------------------------------


def _gf2_rank(rows) -> int:
    rows = [r for r in rows]
    rank = 0
    for bit in range(128):
        piv = next((i for i in range(rank, len(rows)) if (rows[i] >> bit) & 1), None)
        if piv is None:
            continue
        rows[rank], rows[piv] = rows[piv], rows[rank]
        for i in range(len(rows)):
            if i != rank and (rows[i] >> bit) & 1:
                rows[i] ^= rows[rank]
        rank += 1
    return rank


def _oracle_sigma(x: int) -> int:
    """sigma as the oracle computes it: a label over Z_2 packs into four words
    that the fold leaves in place, so its bits are x."""
    res = [(x >> i) & 1 for i in range(128)]
    fx, u, _ = O.hash_parts(2, 3, res, 0, 0)
    assert _int(fx) == x
    return _int(u)


def test_sigma_is_a_linear_orthomorphism():
    cols = [_oracle_sigma(1 << i) for i in range(128)]
    # linear: sigma(x ^ y) = sigma(x) ^ sigma(y) on random pairs
    rng = np.random.default_rng(5)
    for _ in range(20):
        x = int(rng.integers(0, 2 ** 63)) | (int(rng.integers(0, 2 ** 63)) << 64)
        expect = 0
        for i in range(128):
            if (x >> i) & 1:
                expect ^= cols[i]
        assert _oracle_sigma(x) == expect
    # sigma and sigma ^ identity are both bijective: full rank over GF(2)
    assert _gf2_rank(cols) == 128
    assert _gf2_rank([c ^ (1 << i) for i, c in enumerate(cols)]) == 128
    # and it is the stated map ((x_hi ^ x_lo) << 64) | x_hi
    for i in (0, 5, 63, 64, 100, 127):
        assert cols[i] == rspec.sigma(1 << i)


@pytest.mark.parametrize("q", [2, 3, 5, 7, 11, 17, 37, 97, 251, 4, 32, 128])
def test_fold_and_sigma_of_labels(q):
    rng = np.random.default_rng(q)
    for _ in range(5):
        res = rng.integers(0, q, size=O.lam(q))
        x, u, _ = O.hash_parts(q, 5, res, 1, 2)
        words = rspec.pack(q, res)
        assert len(words) == O.words(q)
        assert _int(x) == rspec.fold(words)
        assert _int(u) == rspec.sigma(rspec.fold(words))


# ---------------------------------------------------------------------------
# the hash value and its digits
# ---------------------------------------------------------------------------

PAIRS = [(2, 37), (37, 2), (3, 5), (11, 13), (37, 31), (4, 16), (32, 167), (251, 97), (2, 2), (128, 7)]
TAUS = [0, 3, 2 ** 31 + 1, 2 ** 32, 2 ** 32 + 77, 2 ** 45 + 3, 2 ** 62 - 1, 2 ** 62, 2 ** 63 + 5, 2 ** 64 - 1]
GIDS = [0, 1, 0x7FFFFFFF, 0x80000000, 0xFFFFFFFF]


@pytest.mark.parametrize("q,m", PAIRS)
def test_hash_value_is_aes_mmo_of_sigma_xor_tweak(aes, q, m):
    rng = np.random.default_rng(q * 256 + m)
    n = 1 if m == 2 else 2
    for tau in TAUS:
        gid = GIDS[int(rng.integers(0, len(GIDS)))]
        res = rng.integers(0, q, size=O.lam(q))
        _, u, V = O.hash_parts(q, m, res, gid, tau)
        u = _int(u)
        V = _int(V)
        for j in range(2):
            Uj = (V >> (128 * j)) & rspec.M128
            if j >= n:
                assert Uj == 0
                continue
            t = rspec.tweak(gid, tau, j)
            assert t >> 96 == gid and (t >> 64) & 0xFFFFFFFF == 0
            # U_j xor u xor T_j is AES_K(u xor T_j) under the fixed key 00 01 .. 0f
            assert Uj ^ u ^ t == aes.aes_int(rspec.HASH_KEY, u ^ t), (q, m, tau, j)
        assert V == rspec.hash_value(aes, q, m, res, gid, tau)


@pytest.mark.parametrize("q,m", PAIRS)
def test_hash_digits_are_the_fraction_digits(aes, q, m):
    rng = np.random.default_rng(q * 512 + m)
    for tau in TAUS[::3]:
        gid = int(rng.integers(0, 2 ** 32))
        res = rng.integers(0, q, size=O.lam(q))
        got = [int(v) for v in O.hash_label(q, m, res, gid, tau)]
        assert got == rspec.hash_label(aes, q, m, res, gid, tau)
        _, _, V = O.hash_parts(q, m, res, gid, tau)
        n = 1 if m == 2 else 2
        # as one number: the digits are floor(V m^lambda / 2^(128 n)) in base m
        top = (_int(V) * m ** O.lam(m)) >> (128 * n)
        val = 0
        for d in got:
            val = val * m + d
        assert val == top


# ---------------------------------------------------------------------------
# the PRG and what the garbler draws from it
# ---------------------------------------------------------------------------

IDXS = [0, 1, 2 ** 31 - 1, 2 ** 31, 2 ** 31 + 7, 2 ** 32 + 3, 2 ** 40 + 1, 2 ** 63 + 1]


@pytest.mark.parametrize("seed", [0, 3, 2 ** 33 + 9, 2 ** 64 - 1])
def test_prg_counter_blocks(aes, seed):
    key = seed.to_bytes(16, "little")
    for stream in (1, 2):
        for idx in IDXS:
            V = _int(O.prg_value(seed, stream, idx))
            for h in range(2):
                c = (stream << 120) | ((2 * idx + h) & rspec.M64)
                assert (V >> (128 * h)) & rspec.M128 == aes.aes_int(key, c), (seed, stream, idx, h)


@pytest.mark.parametrize("m", [2, 3, 11, 37, 4, 32, 251])
def test_prg_label_digits(aes, m):
    for seed, stream, idx, first in [(1, 1, 3, True), (2 ** 35 + 1, 2, 2 ** 31 + 4, False),
                                     (7, 2, 2 ** 32 + 1, False), (9, 1, 0, True)]:
        got = [int(v) for v in O.prg_label(seed, stream, idx, m, first)]
        pw = m > 2 and m & (m - 1) == 0
        r0 = (m // 2 if pw else m - 1) if first else m
        exp = rspec.frac_digits(rspec.prg_value(aes, seed, stream, idx), 256, [r0] + [m] * (O.lam(m) - 1))
        assert got == exp


@pytest.mark.parametrize("moduli,S,a", [((2, 3, 5, 7, 11), (4,), 2 ** 31 + 17),
                                         (tuple(rns.first_primes(12)), (11,), 2 ** 29 + 1000),
                                         ((3, 5, 7, 11, 13, 17, 19, 32), (7,), 123456789)])
def test_offsets_and_zero_labels_follow_the_prg(aes, moduli, S, a):
    """A gadget far into the index range (a k + i at or above 2^31)."""
    seed = 2 ** 36 + 41
    op = O.make_params(list(moduli), list(S), 1, seed)
    offs, zin, _, _ = O.garble(op, a, 1, with_tables=False)
    k = len(moduli)
    for i, m in enumerate(moduli):
        R = O.pk32_unpack(m, O.label_view(offs, op, 1, i)[:, 0])
        assert [int(v) for v in R] == rspec.offset(aes, seed, i, m)
        Z = O.pk32_unpack(m, O.label_view(zin, op, 1, i)[:, 0])
        assert [int(v) for v in Z] == rspec.zero_label(aes, seed, a, i, k, m)


def _addmul(m, y, x, c):
    return [(int(a) + c * int(b)) % m for a, b in zip(y, x)]


@pytest.mark.parametrize("moduli,S,a,x", [((2, 3, 5, 7, 11), (4,), 2 ** 29 + 5, -1000),
                                           ((2, 3, 5, 7, 11, 13), (2, 5), 2 ** 28 + 3, 12345),
                                           ((32, 167, 173), (0,), 2 ** 31 + 1, -7)])
def test_every_gate_hash_uses_tweak_a_g_plus_g(aes, moduli, S, a, x):
    """Garbler side: B0 = H(A0 + v0 R_q, a G + g) - (v0 mod m) R_m for every
    gate g of a gadget with a G >= 2^32, gadget id = seed mod 2^32 (seed above
    2^32).  Evaluator side: a gate whose digit label has colour 0 reads no row,
    so its projected label is H(A, a G + g) itself."""
    seed = 2 ** 34 + 99
    gid = seed % 2 ** 32
    op = O.make_params(list(moduli), list(S), 1, seed)
    G = O.sizes(op, 1)["gates"]
    assert a * G >= 2 ** 32
    t = O.trace(op, a, x)
    gates = O.gate_list(op)
    colour0 = 0
    for g, (src, dst, *_r) in enumerate(gates):
        q, m = moduli[src], moduli[dst]
        lq, lm = O.lam(q), O.lam(m)
        Rq, Rm = t["offsets"][src][:lq], t["offsets"][dst][:lm]
        A0 = t["gb_in"][g][:lq]
        v0 = (-int(A0[0])) * pow(int(Rq[0]), -1, q) % q
        H = rspec.hash_label(aes, q, m, _addmul(q, A0, Rq, v0), gid, a * G + g)
        B0 = _addmul(m, H, Rm, (-v0) % m)
        assert [int(v) for v in t["gb_out"][g][:lm]] == B0, g
        A = t["ev_in"][g][:lq]
        if int(A[0]) == 0:
            colour0 += 1
            E = rspec.hash_label(aes, q, m, A, gid, a * G + g)
            assert [int(v) for v in t["ev_out"][g][:lm]] == E, g
    assert G > 0


# ---------------------------------------------------------------------------
# known-answer files
# ---------------------------------------------------------------------------


def _hash_kat():
    with open(os.path.join(GOLDEN, "hash_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            q, m, gid, tau, a, h = line.split()
            yield (int(q), int(m), int(gid, 16), int(tau), [int(v, 16) for v in a.split(",")],
                   [int(v, 16) for v in h.split(",")])


def test_hash_known_answers(aes):
    count = 0
    for q, m, gid, tau, aw, hw in _hash_kat():
        res = O.pk32_unpack(q, np.array(aw, np.uint32))
        assert [int(v) for v in O.pk32_pack(m, O.hash_label(q, m, res, gid, tau))] == hw
        assert rspec.pack(m, rspec.hash_label(aes, q, m, res, gid, tau)) == hw
        count += 1
    assert count >= 100


def test_prg_known_answers(aes):
    count = 0
    with open(os.path.join(GOLDEN, "prg_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            seed, stream, idx, v = line.split()
            V = [int(x, 16) for x in v.split(",")]
            assert [int(x) for x in O.prg_value(int(seed), int(stream), int(idx))] == V
            assert _int(V) == rspec.prg_value(aes, int(seed), int(stream), int(idx))
            count += 1
    assert count == 56


# ---------------------------------------------------------------------------
# the checks above catch plausible mistakes
# ---------------------------------------------------------------------------


def test_planted_mistakes_are_caught(aes):
    rng = np.random.default_rng(9)
    q, m, gid, tau = 11, 13, 0x80000003, 2 ** 32 + 9
    res = rng.integers(0, q, size=O.lam(q))
    _, _, V = O.hash_parts(q, m, res, gid, tau)
    V = _int(V)
    u_ok = rspec.sigma(rspec.fold(rspec.pack(q, res)))

    def value(u, tw):
        out = 0
        for j in range(2):
            t = tw(j)
            out |= (aes.aes_int(rspec.HASH_KEY, u ^ t) ^ u ^ t) << (128 * j)
        return out

    good = value(u_ok, lambda j: rspec.tweak(gid, tau, j))
    assert good == V
    x = rspec.fold(rspec.pack(q, res))
    lo, hi = x & rspec.M64, x >> 64
    swapped = (hi << 64) | (hi ^ lo)
    assert value(swapped, lambda j: rspec.tweak(gid, tau, j)) != V
    assert value(u_ok, lambda j: (gid << 64) | ((4 * tau + j) & rspec.M64)) != V  # gadget id in lane 2
    assert value(u_ok, lambda j: (gid << 96) | ((tau + j) & rspec.M64)) != V  # no factor 4
    assert value(u_ok, lambda j: (gid << 96) | ((4 * (tau & 0xFFFFFFFF) + j))) != V  # tau cut to 32 bits
    # the PRG counter without the factor 2, or with the stream in the wrong byte
    seed, idx = 5, 2 ** 31 + 3
    P = _int(O.prg_value(seed, 2, idx))
    key = seed.to_bytes(16, "little")
    assert aes.aes_int(key, (2 << 120) | idx) != P & rspec.M128
    assert aes.aes_int(key, (2 << 112) | (2 * idx)) != P & rspec.M128
    assert aes.aes_int(key, (2 << 120) | (2 * idx)) == P & rspec.M128
