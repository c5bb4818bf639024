"""Pins of the garbled oracle (oracle/gc_oracle.c).

* AES-128: FIPS-197 Appendix A.1 (key expansion), Appendix B and C.1
  (cipher), S-box entries of FIPS-197 Figure 7, and the system libcrypto on
  random keys and blocks.
* Digit extraction: closed form floor(V * prod(r) / 2^(32 n)) in Python
  integers.
* Garbling algebra (Sec. 2.3): every wire label the evaluator holds equals the
  garbler's zero-label plus the plaintext value (from oracle/rns.py) times
  that modulus's offset, at every gate; every table row decrypts to the
  right label for every input value; colours are distinct.
* Result (Sec. 3.2): decode gives floor(x/s) for every input of small bases.

The paper fixes no hash, PRG or encoding: those are this design's
construction, pinned bit for bit by a second statement on Python integers
with libcrypto's AES (fold, sigma, tweak words, feed-forward, digits, PRG
counters) and by known-answer files in tests/test_oracle_spec.py; the HIP
library implements them once more without shared code.
"""

import ctypes
import ctypes.util
import random

import numpy as np
import pytest

from oracle import oracle as O
from oracle import rns

# ----------------------------------------------------------------------------
# AES-128
# ----------------------------------------------------------------------------


def test_fips197_c1():
    key = bytes(range(16))
    pt = bytes.fromhex("00112233445566778899aabbccddeeff")
    assert O.aes128(key, pt).hex() == "69c4e0d86a7b0430d8cdb78070b4c55a"


def test_fips197_appendix_b():
    key = bytes.fromhex("2b7e151628aed2a6abf7158809cf4f3c")
    pt = bytes.fromhex("3243f6a8885a308d313198a2e0370734")
    assert O.aes128(key, pt).hex() == "3925841d02dc09fbdc118597196a0b32"


def test_fips197_key_expansion_a1():
    w = O.aes128_key_expansion(bytes.fromhex("2b7e151628aed2a6abf7158809cf4f3c"))
    assert w[16:20].hex() == "a0fafe17"  # w[4]
    assert w[172:176].hex() == "b6630ca6"  # w[43]


def test_sbox_entries():
    s = O.sbox()
    assert s[0x00] == 0x63 and s[0x01] == 0x7C and s[0x10] == 0xCA
    assert s[0x53] == 0xED and s[0xFF] == 0x16
    assert sorted(s) == list(range(256))  # a permutation


def _libcrypto():
    name = ctypes.util.find_library("crypto")
    if not name:
        return None
    try:
        return ctypes.CDLL(name)
    except OSError:
        return None


def test_aes_matches_libcrypto():
    lc = _libcrypto()
    if lc is None:
        pytest.skip("libcrypto not available")
    lc.EVP_CIPHER_CTX_new.restype = ctypes.c_void_p
    lc.EVP_aes_128_ecb.restype = ctypes.c_void_p
    lc.EVP_EncryptInit_ex.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_char_p, ctypes.c_char_p]
    lc.EVP_CIPHER_CTX_set_padding.argtypes = [ctypes.c_void_p, ctypes.c_int]
    lc.EVP_EncryptUpdate.argtypes = [ctypes.c_void_p, ctypes.c_char_p, ctypes.POINTER(ctypes.c_int),
                                     ctypes.c_char_p, ctypes.c_int]
    lc.EVP_CIPHER_CTX_free.argtypes = [ctypes.c_void_p]
    rng = random.Random(11)
    for _ in range(200):
        key = bytes(rng.randrange(256) for _ in range(16))
        pt = bytes(rng.randrange(256) for _ in range(16))
        ctx = lc.EVP_CIPHER_CTX_new()
        assert lc.EVP_EncryptInit_ex(ctx, lc.EVP_aes_128_ecb(), None, key, None) == 1
        lc.EVP_CIPHER_CTX_set_padding(ctx, 0)
        out = ctypes.create_string_buffer(32)
        n = ctypes.c_int(0)
        assert lc.EVP_EncryptUpdate(ctx, out, ctypes.byref(n), pt, 16) == 1
        lc.EVP_CIPHER_CTX_free(ctx)
        assert out.raw[:16] == O.aes128(key, pt)


# ----------------------------------------------------------------------------
# label sizes, packing, digits
# ----------------------------------------------------------------------------

PRIMES = rns.first_primes(12)


@pytest.mark.parametrize("m", PRIMES + [97, 107, 167, 173, 251])
def test_lambda_is_minimal(m):
    lam = O.lam(m)
    assert m ** lam >= 2 ** 128 > m ** (lam - 1)


def test_lambda_11_boundary():
    # 11^37 is just below 2^128, so 38 residues are needed.
    assert 11 ** 37 < 2 ** 128 and O.lam(11) == 38


@pytest.mark.parametrize("m", PRIMES)
def test_pk32_round_trip_and_positions(m):
    rng = np.random.default_rng(m)
    lam = O.lam(m)
    res = rng.integers(0, m, size=lam).astype(np.uint32)
    w = O.pk32_pack(m, res)
    assert np.array_equal(O.pk32_unpack(m, w), res)
    b = (m - 1).bit_length()
    g = 32 // b
    assert len(w) == -(-lam // g)
    # residue i sits at bit b*(i mod g) of word i // g
    for i in range(lam):
        assert (int(w[i // g]) >> (b * (i % g))) & ((1 << b) - 1) == res[i]
    # unused bits are zero
    total = sum(int(v) << (32 * j) for j, v in enumerate(w))
    used = sum(int(r) << (32 * (i // g) + b * (i % g)) for i, r in enumerate(res))
    assert total == used


@pytest.mark.parametrize("nl", [4, 8])
def test_fraction_digits_closed_form(nl):
    rng = random.Random(nl)
    for m in (2, 3, 5, 11, 37, 251):
        for _ in range(20):
            V = rng.getrandbits(32 * nl)
            limbs = [(V >> (32 * i)) & 0xFFFFFFFF for i in range(nl)]
            lam = O.lam(m)
            radices = [m] * lam
            if rng.random() < 0.5:
                radices[0] = m - 1
            d = O.frac_digits(limbs, radices)
            prod = 1
            for r in radices:
                prod *= r
            # the digits are the mixed-radix representation of floor(V*prod / 2^(32nl))
            top = (V * prod) >> (32 * nl)
            val = 0
            for r, di in zip(radices, d):
                assert 0 <= di < r
                val = val * r + int(di)
            assert val == top


def test_hash_output_shape_and_tweak_separation():
    rng = np.random.default_rng(1)
    for q, m in [(37, 2), (2, 37), (11, 13), (3, 5), (37, 31)]:
        A = rng.integers(0, q, size=O.lam(q))
        h1 = O.hash_label(q, m, A, 7, 100)
        h2 = O.hash_label(q, m, A, 7, 101)
        h3 = O.hash_label(q, m, A, 8, 100)
        assert len(h1) == O.lam(m) and h1.max() < m
        assert not np.array_equal(h1, h2) and not np.array_equal(h1, h3)


def test_hash_digits_roughly_uniform():
    """Chi-square sanity of the pads over Z_37 (a gross-error check only)."""
    rng = np.random.default_rng(2)
    counts = np.zeros(37)
    for tau in range(400):
        A = rng.integers(0, 11, size=O.lam(11))
        counts += np.bincount(O.hash_label(11, 37, A, 3, tau), minlength=37)
    expected = counts.sum() / 37
    chi2 = ((counts - expected) ** 2 / expected).sum()
    assert chi2 < 80  # 36 degrees of freedom; p ~ 1e-4


def test_prg_offsets_first_residue_nonzero():
    for m in PRIMES:
        for seed in range(5):
            r = O.prg_label(seed, 1, 0, m, True)
            assert r[0] < m - 1  # before the +1
            assert r.max() < m


@pytest.mark.parametrize("m", [4, 8, 16, 32, 64, 128])
def test_offsets_first_residue_is_a_unit_for_powers_of_two(m):
    """For m = 2^l the first offset residue is drawn from m/2 values and mapped
    to the odd residue 2d + 1 (a unit), so the m colours of a wire stay
    distinct (point-and-permute)."""
    seen = set()
    w3 = O.words(3)
    for seed in range(40):
        d = O.prg_label(seed, 1, 1, m, True)  # the draw behind R_m of base (3, m)
        assert d[0] < m // 2 and d.max() < m
        offs = O.garble(O.make_params([3, m], [1], 1, seed), 0, 1, with_tables=False)[0]
        R = O.pk32_unpack(m, offs[w3:w3 + O.words(m)])
        assert int(R[0]) == 2 * int(d[0]) + 1
        assert np.array_equal(R[1:], d[1:])
        seen.add(int(R[0]))
        assert sorted({(int(R[0]) * v) % m for v in range(m)}) == list(range(m))
    assert len(seen) > 1


# ----------------------------------------------------------------------------
# garbling algebra
# ----------------------------------------------------------------------------

TRACE_CASES = [
    (rns.first_primes(5), [4], 0),
    (rns.first_primes(8), [7], 1),
    (rns.first_primes(10), [8, 9], 2),
    (rns.first_primes(12), [11], 3),
    (rns.first_primes(12), [10, 11], 13),
    ([2, 3, 5, 7], [1, 2], 9),
    # power-of-two moduli and odd P (Sec. 4's bases; rounding reading)
    ([5, 7, 8], [2], 21),
    ([3, 5, 7, 16], [0], 22),
    ([3, 5, 7], [0, 1], 23),
    ([32, 167, 173], [0], 24),
]


def _lab(m, zero, R, v):
    lam = O.lam(m)
    return (zero[:lam].astype(np.int64) + int(v) * R[:lam].astype(np.int64)) % m


@pytest.mark.parametrize("base,S,seed", TRACE_CASES)
def test_every_wire_label_is_zero_plus_value_times_offset(base, S, seed):
    P = rns.cardinality(base)
    p = O.make_params(base, S, 1, seed)
    rng = random.Random(seed)
    for trial in range(3):
        a = rng.randrange(0, 1 << 20)
        x = rng.randrange(-(P // 2), P // 2)
        if trial == 0:
            x = -(P // 2)
        tr = O.trace(p, a, x)
        pt = rns.gadget_trace(base, S, x)
        gates = pt["gates"]
        # gate lists agree
        assert [(g[0], g[1], g[2], g[3]) for g in O.gate_list(p)] == \
            [(g.src, g.dst, 0 if g.kind == "sub" else 1, g.coeff) for g in gates]
        R = tr["offsets"]
        for i, m in enumerate(base):
            assert 1 <= R[i][0] < m
        for gi, gate in enumerate(gates):
            q, m = base[gate.src], base[gate.dst]
            v = pt["digit"][gi]
            # slots seen by gate gi
            for i, mi in enumerate(base):
                lam = O.lam(mi)
                assert np.array_equal(tr["ev_slots"][gi][i][:lam],
                                      _lab(mi, tr["gb_slots"][gi][i], R[i], pt["slots"][gi][i]))
            # digit wire label and projected label
            assert np.array_equal(tr["ev_in"][gi][:O.lam(q)], _lab(q, tr["gb_in"][gi], R[gate.src], v))
            assert np.array_equal(tr["ev_out"][gi][:O.lam(m)],
                                  _lab(m, tr["gb_out"][gi], R[gate.dst], v % m))
        G = len(gates)
        for i, mi in enumerate(base):
            lam = O.lam(mi)
            assert np.array_equal(tr["ev_slots"][G][i][:lam],
                                  _lab(mi, tr["gb_slots"][G][i], R[i], pt["slots"][G][i]))
        # outputs after ShiftDown carry floor((x + r)/s), r = floor(P/2) mod s
        s = rns.cardinality([base[i] for i in S])
        y = (x + rns.rounding_offset(base, S)) // s
        for i, mi in enumerate(base):
            lam = O.lam(mi)
            assert np.array_equal(tr["ev_final"][i][:lam], _lab(mi, tr["gb_final"][i], R[i], y % P % mi))


@pytest.mark.parametrize("base,S,seed", TRACE_CASES[:4] + TRACE_CASES[6:8])
def test_every_row_decrypts_for_every_input_value(base, S, seed):
    """For every gate and every v in Z_q: the row selected by the colour of
    A^0 + v R_q, plus the hash of that label, is B^0 + (v mod m) R_m, and the
    colours of the q labels are distinct (point-and-permute)."""
    p = O.make_params(base, S, 1, seed)
    a = 12345
    x = 17
    tr = O.trace(p, a, x)
    offs, zin, zout, tables = O.garble(p, a, 1)
    gates = O.gate_list(p)
    G = len(gates)
    R = tr["offsets"]
    off = 0
    for g, (src, dst, kind, coeff, phase) in enumerate(gates):
        q, m = base[src], base[dst]
        W = O.words(m)
        rows = tables[off: off + (q - 1) * W].reshape(q - 1, W)
        off += (q - 1) * W
        A0 = tr["gb_in"][g]
        B0 = tr["gb_out"][g]
        colours = set()
        for v in range(q):
            Av = _lab(q, A0, R[src], v)
            c = int(Av[0])
            colours.add(c)
            H = O.hash_label(q, m, Av, seed & 0xFFFFFFFF, a * G + g)
            row = O.pk32_unpack(m, rows[c - 1]) if c else np.zeros(O.lam(m), np.int64)
            E = (row.astype(np.int64) + H) % m
            assert np.array_equal(E, _lab(m, B0, R[dst], v % m)), (g, v)
        assert colours == set(range(q))
    assert off == len(tables)


def test_decode_all_inputs_tiny_base():
    """Every input of the 5-prime base (P = 2310), one gadget per input, s = 11."""
    base = rns.first_primes(5)
    P = 2310
    xs = np.arange(-(P // 2), P // 2, dtype=np.int64)
    p = O.make_params(base, [4], len(xs), 0)
    offs, zin, zout, tab = O.garble(p, 0, len(xs))
    X = O.encode(p, xs, zin, offs)
    Y = O.evaluate(p, 0, len(xs), X, tab)
    y, bad = O.decode(p, Y, zout, offs)
    assert bad.sum() == 0
    assert np.array_equal(y, xs // 11)
    # zero-label path: outputs equal encode(floor(x/s)) under the output zero-labels
    assert np.array_equal(Y, O.encode(p, xs // 11, zout, offs))


@pytest.mark.parametrize("base,S", [([2, 3, 5], [1, 2]), ([2, 3, 5, 7], [2, 3]), ([2, 3, 5, 7, 11], [1, 3])])
def test_decode_all_inputs_product_scaling(base, S):
    P = rns.cardinality(base)
    s = rns.cardinality([base[i] for i in S])
    xs = np.arange(-(P // 2), P // 2, dtype=np.int64)
    p = O.make_params(base, S, len(xs), 5)
    offs, zin, zout, tab = O.garble(p, 0, len(xs))
    Y = O.evaluate(p, 0, len(xs), O.encode(p, xs, zin, offs), tab)
    y, bad = O.decode(p, Y, zout, offs)
    assert bad.sum() == 0 and np.array_equal(y, xs // s)


@pytest.mark.parametrize("base,S", [([3, 4, 5], [1]), ([5, 7, 8], [2]), ([3, 5, 7], [2]), ([2, 3, 5], [0]),
                                     ([4, 5, 7, 11], [0, 2])])
def test_decode_all_inputs_rounding_reading(base, S):
    """Every input of small bases with a power-of-two modulus or odd P, one
    gadget per input: decode(eval) = floor((x + r)/s), r = floor(P/2) mod s."""
    P = rns.cardinality(base)
    s = rns.cardinality([base[i] for i in S])
    r = (P // 2) % s
    xs = np.arange(-(P // 2), P - P // 2, dtype=np.int64)
    p = O.make_params(base, S, len(xs), 7)
    offs, zin, zout, tab = O.garble(p, 0, len(xs))
    Y = O.evaluate(p, 0, len(xs), O.encode(p, xs, zin, offs), tab)
    y, bad = O.decode(p, Y, zout, offs)
    assert bad.sum() == 0 and np.array_equal(y, (xs + r) // s)


def test_decode_signed_range_odd_P():
    """Sec. 2.4 signed encoding for odd P: labels of every value of Z_P decode
    to [-floor(P/2), ceil(P/2) - 1] (P = 105: 52 stays 52, 53 becomes -52)."""
    base, S = [3, 5, 7], [2]
    P = 105
    vals = np.arange(-(P // 2), P - P // 2, dtype=np.int64)
    p = O.make_params(base, S, len(vals), 3)
    offs, zin, zout, _ = O.garble(p, 0, len(vals), with_tables=False)
    y, bad = O.decode(p, O.encode(p, vals, zout, offs), zout, offs)
    assert bad.sum() == 0 and np.array_equal(y, vals)
    assert y.max() == 52 and y.min() == -52


def test_zero_label_path_matches_full_garbling():
    base = rns.first_primes(8)
    p = O.make_params(base, [7], 64, 1)
    o1, zi1, zo1, t1 = O.garble(p, 100, 64, with_tables=True)
    o2, zi2, zo2, t2 = O.garble(p, 100, 64, with_tables=False)
    assert t2 is None
    assert np.array_equal(o1, o2) and np.array_equal(zi1, zi2) and np.array_equal(zo1, zo2)


def test_garbling_is_index_addressable():
    """Garbling a slice of gadgets gives the same labels and rows as the slice
    of a full garbling (the PRG and the tweaks depend on the gadget index)."""
    base = rns.first_primes(5)
    p = O.make_params(base, [4], 40, 7)
    o, zi, zo, tab = O.garble(p, 0, 40)
    o2, zi2, zo2, tab2 = O.garble(p, 13, 9)
    assert np.array_equal(o, o2)
    for i in range(5):
        assert np.array_equal(O.label_view(zi, p, 40, i)[:, 13:22], O.label_view(zi2, p, 9, i))
        assert np.array_equal(O.label_view(zo, p, 40, i)[:, 13:22], O.label_view(zo2, p, 9, i))
    off, off2 = 0, 0
    for (src, dst, *_rest) in O.gate_list(p):
        q, W = base[src], O.words(base[dst])
        blk = tab[off: off + 40 * (q - 1) * W].reshape(40, (q - 1) * W)
        blk2 = tab2[off2: off2 + 9 * (q - 1) * W].reshape(9, (q - 1) * W)
        assert np.array_equal(blk[13:22], blk2)
        off += 40 * (q - 1) * W
        off2 += 9 * (q - 1) * W


def test_table_size_matches_ciphertext_count():
    for base, S in [(rns.first_primes(5), [4]), (rns.first_primes(12), [11]), (rns.first_primes(10), [8, 9])]:
        p = O.make_params(base, S, 1, 0)
        a, b = rns.ciphertext_counts(base, S, row_reduction=True)
        words = sum((base[s] - 1) * O.words(base[d]) for (s, d, *_r) in O.gate_list(p))
        assert O.sizes(p, 1)["table_words"] == words
        rows = sum(base[s] - 1 for (s, d, *_r) in O.gate_list(p))
        assert rows == a + b


def test_decode_flags_corrupted_label():
    base = rns.first_primes(5)
    n = 32
    p = O.make_params(base, [4], n, 0)
    xs = np.arange(n, dtype=np.int64) - 16
    offs, zin, zout, tab = O.garble(p, 0, n)
    Y = O.evaluate(p, 0, n, O.encode(p, xs, zin, offs), tab)
    Y2 = Y.copy()
    # flip one residue of gadget 5's label for modulus 3 (m = 7): residue 2
    view = O.label_view(Y2, p, n, 3)
    res = O.pk32_unpack(7, view[:, 5].copy())
    res[2] = (res[2] + 1) % 7
    view[:, 5] = O.pk32_pack(7, res)
    y, bad = O.decode(p, Y2, zout, offs)
    assert bad.tolist() == [1 if a == 5 else 0 for a in range(n)]


def test_corrupted_row_breaks_only_its_gadget():
    base = rns.first_primes(5)
    n = 16
    p = O.make_params(base, [4], n, 4)
    xs = np.arange(n, dtype=np.int64) * 37 - 300
    offs, zin, zout, tab = O.garble(p, 0, n)
    X = O.encode(p, xs, zin, offs)
    tab2 = tab.copy()
    tab2[:] ^= 1  # every row of every gadget changed
    Y = O.evaluate(p, 0, n, X, tab2)
    _, bad = O.decode(p, Y, zout, offs)
    assert bad.sum() > 0


@pytest.mark.parametrize("moduli,S", [
    ([2, 3, 4], [2]),          # 2 and 4 not coprime
    ([3, 9, 11], [2]),         # 9: neither prime nor a power of two
    ([3, 5, 6], [2]),          # 6: neither prime nor a power of two
    ([4, 8, 11], [2]),         # two powers of two
    ([3, 2, 5], [2]),          # not ascending
    ([2, 3, 5], [1, 1]),       # scale set not strictly ascending
    ([2, 3, 5], [0, 1, 2]),    # t = k
    ([2], [0]),                # k < 2
    ([2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37, 41, 241, 251], [14]),  # P >= 2^63
])
def test_bad_params_rejected(moduli, S):
    p = O.make_params(moduli, S, 1, 0)
    assert O.check_params(p) == -1
