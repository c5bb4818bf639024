"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point that include/redash.h declares, validates parameters like
the oracle does, and reports the same buffer sizes as the oracle's layouts."""

from __future__ import annotations

import ctypes

import pytest

from oracle import oracle as O
from oracle import rns
from paper_2506_14489_amd import binding as B
from paper_2506_14489_amd import workloads as WL


def test_library_exports_every_declared_symbol():
    names = B.declared_symbols()
    assert set(names) == {"redash_plan", "redash_garble_scale", "redash_garble_scale_given", "redash_encode", "redash_eval_scale",
                          "redash_eval_scale_noalloc", "redash_decode", "redash_hash_labels", "redash_aes_ctr", "redash_aes_ctr_bitsliced", "redash_strerror", "redash_linear_plan",
                          "redash_linear_prepare", "redash_linear_eval", "redash_linear_garble"}
    L = B.lib()
    for n in names:
        assert hasattr(L, n), n
        assert ctypes.cast(getattr(L, n), ctypes.c_void_p).value


def test_params_struct_layout_matches_header():
    # k, moduli[16], t, scale_idx[16] (4-byte) then n, seed, a0 (8-byte)
    assert ctypes.sizeof(B.Params) == 4 * 34 + 8 * 3
    assert B.Params.n.offset == 136 and B.Params.a0.offset == 152
    # label_words, table_words (8-byte), offset_words, gates (4-byte), work_words (8-byte)
    assert ctypes.sizeof(B.Sizes) == 32
    assert B.Sizes.work_words.offset == 24


def test_strerror_texts():
    assert B.strerror(0) == "ok"
    for code in (-1, -2, -3, -4, -5):
        assert B.strerror(code) != "unknown error"
    assert B.strerror(42) == "unknown error"


PLAN_CASES = [(w.moduli, w.scale_idx) for w in WL.CONFIGS] + [
    (tuple(WL.PRIMES_12), (10, 11)), (tuple(WL.PRIMES_12), (9,)), ((2, 3), (1,)), ((2, 3, 5), (1, 2)),
    (tuple(rns.first_primes(15)), (13, 14)), (tuple(rns.first_primes(15)), (1, 5, 9)), ((2, 97, 251), (2,)),
    ((2, 3, 5, 7, 11, 13), (1, 2, 3, 4, 5)),
] + [(w.moduli, w.scale_idx) for w in WL.SHORT_BASES] + [
    # odd P, and every power of two up to 128 (m = 4 and 16 fill their words)
    ((3, 5, 7), (1,)), ((3, 5, 7, 11, 13), (0, 4)), ((3, 4, 5), (1,)), ((3, 5, 16), (2,)),
    ((5, 7, 64), (0,)), ((3, 128, 251), (1,)), ((4, 5, 7), (0, 2)),
]


@pytest.mark.parametrize("moduli,S", PLAN_CASES)
@pytest.mark.parametrize("n", [0, 1, 1000])
def test_plan_sizes_match_oracle(moduli, S, n):
    sz = B.redash_plan(B.make_params(moduli, S, n, 0))
    osz = O.sizes(O.make_params(list(moduli), list(S), n, 0), n)
    assert sz["label_words"] == osz["label_words"]
    assert sz["table_words"] == osz["table_words"]
    assert sz["offset_words"] == osz["offset_words"]
    assert sz["gates"] == osz["gates"]
    k, t = len(moduli), len(S)
    assert sz["gates"] == k * (k - 1) // 2 + t * (k - t)


@pytest.mark.parametrize("moduli,S", PLAN_CASES)
def test_work_words(moduli, S):
    """The evaluator's working storage holds the Phase-B copies of the
    remaining moduli after the first one (R[0] is only ever a digit)."""
    n = 777
    R = [i for i in range(len(moduli)) if i not in S]
    sz = B.redash_plan(B.make_params(moduli, S, n, 0))
    assert sz["work_words"] == n * sum(O.words(moduli[i]) for i in R[1:])


def test_plan_cache_follows_the_params():
    """The library keeps the last plan per host thread: calls that alternate
    between parameters, invalid ones among them, still get each one's own
    sizes or error."""
    cases = [(PLAN_CASES[i][0], PLAN_CASES[i][1], n) for i, n in ((0, 5), (3, 7), (0, 6), (5, 1000))]
    want = [O.sizes(O.make_params(list(m), list(S), n, 0), n) for m, S, n in cases]
    bad = B.make_params((2, 3, 6), (1,), 10, 0)  # 6 is not a prime or a power of two
    for _ in range(3):
        for (m, S, n), osz in zip(cases, want):
            sz = B.redash_plan(B.make_params(m, S, n, 0))
            assert (sz["label_words"], sz["table_words"]) == (osz["label_words"], osz["table_words"])
            with pytest.raises(RuntimeError):
                B.redash_plan(bad)
    # the same parameters again after a change in an unused entry
    p = B.make_params(PLAN_CASES[0][0], PLAN_CASES[0][1], 5, 0)
    a = B.redash_plan(p)
    p.moduli[15] = 12345
    assert B.redash_plan(p) == a


def test_plan_cache_per_thread():
    """Host threads calling with different parameters at once each get their
    own sizes (the cached plan is per thread)."""
    import threading

    cases = [(m, S, 100 + i) for i, (m, S) in enumerate(PLAN_CASES[:6])]
    want = {c: O.sizes(O.make_params(list(c[0]), list(c[1]), c[2], 0), c[2])["table_words"] for c in cases}
    errors = []

    def run(c):
        p = B.make_params(c[0], c[1], c[2], 0)
        for _ in range(2000):
            if B.redash_plan(p)["table_words"] != want[c]:
                errors.append(c)
                return

    threads = [threading.Thread(target=run, args=(c,)) for c in cases]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors


@pytest.mark.parametrize("m", rns.first_primes(12) + [97, 107, 167, 173, 251, 4, 8, 16, 32, 64, 128])
def test_label_words_match_oracle(m):
    assert B.label_words_of(m) == O.words(m)


BAD = [
    ([3, 9, 11], [2]),
    ([3, 5, 6], [2]),
    ([4, 8, 11], [2]),
    ([2, 3, 4], [2]),
    ([3, 2, 5], [2]),
    ([2, 3, 5], [1, 1]),
    ([2, 3, 5], [0, 1, 2]),
    ([2], [0]),
    ([2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37, 41, 241, 251], [14]),
    ([2, 3, 257], [2]),
    ([2, 3, 5], [3]),
    ([2, 3, 5], []),
    ([3, 5, 6], [0]),
    ([2, 3, 32], [2]),
    ([3, 16, 64], [0]),
    ([9, 11, 13], [0]),
    ([3, 5, 256], [0]),
    (list(rns.first_primes(16)), [15]),
]


@pytest.mark.parametrize("moduli,S", BAD)
def test_bad_params_rejected_like_the_oracle(moduli, S):
    bp = B.make_params(moduli[:16], S, 1, 0)
    assert B.plan_rc(bp) == B.REDASH_E_PARAM
    if len(moduli) <= 16:
        assert O.check_params(O.make_params(moduli, S, 1, 0)) == -1


def test_random_params_accepted_and_sized_like_the_oracle():
    """600 seeded random parameter sets, valid and not (any integer 0..300 as a
    modulus, unsorted or repeated moduli, several even moduli, scaling indices
    out of range, repeated or unsorted, t = 0 or k, k up to 16): the library
    accepts exactly those the oracle accepts, and sizes those the same way."""
    import numpy as np

    rng = np.random.default_rng(515)
    accepted = 0
    for _ in range(600):
        k = int(rng.integers(1, 17))
        if rng.random() < 0.5:
            pool = [m for m in range(2, 256) if rns.is_prime(m) or (m & (m - 1)) == 0]
            moduli = sorted(int(m) for m in rng.choice(pool, size=k, replace=False))
        else:
            moduli = [int(m) for m in rng.integers(0, 301, size=k)]
        t = int(rng.integers(0, k + 1))
        if rng.random() < 0.7:
            S = sorted(int(i) for i in rng.choice(k, size=t, replace=False))
        else:
            S = [int(i) for i in rng.integers(0, k + 2, size=t)]
        n = int(rng.integers(0, 5000))
        ok_lib = B.plan_rc(B.make_params(moduli, S, n, 0)) == 0
        if k > 15:  # the oracle's struct holds at most 16; the library takes at most 15
            assert not ok_lib
            continue
        ok_orc = O.check_params(O.make_params(moduli, S, n, 0)) == 0
        assert ok_lib == ok_orc, (moduli, S)
        if ok_lib:
            accepted += 1
            sz = B.redash_plan(B.make_params(moduli, S, n, 0))
            osz = O.sizes(O.make_params(list(moduli), list(S), n, 0), n)
            assert (sz["label_words"], sz["table_words"], sz["gates"]) == (
                osz["label_words"], osz["table_words"], osz["gates"])
    assert accepted > 50  # 71 with this seed


def test_null_params():
    L = B.lib()
    s = B.Sizes()
    assert L.redash_plan(None, ctypes.byref(s)) == B.REDASH_E_NULL
    assert L.redash_plan(ctypes.byref(B.make_params([2, 3], [1], 1, 0)), None) == B.REDASH_E_NULL


def test_valid_extremes_accepted():
    # largest k, P just below 2^63 is rejected above; first 15 primes are accepted
    assert B.plan_rc(B.make_params(rns.first_primes(15), [14], 1, 0)) == 0
    assert B.plan_rc(B.make_params([2, 251], [1], 1, 0)) == 0


def test_batched_table_footprint():
    """64 GB of garbled rows for the 16x64x56x56 map (fits one 288 GB GPU)."""
    w = WL.BATCHED
    sz = B.redash_plan(B.make_params(w.moduli, w.scale_idx, w.n, w.seed))
    assert sz["table_words"] * 4 == 19932 * w.n
    assert sz["label_words"] * 4 == 252 * w.n


def test_entry_points_validate_before_any_device_work():
    """Invalid parameters and NULL buffers are rejected on the host, before
    any HIP call, so this runs without a GPU."""
    L = B.lib()
    bad = B.make_params([3, 9, 11], [2], 4, 0)  # 9 is neither prime nor a power of two
    good = B.make_params(WL.TINY.moduli, WL.TINY.scale_idx, 4, 0)
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: every call below returns early
    assert L.redash_eval_scale(ctypes.byref(bad), fake, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_garble_scale(ctypes.byref(bad), fake, fake, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_encode(ctypes.byref(bad), fake, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_decode(ctypes.byref(bad), fake, fake, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_eval_scale(ctypes.byref(good), None, fake, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_eval_scale(ctypes.byref(good), fake, None, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_eval_scale(ctypes.byref(good), fake, fake, None, fake, None) == B.REDASH_E_NULL
    assert L.redash_eval_scale(ctypes.byref(good), fake, fake, fake, None, None) == B.REDASH_E_NULL
    huge = B.make_params(WL.TINY.moduli, WL.TINY.scale_idx, 1 << 30, 0)
    assert L.redash_eval_scale(ctypes.byref(huge), fake, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_garble_scale(ctypes.byref(good), None, fake, fake, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_garble_scale(ctypes.byref(good), fake, fake, fake, None, fake, None) == B.REDASH_E_NULL
    assert L.redash_garble_scale(ctypes.byref(good), fake, fake, fake, fake, None, None) == B.REDASH_E_NULL
    assert L.redash_garble_scale(ctypes.byref(huge), fake, fake, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_garble_scale_given(ctypes.byref(bad), fake, fake, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_garble_scale_given(ctypes.byref(good), None, fake, fake, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_garble_scale_given(ctypes.byref(good), fake, None, fake, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_garble_scale_given(ctypes.byref(good), fake, fake, fake, None, fake, None) == B.REDASH_E_NULL
    assert L.redash_garble_scale_given(ctypes.byref(huge), fake, fake, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_encode(ctypes.byref(good), None, fake, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_decode(ctypes.byref(good), fake, fake, fake, fake, None, None) == B.REDASH_E_NULL
    assert L.redash_hash_labels(6, 3, 1, fake, 0, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_hash_labels(3, 9, 1, fake, 0, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_hash_labels(3, 256, 1, fake, 0, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_hash_labels(3, 5, 1, None, 0, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_eval_scale(None, fake, fake, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_eval_scale_noalloc(ctypes.byref(bad), fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_eval_scale_noalloc(ctypes.byref(huge), fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_eval_scale_noalloc(ctypes.byref(good), None, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_eval_scale_noalloc(ctypes.byref(good), fake, None, fake, None) == B.REDASH_E_NULL
    assert L.redash_eval_scale_noalloc(ctypes.byref(good), fake, fake, None, None) == B.REDASH_E_NULL
    assert L.redash_eval_scale_noalloc(None, fake, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_aes_ctr(0, 0, None, None) == B.REDASH_OK
    assert L.redash_aes_ctr(5, 0, None, None) == B.REDASH_E_NULL
    assert L.redash_aes_ctr((1 << 40) + 1, 0, fake, None) == B.REDASH_E_PARAM
    assert L.redash_aes_ctr_bitsliced(0, 0, None, None) == B.REDASH_OK
    assert L.redash_aes_ctr_bitsliced(5, 0, None, None) == B.REDASH_E_NULL
    assert L.redash_aes_ctr_bitsliced((1 << 40) + 1, 0, fake, None) == B.REDASH_E_PARAM


def test_noalloc_size_limit():
    """The allocation-free evaluator takes calls whose working storage fits
    its fixed buffer and rejects larger ones on the host, before any HIP call
    (54 working words per gadget on the 12-prime base: at most 310,689)."""
    L = B.lib()
    w = WL.BATCHED
    per = B.redash_plan(B.make_params(w.moduli, w.scale_idx, 1, w.seed))["work_words"]
    assert per == 54
    n_max = B.NOALLOC_WORK_WORDS // per
    assert n_max == 310689
    fits = B.make_params(w.moduli, w.scale_idx, n_max, w.seed)
    over = B.make_params(w.moduli, w.scale_idx, n_max + 1, w.seed)
    fake = ctypes.c_void_p(0x1000)  # never dereferenced
    assert L.redash_eval_scale_noalloc(ctypes.byref(over), fake, fake, fake, None) == B.REDASH_E_SIZE
    # within the limit the call gets as far as its pointer checks
    assert L.redash_eval_scale_noalloc(ctypes.byref(fits), None, fake, fake, None) == B.REDASH_E_NULL
    # a base without working storage (one remaining modulus) has no limit below 2^30
    two = B.make_params([2, 3], [1], (1 << 30) - 1, 0)
    assert B.redash_plan(two)["work_words"] == 0
    assert L.redash_eval_scale_noalloc(ctypes.byref(two), None, fake, fake, None) == B.REDASH_E_NULL


# ---------------------------------------------------------------------------
# garbled linear layers
# ---------------------------------------------------------------------------

def test_linear_structs_match_header():
    # k, moduli[16], batch, c_in, h_in, w_in, c_out, kh, kw, stride, pad: 26 uint32
    assert ctypes.sizeof(B.LinearParams) == 4 * 26
    # in/out label words, prepared and work bytes (8-byte), h_out, w_out, offset_words (4-byte), padded to 8
    assert ctypes.sizeof(B.LinearSizes) == 48
    assert B.LinearSizes.h_out.offset == 32


LINEAR_CASES = [
    # moduli, batch, c_in, h, w, c_out, kh, kw, stride, pad
    (WL.PRIMES_12, 16, 64, 56, 56, 64, 3, 3, 1, 1),
    (WL.PRIMES_12, 1, 3, 224, 224, 64, 7, 7, 2, 3),
    (WL.PRIMES_12, 1, 64, 56, 56, 128, 1, 1, 2, 0),
    (WL.PRIMES_12, 1, 512, 1, 1, 1000, 1, 1, 1, 0),
    ((32, 167, 173), 7, 10, 5, 6, 3, 2, 3, 1, 1),
    ((2, 3, 5), 1, 1, 1, 1, 1, 1, 1, 1, 0),
]


@pytest.mark.parametrize("case", LINEAR_CASES)
def test_linear_plan_sizes(case):
    from oracle import linear as OL

    moduli, n, c_in, h, w, c_out, kh, kw, stride, pad = case
    sz = B.redash_linear_plan(B.make_linear_params(moduli, n, c_in, h, w, c_out, kh, kw, stride, pad))
    W = sum(OL.label_words(m) for m in moduli)
    _, _, ho, wo = OL.conv_out_shape(n, c_in, h, w, c_out, kh, kw, stride, pad)
    assert (sz["h_out"], sz["w_out"]) == (ho, wo)
    assert sz["in_label_words"] == n * c_in * h * w * W
    assert sz["out_label_words"] == n * c_out * ho * wo * W
    assert sz["offset_words"] == W
    assert sz["prepared_bytes"] >= len(moduli) * c_out * c_in * kh * kw
    # residue planes of one byte per (zero-padded) input position and
    # channel: one residue per byte, or f = 8 / bp residues of bp bits for
    # m <= 16 (bp = 1, 2, 4), grouped within each packed word
    def planes(m):
        b = (m - 1).bit_length()
        lam, g = OL.label_lambda(m), 32 // b
        W = -(-lam // g)
        bp = 1 if b == 1 else 2 if b == 2 else 4 if b <= 4 else 8
        f = 8 // bp
        return (W - 1) * -(-g // f) + -(-(lam - (W - 1) * g) // f)

    assert sz["work_bytes"] >= sum(planes(m) for m in moduli) * n * c_in * h * w


def test_linear_work_of_the_batched_layer():
    """The 3x3 64 -> 64 layer of the batched map over the first 12 primes:
    295 residue planes (16 + 21 + 28 + 23 + 19 + 18 for 2..13, packed 8, 4 and
    2 per byte; 32 + 31 + 29 + 27 + 26 + 25 for 17..37, one per byte) of the
    zero-padded 16 x 58 x 58 input, 64 channel bytes per position."""
    sz = B.redash_linear_plan(B.make_linear_params((2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37), 16, 64, 56, 56,
                                                   64, 3, 3, 1, 1))
    assert sz["work_bytes"] == 295 * 16 * 58 * 58 * 64


LINEAR_BAD = [
    ((2, 3, 6), 1, 4, 4, 4, 2, 3, 3, 1, 1),        # 6 is not a prime or a power of two
    ((2, 3, 4), 1, 4, 4, 4, 2, 3, 3, 1, 1),        # 2 and 4 not coprime
    ((3, 2), 1, 4, 4, 4, 2, 3, 3, 1, 1),           # not ascending
    ((2, 3), 0, 4, 4, 4, 2, 3, 3, 1, 1),           # empty batch
    ((2, 3), 1, 0, 4, 4, 2, 3, 3, 1, 1),
    ((2, 3), 1, 4, 4, 4, 0, 3, 3, 1, 1),
    ((2, 3), 1, 4, 4, 4, 2, 3, 3, 0, 1),           # stride 0
    ((2, 3), 1, 4, 4, 4, 2, 3, 3, 1, 3),           # pad >= kernel
    ((2, 3), 1, 4, 2, 2, 2, 5, 5, 1, 1),           # kernel larger than the padded input
    ((2, 3), 1, 4, 20, 20, 2, 9, 9, 1, 1),         # more than 64 taps
    ((2, 3), 1, 4096, 4, 4, 2, 3, 3, 1, 1),        # c_in kh kw > 32768
    ((2, 3, 251), 1, 16385, 1, 1, 2, 1, 1, 1, 0),  # c_in kh kw = 16385, one above the limit
    ((2, 3), 1, 1821, 4, 4, 2, 3, 3, 1, 1),        # 1821 * 9 = 16389
    ((2, 3), 1024, 64, 128, 128, 2, 1, 1, 1, 0),   # 2^30 input activations
]


LINEAR_LIMIT_OK = [
    ((2, 3, 251), 1, 16384, 1, 1, 2, 1, 1, 1, 0),  # c_in kh kw = 16384, the documented limit
    ((2, 3, 251), 1, 1024, 4, 4, 2, 4, 4, 1, 1),   # 1024 * 16 = 16384 with a 4x4 kernel
    ((251,), 1, 2048, 3, 3, 2, 2, 4, 1, 1),        # 2048 * 8 = 16384, largest modulus alone
]


@pytest.mark.parametrize("case", LINEAR_LIMIT_OK)
def test_linear_reduction_length_limit_accepted(case):
    assert B.linear_plan_rc(B.make_linear_params(*case)) == 0


@pytest.mark.parametrize("case", LINEAR_BAD)
def test_linear_bad_params_rejected(case):
    assert B.linear_plan_rc(B.make_linear_params(*case)) == B.REDASH_E_PARAM


def test_linear_entry_points_validate_before_any_device_work():
    L = B.lib()
    fake = ctypes.c_void_p(4096)
    bad = B.make_linear_params((2, 3, 6), 1, 4, 4, 4, 2, 3, 3, 1, 1)
    good = B.make_linear_params((2, 3, 5), 1, 4, 4, 4, 2, 3, 3, 1, 1)
    assert L.redash_linear_plan(None, ctypes.byref(B.LinearSizes())) == B.REDASH_E_NULL
    assert L.redash_linear_prepare(ctypes.byref(bad), fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_linear_eval(ctypes.byref(bad), fake, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_linear_garble(ctypes.byref(bad), fake, fake, None, fake, fake, fake, None) == B.REDASH_E_PARAM
    assert L.redash_linear_prepare(ctypes.byref(good), None, fake, None) == B.REDASH_E_NULL
    assert L.redash_linear_eval(ctypes.byref(good), fake, None, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_linear_eval(ctypes.byref(good), fake, fake, None, fake, None) == B.REDASH_E_NULL
    assert L.redash_linear_eval(ctypes.byref(good), fake, fake, fake, None, None) == B.REDASH_E_NULL
    assert L.redash_linear_garble(ctypes.byref(good), fake, fake, None, None, fake, fake, None) == B.REDASH_E_NULL
    assert L.redash_linear_garble(ctypes.byref(good), fake, fake, None, fake, None, fake, None) == B.REDASH_E_NULL
