"""GPU parity of the HIP library against the CPU oracle (bit-exact).

Small cases: every word of every output is compared with the oracle, at sizes
that span several 256-thread blocks and end in a ragged tail.  Full-size
workloads (the batched conv map and the ResNet-18 layers) run in the launch
configuration the benchmark times; there every gadget is checked through
decode = floor(x/s) with all labels valid, and a seeded sample of gadgets is
compared word by word with the oracle garbling that one gadget.
"""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import linear as OL  # noqa: E402
from oracle import oracle as O  # noqa: E402
from oracle import rns  # noqa: E402
from paper_2506_14489_amd import binding as B  # noqa: E402
from paper_2506_14489_amd import workloads as WL  # noqa: E402

import gpu_helpers as H  # noqa: E402

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU containers
    pytest.skip("needs a GPU", allow_module_level=True)


def _floor_div(x: np.ndarray, s: int) -> np.ndarray:
    return np.floor_divide(x, s)


def _scaled(x: np.ndarray, moduli, S) -> np.ndarray:
    """What the gadget returns: floor((x + r)/s), r = floor(P/2) mod s
    (0, i.e. floor(x/s), whenever P/(2s) is an integer; the value-level
    oracle's reading of the shift constants of Sec. 3.4)."""
    s = rns.cardinality([moduli[i] for i in S])
    return np.floor_divide(x + rns.rounding_offset(list(moduli), list(S)), s)


def _params_pair(moduli, S, n, seed, a0=0):
    return B.make_params(moduli, S, n, seed, a0), O.make_params(moduli, S, n, seed)


# ---------------------------------------------------------------------------
# hash
# ---------------------------------------------------------------------------

HASH_PAIRS = [(2, 3), (3, 2), (37, 2), (2, 37), (11, 13), (5, 3), (37, 31), (17, 19), (97, 251), (251, 97),
              (3, 5), (7, 37),
              # power-of-two moduli (Sec. 4 bases), including 4 and 16 whose fields fill a word
              (32, 167), (167, 32), (173, 32), (32, 97), (4, 3), (3, 4), (16, 5), (5, 16), (2, 64), (128, 7),
              (8, 19), (251, 8),
              # generic-path and large fast-path moduli
              (41, 197), (241, 59), (61, 47), (53, 211)]


# every modulus the library accepts as the hash's output modulus (its pad's
# digit extraction), each with a seeded random input modulus
_ACCEPTED = [m for m in range(2, 256) if rns.is_prime(m) or (m & (m - 1)) == 0]
HASH_EVERY_M = [(int(q), m) for q, m in zip(np.random.default_rng(99).choice(_ACCEPTED, size=len(_ACCEPTED)),
                                             _ACCEPTED)]


@pytest.mark.parametrize("q,m", HASH_PAIRS + HASH_EVERY_M)
def test_hash_matches_oracle(q, m):
    count = 300
    rng = np.random.default_rng(q * 1000 + m)
    lam_q = O.lam(q)
    res = rng.integers(0, q, size=(count, lam_q)).astype(np.uint32)
    words = np.stack([O.pk32_pack(q, r) for r in res])            # count x W_q
    tau = rng.integers(0, 2 ** 62, size=count, dtype=np.int64)
    gid = int(rng.integers(0, 2 ** 32))
    Wq, Wm = B.label_words_of(q), B.label_words_of(m)
    lab = H.to_dev(np.ascontiguousarray(words.T.reshape(-1)))     # SoA
    out = torch.empty(Wm * count, dtype=torch.int32, device="cuda")
    B.redash_hash_labels(q, m, count, lab, gid, H.to_dev(tau), out)
    got = H.to_u32(out).reshape(Wm, count).T
    for a in range(count):
        exp = O.pk32_pack(m, O.hash_label(q, m, res[a], gid, int(tau[a])))
        assert np.array_equal(got[a], exp), (q, m, a)
    assert Wq == len(words[0])


def test_hash_known_answers():
    """The library's hash against the known-answer file (written from the
    oracle and checked against libcrypto on the CPU)."""
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hash_kat.txt")
    groups = {}
    with open(path) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            q, m, gid, tau, a, h = line.split()
            groups.setdefault((int(q), int(m), int(gid, 16)), []).append(
                (int(tau), [int(v, 16) for v in a.split(",")], [int(v, 16) for v in h.split(",")]))
    done = 0
    for (q, m, gid), rows in groups.items():
        count = len(rows)
        words = np.array([r[1] for r in rows], dtype=np.uint32)          # count x W_q
        tau = np.array([r[0] for r in rows], dtype=np.uint64).view(np.int64)
        Wm = B.label_words_of(m)
        out = torch.empty(Wm * count, dtype=torch.int32, device="cuda")
        B.redash_hash_labels(q, m, count, H.to_dev(np.ascontiguousarray(words.T.reshape(-1))), gid,
                             H.to_dev(tau), out)
        got = H.to_u32(out).reshape(Wm, count).T
        for j, r in enumerate(rows):
            assert [int(v) for v in got[j]] == r[2], (q, m, gid, r[0])
            done += 1
    assert done >= 100


@pytest.mark.parametrize("bitsliced", [False, True])
def test_aes_ctr_matches_oracle(bitsliced):
    """The bare AES kernels (counter mode under the hash key; round tables,
    and bitsliced) against the oracle's FIPS-197 AES, including ragged tails
    and a counter that carries into bit 64."""
    key = bytes(range(16))
    run = B.redash_aes_ctr_bitsliced if bitsliced else B.redash_aes_ctr
    for count, c0 in ((1000, 0), (4099, 2 ** 64 - 2050), (7, 12345), (70000, 2 ** 63 + 5)):
        out = torch.empty(4 * count, dtype=torch.int32, device="cuda")
        run(count, c0, out)
        got = H.to_u32(out).reshape(count, 4)
        for i in list(range(min(count, 300))) + list(range(max(count - 300, 0), count)):
            block = ((c0 + i) % 2 ** 128).to_bytes(16, "little")
            want = np.frombuffer(O.aes128(key, block), dtype="<u4")
            assert np.array_equal(got[i], want), (count, c0, i)


# ---------------------------------------------------------------------------
# small cases: garble, encode, eval, decode, word for word
# ---------------------------------------------------------------------------

SMALL = [
    # name, moduli, S, n, seed, a0
    ("tiny", WL.TINY.moduli, WL.TINY.scale_idx, 1024, 0, 0),
    ("tiny-ragged", WL.TINY.moduli, WL.TINY.scale_idx, 777, 0, 0),
    ("dense", WL.DENSE.moduli, WL.DENSE.scale_idx, 4096, 1, 0),
    ("conv-tail", WL.CONV.moduli, WL.CONV.scale_idx, 600, 2, 65536 - 600),
    ("batched-head", WL.BATCHED.moduli, WL.BATCHED.scale_idx, 300, 3, 0),
    ("resnet-1147", tuple(WL.PRIMES_12), (10, 11), 260, 11, 1000),
    ("k15-product", tuple(rns.first_primes(15)), (13, 14), 300, 77, 5),
    ("base-235-by-15", (2, 3, 5), (1, 2), 30, 5, 0),
    ("base-2357-by-35", (2, 3, 5, 7), (2, 3), 210, 6, 0),
    ("k2", (2, 3), (1,), 6, 9, 0),
    ("large-moduli", (2, 97, 251), (2,), 300, 12, 3),
    # the short and power-of-two bases of Sec. 4 (P/(2s) not an integer)
    ("cpm8-8", WL.CPM8_8.moduli, WL.CPM8_8.scale_idx, 700, 40, 0),
    ("cpm8-32", WL.CPM8_32.moduli, WL.CPM8_32.scale_idx, 600, 41, 100),
    ("short-f", WL.SHORT_F.moduli, WL.SHORT_F.scale_idx, 1000, 42, 0),
    ("short-F", WL.SHORT_BIG_F.moduli, WL.SHORT_BIG_F.scale_idx, 1000, 43, 5),
    ("odd-P", (3, 5, 7, 11, 13), (0, 4), 500, 50, 0),
    ("pow2-4-scaled", (3, 4, 5), (1,), 300, 51, 0),
    ("pow2-4-remaining", (4, 5, 7), (1,), 300, 52, 7),
    ("pow2-16", (3, 5, 7, 11, 16), (4,), 400, 53, 0),
    ("pow2-64", (5, 7, 64, 67), (2,), 400, 54, 0),
    ("pow2-128-product", (3, 128, 251), (0, 1), 400, 55, 0),
    # moduli on the evaluator's generic path (41, 47, 53, 59, 61) and large
    # primes on its fast path (197 to 251)
    ("generic-41-61", (2, 41, 61), (2,), 300, 56, 0),
    ("generic-47-53-59", (2, 47, 53, 59), (1, 3), 300, 57, 11),
    ("fast-197-241", (3, 197, 241), (1,), 300, 58, 0),
    ("fast-199-211-251", (2, 199, 211, 251), (3,), 300, 59, 4),
]


def _random_bases(count: int, seed: int):
    """Seeded random bases the library accepts: k from 2 to 15 moduli drawn
    from the primes and powers of two up to 255 (at most one of them even),
    P < 2^63, a random non-empty proper scaling set."""
    rng = np.random.default_rng(seed)
    accepted = [m for m in range(2, 256) if rns.is_prime(m) or (m & (m - 1)) == 0]
    out = []
    while len(out) < count:
        k = int(rng.integers(2, 16))
        base = sorted(int(m) for m in rng.choice(accepted, size=k, replace=False))
        if sum(1 for m in base if m % 2 == 0) > 1 or rns.cardinality(base) >= 2 ** 63:
            continue
        t = int(rng.integers(1, k))
        S = tuple(sorted(int(i) for i in rng.choice(k, size=t, replace=False)))
        n = int(rng.integers(1, 400))
        out.append((f"rand{len(out)}-k{k}-t{t}", tuple(base), S, n, 900 + len(out), int(rng.integers(0, 1 << 20))))
    return out


RANDOM_BASES = _random_bases(24, 2026)


@pytest.mark.parametrize("case", RANDOM_BASES, ids=[c[0] for c in RANDOM_BASES])
def test_random_bases_match_oracle(case):
    """Garbled tables, offsets and zero-labels, and the evaluator's output
    labels on the oracle's tables, word for word on seeded random bases;
    every output decodes to the scaled value."""
    name, moduli, S, n, seed, a0 = case
    print(f"random base {name}: moduli={moduli} S={S} n={n} a0={a0}", flush=True)
    bp, op = _params_pair(moduli, S, n, seed, a0)
    offs, zin, zout, tab = O.garble(op, a0, n)
    buf = B.Buffers(bp)
    B.redash_garble_scale(bp, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work)
    torch.cuda.synchronize()
    assert np.array_equal(H.to_u32(buf.offsets), offs)
    assert np.array_equal(H.to_u32(buf.in_zero), zin)
    assert np.array_equal(H.to_u32(buf.out_zero), zout)
    assert np.array_equal(H.to_u32(buf.tables)[: len(tab)], tab)
    x = _small_inputs(moduli, n, seed)
    X = O.encode(op, x, zin, offs)
    Y = O.evaluate(op, a0, n, X, tab)
    out = torch.empty(len(X), dtype=torch.int32, device="cuda")
    work = torch.empty(max(B.redash_plan(bp)["work_words"], 1), dtype=torch.int32, device="cuda")
    B.redash_eval_scale(bp, H.to_dev(X), H.to_dev(tab), out, work)
    torch.cuda.synchronize()
    got = H.to_u32(out)
    assert np.array_equal(got, Y)
    y, bad = O.decode(op, got, zout, offs)
    assert bad.sum() == 0 and np.array_equal(y, _scaled(x, moduli, S))


def _small_inputs(moduli, n, seed):
    P = rns.cardinality(moduli)
    rng = np.random.default_rng(seed + 1000)
    lo, hi = -(P // 2), P - P // 2  # the signed range [-floor(P/2), ceil(P/2) - 1]
    x = rng.integers(lo, hi, size=n, dtype=np.int64)
    if n >= 2:
        x[0], x[1] = lo, hi - 1  # both ends of the signed range
    return x


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_garble_matches_oracle(case):
    name, moduli, S, n, seed, a0 = case
    bp, op = _params_pair(moduli, S, n, seed, a0)
    buf = B.Buffers(bp)
    B.redash_garble_scale(bp, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work)
    torch.cuda.synchronize()
    offs, zin, zout, tab = O.garble(op, a0, n)
    assert np.array_equal(H.to_u32(buf.offsets), offs)
    assert np.array_equal(H.to_u32(buf.in_zero), zin)
    assert np.array_equal(H.to_u32(buf.out_zero), zout)
    assert np.array_equal(H.to_u32(buf.tables)[: len(tab)], tab)


@pytest.mark.parametrize("case", SMALL + RANDOM_BASES, ids=[c[0] for c in SMALL + RANDOM_BASES])
def test_garble_on_given_zero_labels_matches_oracle(case):
    """redash_garble_scale_given on arbitrary valid zero-labels (as a free
    operation would leave them) against the oracle, word for word; the
    given labels are left untouched."""
    name, moduli, S, n, seed, a0 = case
    bp, op = _params_pair(moduli, S, n, seed, a0)
    rng = np.random.default_rng(seed + 500)
    zin = OL.pack(moduli, [rng.integers(0, m, size=(n, O.lam(m))) for m in moduli], n)
    buf = B.Buffers(bp)
    zd = H.to_dev(zin)
    B.redash_garble_scale_given(bp, buf.offsets, zd, buf.out_zero, buf.tables, buf.work)
    torch.cuda.synchronize()
    offs, zout, tab = O.garble_given(op, a0, n, zin)
    assert np.array_equal(H.to_u32(buf.offsets), offs)
    assert np.array_equal(H.to_u32(buf.out_zero), zout)
    assert np.array_equal(H.to_u32(buf.tables)[: len(tab)], tab)
    assert np.array_equal(H.to_u32(zd), zin)


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_eval_on_oracle_tables_matches_oracle(case):
    name, moduli, S, n, seed, a0 = case
    bp, op = _params_pair(moduli, S, n, seed, a0)
    offs, zin, zout, tab = O.garble(op, a0, n)
    x = _small_inputs(moduli, n, seed)
    X = O.encode(op, x, zin, offs)
    Y = O.evaluate(op, a0, n, X, tab)
    out = torch.empty(len(X), dtype=torch.int32, device="cuda")
    work = torch.empty(max(B.redash_plan(bp)["work_words"], 1), dtype=torch.int32, device="cuda")
    B.redash_eval_scale(bp, H.to_dev(X), H.to_dev(tab), out, work)
    torch.cuda.synchronize()
    got = H.to_u32(out)
    assert np.array_equal(got, Y)
    y, bad = O.decode(op, got, zout, offs)
    assert bad.sum() == 0 and np.array_equal(y, _scaled(x, moduli, S))


@pytest.mark.parametrize("case", SMALL + RANDOM_BASES, ids=[c[0] for c in SMALL + RANDOM_BASES])
def test_encode_and_decode_match_oracle(case):
    name, moduli, S, n, seed, a0 = case
    bp, op = _params_pair(moduli, S, n, seed, a0)
    offs, zin, zout, _ = O.garble(op, a0, n, with_tables=False)
    x = _small_inputs(moduli, n, seed)
    lab = torch.empty(len(zin), dtype=torch.int32, device="cuda")
    B.redash_encode(bp, H.to_dev(x), H.to_dev(zin), H.to_dev(offs), lab)
    torch.cuda.synchronize()
    X = O.encode(op, x, zin, offs)
    assert np.array_equal(H.to_u32(lab), X)
    # decode: labels of floor(x/s) under the output zero-labels, one corrupted
    s = rns.cardinality([moduli[i] for i in S])
    Yv = O.encode(op, _floor_div(x, s), zout, offs)
    bad_at = n // 2
    view = O.label_view(Yv, op, n, len(moduli) - 1)
    m_last = moduli[-1]
    r = O.pk32_unpack(m_last, view[:, bad_at].copy())
    r[-1] = (r[-1] + 1) % m_last
    view[:, bad_at] = O.pk32_pack(m_last, r)
    y = torch.empty(n, dtype=torch.int64, device="cuda")
    badc = torch.zeros(1, dtype=torch.int64, device="cuda")
    B.redash_decode(bp, H.to_dev(Yv), H.to_dev(zout), H.to_dev(offs), y, badc)
    torch.cuda.synchronize()
    oy, obad = O.decode(op, Yv, zout, offs)
    assert np.array_equal(y.cpu().numpy(), oy)
    assert int(badc.item()) == int(obad.sum()) == 1
    keep = np.arange(n) != bad_at
    assert np.array_equal(oy[keep], _floor_div(x, s)[keep])


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_gpu_pipeline_decodes_floor(case):
    name, moduli, S, n, seed, a0 = case
    bp = B.make_params(moduli, S, n, seed, a0)
    x = _small_inputs(moduli, n, seed)
    buf = H.gpu_pipeline(bp, x)
    assert int(buf.bad.item()) == 0
    assert np.array_equal(buf.y.cpu().numpy()[:n], _scaled(x, moduli, S))


def test_eval_is_repeatable_and_leaves_inputs():
    """The benchmark calls eval repeatedly on the same buffers."""
    w = WL.DENSE
    bp = B.make_params(w.moduli, w.scale_idx, 2048, w.seed)
    x = _small_inputs(w.moduli, 2048, 4)
    buf = H.gpu_pipeline(bp, x)
    first = H.to_u32(buf.out_labels).copy()
    inp = H.to_u32(buf.in_labels).copy()
    for _ in range(3):
        B.redash_eval_scale(bp, buf.in_labels, buf.tables, buf.out_labels, buf.work)
    torch.cuda.synchronize()
    assert np.array_equal(H.to_u32(buf.out_labels), first)
    assert np.array_equal(H.to_u32(buf.in_labels), inp)


def test_empty_calls_are_noops():
    bp = B.make_params(WL.TINY.moduli, WL.TINY.scale_idx, 0, 0)
    sz = B.redash_plan(bp)
    assert sz["label_words"] == 0 and sz["table_words"] == 0
    offs = torch.empty(sz["offset_words"], dtype=torch.int32, device="cuda")
    e = torch.empty(1, dtype=torch.int32, device="cuda")
    B.redash_garble_scale(bp, offs, e, e, e, e)
    offs2 = torch.empty_like(offs)
    B.redash_garble_scale_given(bp, offs2, e, e, e, e)
    B.redash_eval_scale(bp, e, e, e, e)
    bad = torch.full((1,), 7, dtype=torch.int64, device="cuda")
    B.redash_decode(bp, e, e, offs, torch.empty(1, dtype=torch.int64, device="cuda"), bad)
    torch.cuda.synchronize()
    assert int(bad.item()) == 0
    assert np.array_equal(H.to_u32(offs), O.garble(O.make_params(WL.TINY.moduli, WL.TINY.scale_idx, 1, 0), 0, 1)[0])
    assert np.array_equal(H.to_u32(offs2), H.to_u32(offs))


# ---------------------------------------------------------------------------
# full-size workloads in the benchmark's launch configuration
# ---------------------------------------------------------------------------

def _sample_gadgets(n: int, seed: int, head: int, tail: int, rand: int) -> np.ndarray:
    """The first `head` and last `tail` gadgets and `rand` seeded random ones
    (every gadget when that covers the call), sorted."""
    if head + tail + rand >= n:
        return np.arange(n, dtype=np.int64)
    rng = np.random.default_rng(seed + 777)
    mid = rng.choice(np.arange(head, n - tail), size=rand, replace=False)
    return np.unique(np.concatenate([np.arange(head), np.arange(n - tail, n), mid])).astype(np.int64)


def _runs(gad: np.ndarray):
    """Contiguous runs (first, count) of a sorted index list."""
    cut = np.flatnonzero(np.diff(gad) != 1) + 1
    return [(int(r[0]), len(r)) for r in np.split(gad, cut)]


def _oracle_zero_labels(op, moduli, gad: np.ndarray):
    """Offsets, input and output zero-labels of the given gadgets from the
    oracle's zero-label path (one hash per gate, no rows), laid out as a
    LabelTensor with stride len(gad)."""
    k = len(moduli)
    zi = [[] for _ in range(k)]
    zo = [[] for _ in range(k)]
    offs = None
    for a, c in _runs(gad):
        offs, zin, zout, _ = O.garble(op, a, c, with_tables=False)
        for i in range(k):
            zi[i].append(O.label_view(zin, op, c, i))
            zo[i].append(O.label_view(zout, op, c, i))
    cat = lambda parts: np.concatenate([np.concatenate(p, axis=1).reshape(-1) for p in parts])  # noqa: E731
    return offs, cat(zi), cat(zo)


def _check_full(w: WL.Workload, head: int, tail: int, rand: int, rows: int = 16):
    """Garble, encode, evaluate and decode one full-size workload in the
    benchmark's launch configuration; check every gadget through decode, the
    sampled gadgets' input zero-labels, output zero-labels and output labels
    word for word against the oracle's zero-label path, and the table rows of
    `rows` gadgets at each end and `rows` random ones against the oracle's
    garbling."""
    x = WL.make_inputs(w)
    n = w.n
    bp = B.make_params(w.moduli, w.scale_idx, n, w.seed)
    op = O.make_params(list(w.moduli), list(w.scale_idx), 1, w.seed)
    print(f"full-size {w.name}: n={n} moduli={w.moduli} S={w.scale_idx} seed={w.seed}", flush=True)
    buf = H.gpu_pipeline(bp, x)
    # every gadget: decode = floor(x/s) (floor((x + r)/s), see _scaled) and every label valid
    expect = _scaled(x, w.moduli, w.scale_idx)
    assert int(buf.bad.item()) == 0
    assert np.array_equal(buf.y.cpu().numpy()[:n], expect)
    # sampled gadgets: labels word for word against the oracle's zero-label path
    gad = _sample_gadgets(n, w.seed, head, tail, rand)
    li = H.label_index(w.moduli, n, gad)
    offs, zin, zout = _oracle_zero_labels(op, w.moduli, gad)
    assert np.array_equal(H.to_u32(buf.offsets), offs)
    assert np.array_equal(H.gather(buf.in_zero, li), zin)
    assert np.array_equal(H.gather(buf.out_zero, li), zout)
    # expected evaluator output: output zero-label + floor(x/s) * R
    Yexp = O.encode(op, expect[gad], zout, offs)
    got = H.gather(buf.out_labels, li)
    if not np.array_equal(got, Yexp):
        bad_words = np.flatnonzero(got != Yexp) % len(gad)
        raise AssertionError(f"{w.name}: output labels differ at gadgets {np.unique(gad[bad_words])[:10]}")
    # table rows of a few gadgets at both ends and in between
    rgad = _sample_gadgets(n, w.seed + 1, rows, rows, rows)
    gates = O.gate_list(op)
    gq = H.gate_list_sizes(gates, w.moduli)
    ti = H.table_index(gq, n, rgad)
    g_tab = H.gather(buf.tables, ti)
    for j, a in enumerate(rgad):
        _, _, _, tab = O.garble(op, int(a), 1)
        # rows: gate blocks of (q-1) W words, gadget-major inside each gate
        tsel, base = [], 0
        for (q, W) in gq:
            per = (q - 1) * W
            tsel.append(base + j * per + np.arange(per))
            base += len(rgad) * per
        assert np.array_equal(g_tab[np.concatenate(tsel)], tab), a
    del buf
    torch.cuda.empty_cache()


def test_full_size_conv():
    """The 64x32x32 conv map: every one of its 65,536 gadgets word for word."""
    _check_full(WL.CONV, WL.CONV.n, 0, 0, 32)


def test_full_size_batched():
    """The benchmark workload: 16x64x56x56 gadgets, 12 primes, s = 37;
    4,096 gadgets at each end and 8,192 random ones word for word."""
    _check_full(WL.BATCHED, 4096, 4096, 8192, 32)


# The evaluator's launch thresholds on this GPU.  Calls of up to one round of
# two workgroups per CU with 64, 192 or 384 gadgets per workgroup give each
# group of 64 gadgets 12, 4 or 2 waves; a call above one full round of the 4-
# or 2-wave split by at most 64 gadgets per CU runs that round on the split and
# the rest on 12 waves per 64 gadgets in the same launch; larger calls take
# one gadget per lane on whole rounds of 768-gadget workgroups, and a rest that
# the 12-wave split holds in one round (64 gadgets per workgroup) goes to it,
# starting at the first gadget after the rounds.  Each threshold and one gadget
# past it.  (name, whole rounds, gadgets per workgroup of the two per CU,
# gadgets per CU, extra): n = 2 cus (768 rounds + per) + cus per_cu + extra.
LAUNCH_EDGES = [("split12-last", 0, 64, 0, 0), ("split4-first", 0, 64, 0, 1), ("split4-last", 0, 192, 0, 0),
                ("split4-round-rest-first", 0, 192, 0, 1), ("split4-round-rest-last", 0, 192, 64, 0),
                ("split2-first", 0, 192, 64, 1), ("split2-last", 0, 384, 0, 0),
                ("split2-round-rest-first", 0, 384, 0, 1), ("split2-round-rest-last", 0, 384, 64, 0),
                ("one-per-lane-first", 0, 384, 64, 1), ("round-rest-one", 1, 0, 0, 1),
                ("round-rest-split12-last", 1, 64, 0, 0), ("round-rest-past-split12", 1, 64, 0, 1)]


@pytest.mark.parametrize("rounds,per,per_cu,extra", [e[1:] for e in LAUNCH_EDGES], ids=[e[0] for e in LAUNCH_EDGES])
def test_evaluator_launch_thresholds(rounds, per, per_cu, extra):
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 2 * cus * (768 * rounds + per) + cus * per_cu + extra
    P = rns.cardinality(WL.PRIMES_12)
    w = WL.Workload(f"edge-{n}", tuple(WL.PRIMES_12), (11,), n, 60 + per + per_cu + extra, "uniform", -(P // 2),
                    P - P // 2)
    _check_full(w, 4096, 4096, 8192)


def _round_and_rest_call(seed: int):
    """A layer-1-sized call (one full round of the 2-wave split and a rest of
    4,096 gadgets on 12 waves per 64 in the same launch), garbled and encoded."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 2 * cus * 384 + 4096
    w = WL.by_name("resnet18.l1.1.a")
    bp = B.make_params(w.moduli, w.scale_idx, n, seed)
    x = np.resize(WL.make_inputs(w), n)
    buf = B.Buffers(bp, "cuda")
    B.redash_garble_scale(bp, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work)
    B.redash_encode(bp, torch.from_numpy(x).cuda(), buf.in_zero, buf.offsets, buf.in_labels)
    torch.cuda.synchronize()
    return w, bp, x, buf


def test_round_and_rest_follow_the_callers_stream():
    """On a stream of the caller's other than the null stream, work queued
    after the call (decode) sees every gadget of the round and the rest, and a
    second call into fresh output buffers right behind the first gives the
    same labels."""
    w, bp, x, buf = _round_and_rest_call(81)
    s = torch.cuda.Stream()
    out2 = torch.full_like(buf.out_labels, -1)
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        buf.out_labels.fill_(-1)
        B.redash_eval_scale(bp, buf.in_labels, buf.tables, buf.out_labels, buf.work, s)
        B.redash_decode(bp, buf.out_labels, buf.out_zero, buf.offsets, buf.y, buf.bad, s)
        B.redash_eval_scale(bp, buf.in_labels, buf.tables, out2, buf.work, s)
    s.synchronize()
    assert int(buf.bad.item()) == 0
    assert np.array_equal(buf.y.cpu().numpy()[:len(x)], _scaled(x, w.moduli, w.scale_idx))
    assert torch.equal(out2, buf.out_labels)


def test_round_and_rest_under_graph_capture():
    """Captured in a graph: three replays, with eager calls and
    synchronizations between them, each equal to the eager call."""
    w, bp, x, buf = _round_and_rest_call(82)
    B.redash_eval_scale(bp, buf.in_labels, buf.tables, buf.out_labels, buf.work)
    torch.cuda.synchronize()
    ref = buf.out_labels.clone()
    out_g = torch.full_like(buf.out_labels, -1)
    work_g = torch.empty_like(buf.work)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, capture_error_mode="thread_local"):
        B.redash_eval_scale(bp, buf.in_labels, buf.tables, out_g, work_g)
    for _ in range(3):
        out_g.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        B.redash_eval_scale(bp, buf.in_labels, buf.tables, buf.out_labels, buf.work)
        torch.cuda.synchronize()
        assert torch.equal(out_g, ref)
        assert torch.equal(buf.out_labels, ref)
    del g


# Bases beyond the workloads' on the one-gadget-per-lane evaluator (its target-major
# schedule differs with k, t and the moduli: product scaling, 15 moduli, odd P,
# powers of two among the remaining moduli, moduli on the generic and the
# no-table fast paths): one gadget past the two-wave split's last call size.
K_EVAL_BASES = [
    ("k15-product", tuple(rns.first_primes(15)), (13, 14)),
    ("conv-base", tuple(WL.PRIMES_12[:10]), (8, 9)),
    ("generic-47-53-59", (2, 47, 53, 59), (1, 3)),
    ("large-moduli", (2, 97, 251), (2,)),
    ("pow2-128-product", (3, 128, 251), (0, 1)),
    ("pow2-4-remaining", (4, 5, 7), (1,)),
    ("odd-P", (3, 5, 7, 11, 13), (0, 4)),
    ("k2", (2, 3), (1,)),
]


@pytest.mark.parametrize("name,moduli,S", K_EVAL_BASES, ids=[b[0] for b in K_EVAL_BASES])
def test_one_gadget_per_lane_on_varied_bases(name, moduli, S):
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 2 * cus * 384 + 1
    P = rns.cardinality(moduli)
    w = WL.Workload(f"lane-{name}", tuple(moduli), tuple(S), n, 70 + len(moduli), "uniform", -(P // 2), P - P // 2)
    _check_full(w, 2048, 2048, 2048, 8)


RANDOM_LANE_BASES = [c[:3] for c in _random_bases(4, 7207)]


@pytest.mark.parametrize("name,moduli,S", RANDOM_LANE_BASES, ids=[b[0] for b in RANDOM_LANE_BASES])
def test_one_gadget_per_lane_on_random_bases(name, moduli, S):
    """Seeded random bases on the one-gadget-per-lane evaluator (one gadget
    past the sizes that run on the split evaluator)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 2 * cus * 384 + cus * 64 + 1
    P = rns.cardinality(moduli)
    w = WL.Workload(f"lane-{name}", tuple(moduli), tuple(S), n, 80 + len(moduli), "uniform", -(P // 2), P - P // 2)
    _check_full(w, 2048, 2048, 2048, 8)


# Seeded random bases (up to 6 moduli) at one size in each launch regime of
# the evaluator, as multiples of the CU count: the 12-wave split, the 4-wave
# split, a full 4-wave round and its rest, the 2-wave split, a full 2-wave
# round and its rest, and whole one-gadget-per-lane rounds with a rest.
REGIME_SIZES = [("split12", 0, 60, 7), ("split4", 0, 250, 11), ("split4-round-rest", 2 * 192, 40, 3),
                ("split2", 0, 600, 13), ("split2-round-rest", 2 * 384, 20, 5), ("lane-rounds-rest", 2 * 768, 100, 9)]
REGIME_BASES = [b for b in _random_bases(60, 3131) if len(b[1]) <= 6][: len(REGIME_SIZES)]


@pytest.mark.parametrize("regime,base", list(zip(REGIME_SIZES, REGIME_BASES)), ids=[r[0] for r in REGIME_SIZES])
def test_launch_regimes_on_random_bases(regime, base):
    name, rounds_per_cu, per_cu, extra = regime
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = cus * (rounds_per_cu + per_cu) + extra
    _, moduli, S = base[:3]
    P = rns.cardinality(moduli)
    w = WL.Workload(f"regime-{name}-{base[0]}", tuple(moduli), tuple(S), n, 90 + len(moduli), "uniform", -(P // 2),
                    P - P // 2)
    _check_full(w, 2048, 2048, 2048, 8)


@pytest.mark.parametrize("layer", WL.RESNET18, ids=[w.name for w in WL.RESNET18])
def test_full_size_resnet18_layer(layer):
    if layer.n >= 400_000:  # the stem, run like the benchmark workload
        _check_full(layer, 4096, 4096, 8192)
    else:
        _check_full(layer, 1024, 1024, 2048)


@pytest.mark.parametrize("w", WL.SHORT_BASES, ids=[w.name for w in WL.SHORT_BASES])
def test_short_base_micro_benchmark_size(w):
    """The paper's micro-benchmark size, 2^14 gadgets, every one word for word."""
    _check_full(w, w.n, 0, 0)


@pytest.mark.parametrize("w", WL.SHORT_BASES, ids=[w.name for w in WL.SHORT_BASES])
def test_short_base_at_batched_size(w):
    """As many gadgets as the 16x64x56x56 map, the size the benchmark times."""
    _check_full(WL.at_size(w, WL.BATCHED.n), 1024, 1024, 2048)
