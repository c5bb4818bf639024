"""Pins of the linear-layer oracle (oracle/linear.py) against what the
mathematics fixes, independent of the oracle's own arithmetic:

* packing: the numpy PK32 unpack/pack agree with the C oracle's PK32 (an
  independent implementation of the same layout definition);
* values: decoding the evaluator's output labels under the garbler's output
  zero-labels gives the exact integer layer output y = W x + b, computed here
  by direct Python loops over the convolution's definition (Sec. 2.3: free
  additions and constant multiplications; the garbler sets Z = sum w Z - b R);
* brute force: a dense layer over every input pair of a tiny base;
* special cases: identity weights return the input labels; zero weights
  return the all-zero label; linearity in the labels.

Decoding uses the gadget oracle's decode (label check included), so a label
that is not zero-label + value * R anywhere fails as a bad label.
"""

from __future__ import annotations

import numpy as np
import pytest

from oracle import linear as L
from oracle import oracle as O
from oracle import rns


def _op(moduli, n, seed=0):
    # scale set irrelevant to encode/decode; any valid one
    return O.make_params(list(moduli), [len(moduli) - 1], n, seed)


def _labels_for(moduli, x, seed):
    """Garbler material (offsets, input zero-labels) from the gadget oracle's
    PRG, and the evaluator's input labels of values x."""
    op = _op(moduli, len(x), seed)
    offs, zin, _zout, _ = O.garble(op, 0, len(x), with_tables=False)
    X = O.encode(op, np.asarray(x, np.int64), zin, offs)
    return op, offs, zin, X


def _direct_conv(x, w, b, stride, pad):
    """y[n,o,i,j] = b[o] + sum_{c,dy,dx} w[o,c,dy,dx] x[n,c,i s+dy-p, j s+dx-p]
    with zero padding, by plain loops over the definition."""
    n, c_in, h, wd = x.shape
    c_out, _, kh, kw = w.shape
    ho, wo = (h + 2 * pad - kh) // stride + 1, (wd + 2 * pad - kw) // stride + 1
    y = np.zeros((n, c_out, ho, wo), dtype=object)
    for a in range(n):
        for o in range(c_out):
            for i in range(ho):
                for j in range(wo):
                    s = int(b[o])
                    for c in range(c_in):
                        for dy in range(kh):
                            for dx in range(kw):
                                yi, xj = i * stride + dy - pad, j * stride + dx - pad
                                if 0 <= yi < h and 0 <= xj < wd:
                                    s += int(w[o, c, dy, dx]) * int(x[a, c, yi, xj])
                    y[a, o, i, j] = s
    return y


@pytest.mark.parametrize("m", [2, 3, 5, 7, 11, 13, 16, 32, 37, 97, 173, 251])
def test_pack_matches_c_oracle(m):
    rng = np.random.default_rng(m)
    count = 7
    lam = L.label_lambda(m)
    assert lam == O.lam(m) and L.label_words(m) == O.words(m)
    res = rng.integers(0, m, size=(count, lam))
    packed = L.pack([m], [res], count)
    W = O.words(m)
    for a in range(count):
        assert np.array_equal(packed.reshape(W, count)[:, a], O.pk32_pack(m, res[a]))
    back = L.unpack([m], packed, count)[0]
    assert np.array_equal(back, res)


CONV_CASES = [
    # moduli, (n, c_in, h, w), c_out, kh, kw, stride, pad
    ((2, 3, 5, 7, 11, 13), (2, 3, 5, 4), 2, 3, 3, 1, 1),
    ((3, 5, 7, 11, 13, 32), (1, 2, 6, 7), 3, 3, 2, 2, 1),
    ((2, 3, 5, 7, 11, 13, 17), (1, 4, 4, 4), 5, 1, 1, 1, 0),
    ((5, 7, 97, 251), (2, 3, 3, 5), 2, 2, 3, 1, 0),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_decodes_to_exact_layer_output(case):
    moduli, shape, c_out, kh, kw, stride, pad = case
    rng = np.random.default_rng(sum(shape) + c_out)
    n, c_in, h, w = shape
    x = rng.integers(-5, 6, size=shape)
    wts = rng.integers(-9, 10, size=(c_out, c_in, kh, kw))
    wts[0, 0, 0, -1] = 300  # a weight above most moduli (acts through its residue)
    b = rng.integers(-50, 51, size=c_out)
    op, offs, zin, X = _labels_for(moduli, x.reshape(-1), 5)
    Y = L.conv_labels(moduli, X, shape, wts, stride, pad)
    Z = L.garble_conv(moduli, zin, shape, wts, b, offs, stride, pad)
    y, bad = O.decode(op, Y, Z, offs)
    exact = _direct_conv(x, wts, b, stride, pad).reshape(-1)
    P = rns.cardinality(moduli)
    assert all(abs(v) < P // 2 for v in exact)
    assert bad.sum() == 0
    assert [int(v) for v in y] == list(exact)


def test_dense_brute_force_tiny_base():
    """Every input pair of the base (3, 5): y = 2 x0 - 7 x1 + 4 wrapped into
    the signed range of Z_15."""
    moduli = (3, 5)
    P = 15
    wts = np.array([[2, -7]])
    b = [4]
    xs = np.array([(u, v) for u in range(-7, 8) for v in range(-7, 8)])
    flat = xs.reshape(-1)
    op, offs, zin, X = _labels_for(moduli, flat, 9)
    batch = len(xs)
    Y = L.dense_labels(moduli, X, batch, wts)
    Z = L.garble_dense(moduli, zin, batch, wts, b, offs)
    y, bad = O.decode(_op(moduli, batch), Y, Z, offs)
    assert bad.sum() == 0
    for (x0, x1), got in zip(xs, y):
        v = (2 * x0 - 7 * x1 + 4) % P
        assert got == (v if v < (P + 1) // 2 else v - P)


def test_identity_and_zero_weights():
    moduli = (2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37)
    shape = (1, 3, 4, 5)
    x = np.random.default_rng(1).integers(-1000, 1000, size=shape)
    op, offs, zin, X = _labels_for(moduli, x.reshape(-1), 2)
    eye = np.zeros((3, 3, 1, 1), np.int64)
    for c in range(3):
        eye[c, c, 0, 0] = 1
    assert np.array_equal(L.conv_labels(moduli, X, shape, eye), X)
    assert not L.conv_labels(moduli, X, shape, np.zeros((2, 3, 3, 3), np.int64), 1, 1).any()
    # weight m_i * k acts as 0 on modulus i only: P acts as 0 everywhere
    Pw = np.full((1, 3, 1, 1), rns.cardinality(moduli), np.int64)
    assert not L.conv_labels(moduli, X, shape, Pw).any()


def test_linear_in_labels():
    """conv(X1) + conv(X2) = conv(X1 + X2) residue-wise (free addition)."""
    moduli = (3, 5, 7, 32)
    shape = (1, 2, 5, 5)
    rng = np.random.default_rng(4)
    wts = rng.integers(-100, 100, size=(3, 2, 3, 3))
    X1 = L.pack(moduli, [rng.integers(0, m, size=(50, L.label_lambda(m))) for m in moduli], 50)
    X2 = L.pack(moduli, [rng.integers(0, m, size=(50, L.label_lambda(m))) for m in moduli], 50)
    S = L.pack(moduli, [(a + b) % m for a, b, m in zip(L.unpack(moduli, X1, 50), L.unpack(moduli, X2, 50), moduli)],
               50)
    Y1, Y2, YS = (L.unpack(moduli, L.conv_labels(moduli, X, shape, wts, 1, 1), 75) for X in (X1, X2, S))
    for a, b, s, m in zip(Y1, Y2, YS, moduli):
        assert np.array_equal((a + b) % m, s)


def test_sampled_equals_full():
    moduli = (2, 3, 5, 7, 11, 16)
    shape = (2, 3, 6, 5)
    rng = np.random.default_rng(7)
    wts = rng.integers(-300, 300, size=(4, 3, 3, 3))
    X = L.pack(moduli, [rng.integers(0, m, size=(180, L.label_lambda(m))) for m in moduli], 180)
    for stride, pad in ((1, 1), (2, 1), (2, 0)):
        full = L.conv_labels(moduli, X, shape, wts, stride, pad)
        count = int(np.prod(L.conv_out_shape(*shape, 4, 3, 3, stride, pad)))
        items = np.array(sorted(rng.choice(count, size=min(17, count), replace=False)))
        samp = L.conv_labels_sampled(moduli, X, shape, wts, stride, pad, items)
        res_full = L.unpack(moduli, full, count)
        res_samp = L.unpack(moduli, samp, len(items))
        for rf, rs in zip(res_full, res_samp):
            assert np.array_equal(rf[items], rs)


def test_garble_given_equals_garble_on_its_own_zero_labels():
    """Garbling on given input zero-labels reproduces the PRG garbling when
    given the PRG's zero-labels (same offsets, output zero-labels, rows)."""
    moduli, S, n, seed = (2, 3, 5, 7, 11), [4], 37, 3
    op = O.make_params(list(moduli), S, n, seed)
    offs, zin, zout, tab = O.garble(op, 5, n)
    offs2, zout2, tab2 = O.garble_given(op, 5, n, zin)
    assert np.array_equal(offs, offs2) and np.array_equal(zout, zout2) and np.array_equal(tab, tab2)


@pytest.mark.parametrize("moduli,S", [((2, 3, 5, 7, 11, 13), [5]), ((3, 5, 7, 11, 32), [4]),
                                      ((2, 3, 5, 7, 11, 13, 17), [5, 6])])
def test_conv_layer_feeds_the_gadget(moduli, S):
    """A conv layer on labels, then the scaling gadget garbled on the layer's
    output zero-labels: decoding the gadget's output labels gives
    floor((W x + b + r) / s), r = floor(P/2) mod s (Sec. 2.3 free operations,
    then Sec. 3.4), computed here from the plain integer convolution."""
    shape, c_out, kh, kw, stride, pad = (1, 3, 4, 5), 2, 3, 3, 1, 1
    rng = np.random.default_rng(len(moduli))
    x = rng.integers(-6, 7, size=shape)
    wts = rng.integers(-9, 10, size=(c_out, shape[1], kh, kw))
    b = rng.integers(-40, 41, size=c_out)
    n_in = int(np.prod(shape))
    op_in = O.make_params(list(moduli), S, n_in, 21)
    offs, zin, _zout, _ = O.garble(op_in, 0, n_in, with_tables=False)
    X = O.encode(op_in, x.reshape(-1), zin, offs)
    Y = L.conv_labels(moduli, X, shape, wts, stride, pad)
    Z = L.garble_conv(moduli, zin, shape, wts, b, offs, stride, pad)
    n_out = int(np.prod(L.conv_out_shape(*shape, c_out, kh, kw, stride, pad)))
    op = O.make_params(list(moduli), S, n_out, 21)  # the same seed: the same offsets R
    a0 = 1000                                         # gadgets with their own tweaks
    offs2, gz_out, tab = O.garble_given(op, a0, n_out, Z)
    assert np.array_equal(offs2, offs)
    out = O.evaluate(op, a0, n_out, Y, tab)
    y, bad = O.decode(op, out, gz_out, offs)
    lin = np.array([int(v) for v in _direct_conv(x, wts, b, stride, pad).reshape(-1)], dtype=np.int64)
    s_ = rns.cardinality([moduli[i] for i in S])
    r = rns.rounding_offset(list(moduli), list(S))
    assert bad.sum() == 0
    assert np.array_equal(y, np.floor_divide(lin + r, s_))
