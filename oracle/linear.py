"""Garbled linear layers (dense and 2-D convolution) on LabelTensors: a plain,
slow numpy oracle.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module.  It shares no code
with the HIP library.

What it follows (Sec. 2.3): an arithmetic-garbled wire over Z_m carries the
label l_a = l_0 + a R; adding labels and multiplying a label by a public
constant are free, residue by residue mod m.  A linear layer with public
integer weights w and bias b, y_o = sum_j w_oj x_j + b_o, is therefore
evaluated on labels as

    Y_o = sum_j w_oj X_j            (mod m, every residue, every modulus)

and the garbler, who knows R, sets the output zero-label so that Y_o carries
y_o:

    Z_o = sum_j w_oj Z_j - b_o R    (mod m),

since sum_j w_oj (Z_j + x_j R) = Z_o + (sum_j w_oj x_j + b_o) R.  The paper
runs dense and convolution layers this way on LabelTensors with 32-bit
residues (Sec. 3.6); it fixes no layout.  Layers here:

  * conv2d: input NCHW (n, c_in, h, w), weights OIHW (c_out, c_in, kh, kw),
    stride s, zero padding p (a padded input is the public constant 0, whose
    label and zero-label are both the all-zero label), output
    (n, c_out, (h + 2p - kh)/s + 1, (w + 2p - kw)/s + 1);
  * dense: input (batch, in), weights (out, in) -- the conv with
    h = w = kh = kw = 1.

Labels use the packed LabelTensor layout of the scaling gadget (PK32: residue
r of a label over Z_m in word r // g at bit b (r % g), b = bit length of
m - 1, g = 32 // b; modulus blocks of W_m * count words, word w of item a at
w * count + a).  Unpacking and packing are restated here from that
definition.

The arithmetic is int64 numpy: weights are reduced mod m first, so every
product is below 2^16 and every sum of up to 2^40 products is exact.
"""

from __future__ import annotations

import numpy as np


def label_lambda(m: int) -> int:
    """Residues per label: the least lambda with m^lambda >= 2^128."""
    lam, v = 0, 1
    while v < (1 << 128):
        v *= m
        lam += 1
    return lam


def _field_bits(m: int) -> int:
    return (m - 1).bit_length()


def label_words(m: int) -> int:
    g = 32 // _field_bits(m)
    return -(-label_lambda(m) // g)


def unpack(moduli, buf: np.ndarray, count: int) -> list:
    """The residues of every label of a LabelTensor: one int64 array of shape
    (count, lambda_m) per modulus."""
    out, off = [], 0
    buf = np.asarray(buf, dtype=np.uint32)
    for m in moduli:
        b, lam, W = _field_bits(m), label_lambda(m), label_words(m)
        g = 32 // b
        words = buf[off: off + W * count].reshape(W, count).astype(np.int64)
        res = np.zeros((count, lam), np.int64)
        for r in range(lam):
            res[:, r] = (words[r // g] >> (b * (r % g))) & ((1 << b) - 1)
        out.append(res)
        off += W * count
    return out


def pack(moduli, residues: list, count: int) -> np.ndarray:
    """Inverse of unpack: residues (count, lambda_m) per modulus -> packed words."""
    blocks = []
    for m, res in zip(moduli, residues):
        b, lam, W = _field_bits(m), label_lambda(m), label_words(m)
        g = 32 // b
        assert res.shape == (count, lam) and res.min(initial=0) >= 0 and res.max(initial=0) < m
        words = np.zeros((W, count), np.int64)
        for r in range(lam):
            words[r // g] |= res[:, r].astype(np.int64) << (b * (r % g))
        blocks.append(words.reshape(-1))
    return np.concatenate(blocks).astype(np.uint32) if blocks else np.zeros(0, np.uint32)


def conv_out_shape(n, c_in, h, w, c_out, kh, kw, stride, pad):
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (w + 2 * pad - kw) // stride + 1
    return (n, c_out, ho, wo)


def conv_residues(res: np.ndarray, m: int, shape, weights: np.ndarray, stride: int, pad: int) -> np.ndarray:
    """One modulus: res (n*c_in*h*w, lambda) residues of the input labels in
    NCHW order -> (n*c_out*ho*wo, lambda) residues of sum w X mod m."""
    n, c_in, h, w = shape
    c_out, _, kh, kw = weights.shape
    lam = res.shape[1]
    x = res.reshape(n, c_in, h, w, lam)
    xp = np.zeros((n, c_in, h + 2 * pad, w + 2 * pad, lam), np.int64)
    xp[:, :, pad: pad + h, pad: pad + w, :] = x
    _, _, ho, wo = conv_out_shape(n, c_in, h, w, c_out, kh, kw, stride, pad)
    wm = np.mod(weights.astype(np.int64), m)  # a public constant acts through its residue mod m
    acc = np.zeros((n, c_out, ho, wo, lam), np.int64)
    for dy in range(kh):
        for dx in range(kw):
            # input window of tap (dy, dx) for every output position
            win = xp[:, :, dy: dy + stride * (ho - 1) + 1: stride, dx: dx + stride * (wo - 1) + 1: stride, :]
            # sum over input channels c of w[o, c, dy, dx] * X[n, c, ...]
            acc += np.einsum("oc,nchwr->nohwr", wm[:, :, dy, dx], win)
            acc %= m
    return acc.reshape(n * c_out * ho * wo, lam)


def conv_labels(moduli, labels: np.ndarray, shape, weights: np.ndarray, stride: int = 1, pad: int = 0):
    """Evaluator: output labels Y = sum w X (Sec. 2.3 free operations) of a
    conv2d layer on the packed input labels (count = n*c_in*h*w)."""
    n, c_in, h, w = shape
    c_out, c_w, kh, kw = weights.shape
    assert c_w == c_in
    count_in = n * c_in * h * w
    out_shape = conv_out_shape(n, c_in, h, w, c_out, kh, kw, stride, pad)
    count_out = int(np.prod(out_shape))
    res = unpack(moduli, labels, count_in)
    out = [conv_residues(r, m, shape, weights, stride, pad) for r, m in zip(res, moduli)]
    return pack(moduli, out, count_out)


def garble_conv(moduli, zero_in: np.ndarray, shape, weights: np.ndarray, bias, offsets: np.ndarray,
                stride: int = 1, pad: int = 0):
    """Garbler: output zero-labels Z_o = sum w Z - b_o R (Sec. 2.3), so that
    the evaluator's output label of item o carries y_o = sum w x + b_o."""
    n, c_in, h, w = shape
    c_out = weights.shape[0]
    out_shape = conv_out_shape(n, c_in, h, w, c_out, weights.shape[2], weights.shape[3], stride, pad)
    count_out = int(np.prod(out_shape))
    conv = unpack(moduli, conv_labels(moduli, zero_in, shape, weights, stride, pad), count_out)
    R = unpack(moduli, offsets, 1)
    b = np.zeros(c_out, np.int64) if bias is None else np.asarray(bias, np.int64)
    # the output channel of every output item (NCHW order)
    o_of = np.broadcast_to(np.arange(c_out)[None, :, None, None], out_shape).reshape(-1)
    out = []
    for m, z, Rm in zip(moduli, conv, R):
        bm = np.mod(b, m)[o_of]                       # b_o mod m per item
        out.append(np.mod(z - bm[:, None] * Rm[0][None, :], m))
    return pack(moduli, out, count_out)


def dense_labels(moduli, labels, batch: int, weights: np.ndarray):
    """Evaluator for a dense layer: input (batch, in), weights (out, in)."""
    out_f, in_f = weights.shape
    return conv_labels(moduli, labels, (batch, in_f, 1, 1), weights.reshape(out_f, in_f, 1, 1))


def garble_dense(moduli, zero_in, batch: int, weights: np.ndarray, bias, offsets):
    out_f, in_f = weights.shape
    return garble_conv(moduli, zero_in, (batch, in_f, 1, 1), weights.reshape(out_f, in_f, 1, 1), bias, offsets)


def conv_labels_sampled(moduli, labels: np.ndarray, shape, weights: np.ndarray, stride: int, pad: int,
                        out_items: np.ndarray) -> np.ndarray:
    """conv_labels for selected output items only (flat NCHW indices into the
    output), for tensors too large to unpack whole.  Returns the packed
    labels of those items as a LabelTensor with stride len(out_items)."""
    n, c_in, h, w = shape
    c_out, _, kh, kw = weights.shape
    _, _, ho, wo = conv_out_shape(n, c_in, h, w, c_out, kh, kw, stride, pad)
    count_in = n * c_in * h * w
    out_items = np.asarray(out_items, np.int64)
    nn, rem = np.divmod(out_items, c_out * ho * wo)
    oo, rem = np.divmod(rem, ho * wo)
    yy, xx = np.divmod(rem, wo)
    labels = np.asarray(labels, np.uint32)
    out, off = [], 0
    for m in moduli:
        b, lam, W = _field_bits(m), label_lambda(m), label_words(m)
        g = 32 // b
        block = labels[off: off + W * count_in].reshape(W, count_in)
        wm = np.mod(weights.astype(np.int64), m)
        acc = np.zeros((len(out_items), lam), np.int64)
        for c in range(c_in):
            for dy in range(kh):
                for dx in range(kw):
                    iy, ix = yy * stride + dy - pad, xx * stride + dx - pad
                    inside = (iy >= 0) & (iy < h) & (ix >= 0) & (ix < w)
                    src = ((nn * c_in + c) * h + np.clip(iy, 0, h - 1)) * w + np.clip(ix, 0, w - 1)
                    words = block[:, src].astype(np.int64)            # (W, items)
                    for r in range(lam):
                        v = (words[r // g] >> (b * (r % g))) & ((1 << b) - 1)
                        acc[:, r] += np.where(inside, wm[oo, c, dy, dx] * v, 0)
            acc %= m
        out.append(acc)
        off += W * count_in
    return pack(moduli, out, len(out_items))
