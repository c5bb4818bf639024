"""GPU parity of the garbled linear layers (redash_linear_*) against the
linear-layer oracle (oracle/linear.py), bit for bit.

Small layers: every word of the evaluator's output labels and of the
garbler's output zero-labels is compared with the oracle, over shapes that
cover dense layers, strides, padding, several channel chunks, several groups
of 64 output channels, ragged tiles, power-of-two and large moduli.  Full-size
layers (the 3x3x64 convolution that produces the 16x64x56x56 batched map, and
ResNet-18 layers) run end to end on the GPU: every output decodes to the
exact integer convolution, and a seeded sample of output labels is compared
with the oracle item by item.
"""

from __future__ import annotations

import zlib

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import linear as OL  # noqa: E402
from paper_2506_14489_amd import binding as B  # noqa: E402
from paper_2506_14489_amd import workloads as WL  # noqa: E402

import gpu_helpers as H  # noqa: E402

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU containers
    pytest.skip("needs a GPU", allow_module_level=True)


def _dev_u8(n):
    return torch.empty(max(int(n), 1), dtype=torch.uint8, device="cuda")


def _random_labels(moduli, count, rng):
    return OL.pack(moduli, [rng.integers(0, m, size=(count, OL.label_lambda(m))) for m in moduli], count)


SMALL = [
    # name, moduli, (batch, c_in, h, w), c_out, kh, kw, stride, pad
    ("conv3x3-12primes", tuple(WL.PRIMES_12), (2, 5, 6, 7), 3, 3, 3, 1, 1),
    ("conv3x3-wide-row", (2, 3, 5, 7, 11), (1, 16, 3, 70), 8, 3, 3, 1, 1),
    ("conv-stride2", (3, 5, 7, 32), (1, 20, 9, 18), 6, 3, 3, 2, 1),
    ("stem-like-7x7s2", (5, 7, 11), (1, 3, 20, 21), 9, 7, 7, 2, 3),
    ("conv-chunks-and-groups", (2, 251), (1, 130, 3, 4), 70, 3, 3, 1, 1),
    ("conv-1x1-stride2", (13, 16, 17), (2, 17, 6, 6), 5, 1, 1, 2, 0),
    ("conv-2x3-nopad", (4, 5, 7), (1, 4, 5, 6), 3, 2, 3, 1, 0),
    ("dense", tuple(WL.PRIMES_12), (33, 100, 1, 1), 70, 1, 1, 1, 0),
    ("dense-batch1", (32, 167, 173), (1, 512, 1, 1), 10, 1, 1, 1, 0),
    ("short-base-conv", (32, 97, 107), (1, 64, 5, 5), 64, 3, 3, 1, 1),
    # one 64-channel chunk: the kernel with independent waves, 3x3 paths
    ("conv3x3-64ch-ragged-tiles", (3, 5, 7, 11, 13), (1, 64, 4, 70), 8, 3, 3, 1, 1),
    ("conv3x3-64ch-stride2", (2, 3, 5, 7), (2, 64, 9, 20), 6, 3, 3, 2, 1),
    ("conv3x3-64ch-m251-three-groups", (2, 251), (1, 64, 5, 9), 130, 3, 3, 1, 1),
    ("conv3x3-64ch-whole-tiles", (5, 7, 64), (1, 64, 3, 64), 64, 3, 3, 1, 1),
    # kernels one column wide and taller than one row (the tap's row and column
    # from one division by kw = 1), and one row high
    ("conv-3x1", (2, 3, 5, 7), (1, 20, 9, 7), 6, 3, 1, 1, 0),
    ("conv-5x1-two-chunks", (3, 4, 5, 13), (2, 119, 9, 6), 5, 5, 1, 1, 0),
    ("conv-2x1-stride3-two-chunks", (3, 4, 5, 13), (2, 119, 9, 6), 5, 2, 1, 3, 0),
    ("conv-1x3", (2, 3, 5, 7, 11), (1, 33, 5, 12), 9, 1, 3, 1, 0),
    # several 64-channel chunks, 3x3, rows of at most 16 outputs: the next
    # chunk's weights are loaded into registers while a stage computes
    ("conv3x3-three-chunks-7x7", (2, 3, 5, 7, 37), (1, 192, 7, 7), 64, 3, 3, 1, 1),
    ("conv3x3-two-chunks-stride2", (3, 5, 7, 31), (1, 128, 14, 14), 70, 3, 3, 2, 1),
    # flattened tiles (3x3 stride 1 over several chunks, rows of at most 8 outputs)
    ("flat-narrow-batch2-ragged", (2, 3, 5, 7, 37), (2, 128, 5, 6), 70, 3, 3, 1, 1),
    ("flat-narrow-nopad-m251", (3, 5, 251), (1, 130, 9, 10), 9, 3, 3, 1, 0),
    # column fold (fewer than 16 channels, kw c_in <= 64: kh x 1 over kw c_in channels)
    ("fold-63-channels-m251", (2, 251), (1, 9, 11, 13), 5, 7, 7, 1, 3),
    ("no-fold-63-channels-stride2-halo", (2, 251), (1, 9, 11, 13), 5, 7, 7, 2, 3),
    ("fold-one-channel-5x5", (3, 5, 7, 11), (2, 1, 9, 23), 4, 5, 5, 1, 2),
    ("fold-1x4-stride3", (2, 3, 5, 7), (1, 2, 4, 17), 6, 1, 4, 3, 0),
    ("no-fold-65-channels", (5, 7), (1, 13, 6, 8), 3, 5, 5, 1, 2),
]


def _random_linear(count: int, seed: int):
    """Seeded random layers: bases of 1 to 6 moduli drawn mostly from the
    small ones (2, 3, 4, 5, 7, 8, 11, 13, 16, whose residues share plane
    bytes) and some larger, at most one of them even; random shapes, kernels,
    strides and padding that the plan accepts."""
    rng = np.random.default_rng(seed)
    small = [2, 3, 4, 5, 7, 8, 11, 13, 16]
    large = [17, 19, 23, 29, 31, 32, 37, 41, 64, 97, 127, 128, 251]
    out = []
    while len(out) < count:
        k = int(rng.integers(1, 7))
        pool = small if rng.random() < 0.7 else small + large
        base = sorted(int(m) for m in rng.choice(pool, size=min(k, len(pool)), replace=False))
        if sum(1 for m in base if m % 2 == 0) > 1:
            continue
        kh, kw = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        shape = (int(rng.integers(1, 3)), int(rng.integers(1, 131)), int(rng.integers(kh, 13)),
                 int(rng.integers(kw, 13)))
        c_out = int(rng.integers(1, 81))
        stride = int(rng.integers(1, 4))
        pad = int(rng.integers(0, min(kh, kw)))
        lp = B.make_linear_params(tuple(base), *shape, c_out, kh, kw, stride, pad)
        if B.linear_plan_rc(lp) != 0:
            continue
        out.append((f"rand{len(out)}-{'-'.join(map(str, base))}", tuple(base), shape, c_out, kh, kw, stride, pad))
    return out


RANDOM_LINEAR = _random_linear(16, 4242)


def _random_linear_wide(count: int, seed: int):
    """Seeded random layers over wider shapes: any accepted modulus up to 251,
    dense layers of up to 300 inputs and 40 rows, convolutions of up to 199
    channels (several channel chunks), up to 139 outputs (several groups of
    64), kernels up to 7x7 (at most 64 taps), strides 1 to 4; sized so that
    the oracle's plain convolution stays small."""
    rng = np.random.default_rng(seed)
    pool = [2, 3, 4, 5, 7, 8, 11, 13, 16, 17, 19, 23, 29, 31, 32, 37, 41, 64, 97, 127, 128, 251]
    out = []
    while len(out) < count:
        k = int(rng.integers(1, 7))
        base = sorted(int(m) for m in rng.choice(pool, size=k, replace=False))
        if sum(1 for m in base if m % 2 == 0) > 1:
            continue
        if rng.random() < 0.25:
            shape, kh, kw, stride, pad = (int(rng.integers(1, 40)), int(rng.integers(1, 300)), 1, 1), 1, 1, 1, 0
        else:
            kh, kw = int(rng.integers(1, 8)), int(rng.integers(1, 8))
            if kh * kw > 64:
                continue
            shape = (int(rng.integers(1, 3)), int(rng.integers(1, 200)), int(rng.integers(kh, 11)),
                     int(rng.integers(kw, 11)))
            stride, pad = int(rng.integers(1, 5)), int(rng.integers(0, min(kh, kw)))
        c_out = int(rng.integers(1, 140))
        n, c_in, h, w = shape
        ho, wo = (h + 2 * pad - kh) // stride + 1, (w + 2 * pad - kw) // stride + 1
        if n * ho * wo * c_out * c_in * kh * kw * sum(OL.label_lambda(m) for m in base) > 3e8:
            continue
        lp = B.make_linear_params(tuple(base), *shape, c_out, kh, kw, stride, pad)
        if B.linear_plan_rc(lp) != 0:
            continue
        out.append((f"wide{len(out)}-{'-'.join(map(str, base))}", tuple(base), shape, c_out, kh, kw, stride, pad))
    return out


RANDOM_LINEAR += _random_linear_wide(32, 777)


@pytest.mark.parametrize("case", SMALL + RANDOM_LINEAR, ids=[c[0] for c in SMALL + RANDOM_LINEAR])
def test_linear_matches_oracle(case):
    name, moduli, shape, c_out, kh, kw, stride, pad = case
    print(f"linear {name}: moduli={moduli} shape={shape} c_out={c_out} k={kh}x{kw} s={stride} p={pad}", flush=True)
    n, c_in, h, w = shape
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    lp = B.make_linear_params(moduli, n, c_in, h, w, c_out, kh, kw, stride, pad)
    sz = B.redash_linear_plan(lp)
    count_in = n * c_in * h * w
    X = _random_labels(moduli, count_in, rng)
    Z = _random_labels(moduli, count_in, rng)
    R = _random_labels(moduli, 1, rng)
    wts = rng.integers(-2 ** 31, 2 ** 31, size=(c_out, c_in, kh, kw), dtype=np.int64)
    wts[:, :, 0, 0] = rng.integers(-3, 4, size=(c_out, c_in))  # small weights too
    bias = rng.integers(-2 ** 62, 2 ** 62, size=c_out, dtype=np.int64)
    prep = _dev_u8(sz["prepared_bytes"])
    work = _dev_u8(sz["work_bytes"])
    B.redash_linear_prepare(lp, H.to_dev(wts.astype(np.int32)), prep)
    out = torch.empty(sz["out_label_words"], dtype=torch.int32, device="cuda")
    B.redash_linear_eval(lp, H.to_dev(X), prep, work, out)
    zout = torch.empty(sz["out_label_words"], dtype=torch.int32, device="cuda")
    B.redash_linear_garble(lp, H.to_dev(Z), prep, H.to_dev(bias), H.to_dev(R), work, zout)
    torch.cuda.synchronize()
    w32 = wts.astype(np.int32).astype(np.int64)  # the int32 weights the library was given
    assert np.array_equal(H.to_u32(out), OL.conv_labels(moduli, X, shape, w32, stride, pad))
    assert np.array_equal(H.to_u32(zout), OL.garble_conv(moduli, Z, shape, w32, bias, R, stride, pad))


def test_linear_garble_without_bias_and_repeatability():
    moduli = (2, 3, 5, 7, 11, 13)
    shape, c_out = (1, 8, 5, 5), 4
    rng = np.random.default_rng(3)
    lp = B.make_linear_params(moduli, *shape, c_out, 3, 3, 1, 1)
    sz = B.redash_linear_plan(lp)
    Z = _random_labels(moduli, int(np.prod(shape)), rng)
    R = _random_labels(moduli, 1, rng)
    wts = rng.integers(-50, 50, size=(c_out, shape[1], 3, 3))
    prep = _dev_u8(sz["prepared_bytes"])
    work = _dev_u8(sz["work_bytes"])
    B.redash_linear_prepare(lp, H.to_dev(wts.astype(np.int32)), prep)
    zout = torch.empty(sz["out_label_words"], dtype=torch.int32, device="cuda")
    zd = H.to_dev(Z)
    B.redash_linear_garble(lp, zd, prep, None, H.to_dev(R), work, zout)
    torch.cuda.synchronize()
    first = H.to_u32(zout).copy()
    assert np.array_equal(first, OL.garble_conv(moduli, Z, shape, wts, None, R, 1, 1))
    for _ in range(3):
        B.redash_linear_garble(lp, zd, prep, None, H.to_dev(R), work, zout)
    torch.cuda.synchronize()
    assert np.array_equal(H.to_u32(zout), first)
    assert np.array_equal(H.to_u32(zd), Z)


# ---------------------------------------------------------------------------
# full-size layers on the GPU: garble inputs with the gadget garbler's PRG,
# encode the int8 activations, run the layer both ways, decode every output
# ---------------------------------------------------------------------------

def _run_full_layer(w: WL.Workload):
    """Garble the layer's inputs with the gadget garbler (PRG over n_in items,
    gadgets 0..n_in-1), encode the int8 activations, run the layer both ways.
    Returns (shape, kshape, wt, X, Y, Zo, offsets)."""
    a, wt = WL.layer_operands(w)
    moduli = w.moduli
    if w.kind == "fc":
        batch, c_in = w.in_shape
        lp = B.make_linear_params(moduli, batch, c_in, 1, 1, w.w_shape[0])
        shape, kshape = (batch, c_in, 1, 1), (w.w_shape[0], c_in, 1, 1)
    else:
        n, c_in, h, wd = w.in_shape
        c_out, _, kh, kw = w.w_shape
        lp = B.make_linear_params(moduli, n, c_in, h, wd, c_out, kh, kw, w.stride, w.pad)
        shape, kshape = w.in_shape, w.w_shape
    sz = B.redash_linear_plan(lp)
    n_in = int(np.prod(shape))
    gp_in = B.make_params(moduli, w.scale_idx, n_in, w.seed)
    g = B.Buffers(gp_in)
    B.redash_garble_scale(gp_in, g.offsets, g.in_zero, g.out_zero, g.tables, g.work)
    xa = torch.from_numpy(a.reshape(-1).astype(np.int64)).cuda()
    B.redash_encode(gp_in, xa, g.in_zero, g.offsets, g.in_labels)
    zin, X, offsets = g.in_zero, g.in_labels, g.offsets
    del g
    torch.cuda.empty_cache()
    wts = torch.from_numpy(wt.reshape(kshape).astype(np.int32)).cuda()
    prep = _dev_u8(sz["prepared_bytes"])
    work = _dev_u8(sz["work_bytes"])
    B.redash_linear_prepare(lp, wts, prep)
    Y = torch.empty(sz["out_label_words"], dtype=torch.int32, device="cuda")
    Zo = torch.empty(sz["out_label_words"], dtype=torch.int32, device="cuda")
    B.redash_linear_eval(lp, X, prep, work, Y)
    B.redash_linear_garble(lp, zin, prep, None, offsets, work, Zo)
    del work, zin
    torch.cuda.empty_cache()
    return shape, kshape, wt, X, Y, Zo, offsets


def _check_full_layer(w: WL.Workload, n_sample: int):
    moduli, n_out = w.moduli, w.n
    shape, kshape, wt, X, Y, Zo, offsets = _run_full_layer(w)
    # decode every output with the gadget library's decode (any scale set of the base)
    gp_out = B.make_params(moduli, w.scale_idx, n_out, w.seed)
    y = torch.empty(n_out, dtype=torch.int64, device="cuda")
    bad = torch.zeros(1, dtype=torch.int64, device="cuda")
    B.redash_decode(gp_out, Y, Zo, offsets, y, bad)
    torch.cuda.synchronize()
    assert int(bad.item()) == 0
    assert np.array_equal(y.cpu().numpy(), WL.make_inputs(w))
    # sampled output labels against the oracle, item by item
    rng = np.random.default_rng(w.seed + 99)
    items = np.unique(np.concatenate([np.arange(8), np.arange(n_out - 8, n_out),
                                      rng.choice(n_out, size=min(n_sample, n_out), replace=False)]))
    # the oracle needs the input labels of the receptive fields: fetch the whole input tensor
    Xh = H.to_u32(X)
    exp = OL.conv_labels_sampled(moduli, Xh, shape, wt.reshape(kshape).astype(np.int64),
                                 1 if w.kind == "fc" else w.stride, 0 if w.kind == "fc" else w.pad, items)
    li = H.label_index(moduli, n_out, items)
    assert np.array_equal(H.gather(Y, li), exp)


def test_full_size_batched_map_layer():
    """The 3x3x64 convolution producing the 16x64x56x56 batched map (12 primes)."""
    _check_full_layer(WL.BATCHED, 48)


@pytest.mark.parametrize("layer", [WL.RESNET18[0], WL.RESNET18[5], WL.RESNET18[7], WL.RESNET18[16],
                                   WL.RESNET18[-1]], ids=lambda w: w.name)
def test_full_size_resnet18_layer(layer):
    _check_full_layer(layer, 24)


def test_full_size_several_chunks_one_workgroup_per_modulus():
    """Two images of ResNet-18's 128-channel 28x28 layer: a grid large enough
    (2,688 workgroups) that the several-chunk contraction gives each modulus
    one workgroup; the batch-1 layers above give each packed word one."""
    w = WL._conv("l2.b-batch2", WL.PRIMES_12, (11,), 31, (2, 128, 28, 28), 128, 3, 1, 1)
    _check_full_layer(w, 24)


# ---------------------------------------------------------------------------
# a layer feeding the scaling gadget: the gadget is garbled on the layer's
# output zero-labels (redash_garble_scale_given), evaluated on its output
# labels, and decodes to floor((W x + b + r)/s)
# ---------------------------------------------------------------------------

def _scaled(x, moduli, S):
    s_ = 1
    for i in S:
        s_ *= moduli[i]
    P = 1
    for m in moduli:
        P *= m
    return np.floor_divide(np.asarray(x, np.int64) + (P // 2) % s_, s_)


CHAIN = [
    # name, moduli, S, (batch, c_in, h, w), c_out, k, stride, pad
    ("12primes-conv3x3", tuple(WL.PRIMES_12), (10, 11), (2, 9, 7, 6), 5, 3, 1, 1),
    ("short-base-dense", WL.SHORT_F.moduli, WL.SHORT_F.scale_idx, (40, 70, 1, 1), 9, 1, 1, 0),
    ("pow2-conv-stride2", (3, 5, 7, 11, 32), (4,), (1, 6, 9, 8), 4, 3, 2, 1),
]


def _random_chain(count: int, seed: int):
    """Seeded random layer-then-gadget cases: bases of 2 to 8 moduli with
    P > 2^26 (the layer's outputs, at most 9 * 7 * 7 * 8 * 20 + 100 in size,
    stay inside the signed range), a random scaling set, a random square
    kernel, stride and padding."""
    from oracle import rns

    rng = np.random.default_rng(seed)
    pool = [m for m in range(2, 256) if rns.is_prime(m) or (m & (m - 1)) == 0]
    out = []
    while len(out) < count:
        k = int(rng.integers(2, 9))
        base = sorted(int(m) for m in rng.choice(pool, size=k, replace=False))
        P = rns.cardinality(base)
        if sum(1 for m in base if m % 2 == 0) > 1 or not (1 << 26) < P < (1 << 63):
            continue
        t = int(rng.integers(1, k))
        S = tuple(sorted(int(i) for i in rng.choice(k, size=t, replace=False)))
        ks = int(rng.integers(1, 4))
        shape = (int(rng.integers(1, 3)), int(rng.integers(1, 10)), int(rng.integers(ks, 8)), int(rng.integers(ks, 8)))
        out.append((f"rand{len(out)}-k{k}-t{t}", tuple(base), S, shape, int(rng.integers(1, 7)), ks,
                    int(rng.integers(1, 3)), int(rng.integers(0, ks))))
    return out


CHAIN += _random_chain(4, 5150)


@pytest.mark.parametrize("case", CHAIN, ids=[c[0] for c in CHAIN])
def test_layer_feeds_gadget_matches_oracle(case):
    from oracle import oracle as O

    name, moduli, S, shape, c_out, k, stride, pad = case
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    seed, n_in = 31, int(np.prod(shape))
    x = rng.integers(-8, 9, size=shape)
    wts = rng.integers(-20, 21, size=(c_out, shape[1], k, k))
    bias = rng.integers(-100, 101, size=c_out)
    out_shape = OL.conv_out_shape(*shape, c_out, k, k, stride, pad)
    n_out = int(np.prod(out_shape))
    a0 = n_in  # the layer-output gadgets follow the input gadgets: distinct tweaks
    # oracle chain
    op_in = O.make_params(list(moduli), list(S), n_in, seed)
    offs, zin, _z, _t = O.garble(op_in, 0, n_in, with_tables=False)
    Xo = O.encode(op_in, x.reshape(-1), zin, offs)
    Yo = OL.conv_labels(moduli, Xo, shape, wts, stride, pad)
    Zo = OL.garble_conv(moduli, zin, shape, wts, bias, offs, stride, pad)
    op = O.make_params(list(moduli), list(S), n_out, seed)
    _o, gz_exp, tab_exp = O.garble_given(op, a0, n_out, Zo)
    out_exp = O.evaluate(op, a0, n_out, Yo, tab_exp)
    # GPU chain
    gp_in = B.make_params(moduli, S, n_in, seed)
    g = B.Buffers(gp_in)
    B.redash_garble_scale(gp_in, g.offsets, g.in_zero, g.out_zero, g.tables, g.work)
    B.redash_encode(gp_in, torch.from_numpy(x.reshape(-1).astype(np.int64)).cuda(), g.in_zero, g.offsets,
                    g.in_labels)
    lp = B.make_linear_params(moduli, *shape, c_out, k, k, stride, pad)
    sz = B.redash_linear_plan(lp)
    prep, work = _dev_u8(sz["prepared_bytes"]), _dev_u8(sz["work_bytes"])
    B.redash_linear_prepare(lp, H.to_dev(wts.astype(np.int32)), prep)
    Y = torch.empty(sz["out_label_words"], dtype=torch.int32, device="cuda")
    Z = torch.empty(sz["out_label_words"], dtype=torch.int32, device="cuda")
    B.redash_linear_eval(lp, g.in_labels, prep, work, Y)
    B.redash_linear_garble(lp, g.in_zero, prep, H.to_dev(bias.astype(np.int64)), g.offsets, work, Z)
    gp = B.make_params(moduli, S, n_out, seed, a0)
    gb = B.Buffers(gp)
    B.redash_garble_scale_given(gp, gb.offsets, Z, gb.out_zero, gb.tables, gb.work)
    B.redash_eval_scale(gp, Y, gb.tables, gb.out_labels, gb.work)
    B.redash_decode(gp, gb.out_labels, gb.out_zero, gb.offsets, gb.y, gb.bad)
    torch.cuda.synchronize()
    assert np.array_equal(H.to_u32(gb.offsets), offs)
    assert np.array_equal(H.to_u32(Z), Zo) and np.array_equal(H.to_u32(Y), Yo)
    assert np.array_equal(H.to_u32(gb.out_zero), gz_exp)
    assert np.array_equal(H.to_u32(gb.tables)[: len(tab_exp)], tab_exp)
    assert np.array_equal(H.to_u32(gb.out_labels), out_exp)
    # the decoded value, from the plain integer convolution
    lin = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(wts).double(),
                                     torch.from_numpy(bias).double(), stride=stride, padding=pad)
    assert int(gb.bad.item()) == 0
    assert np.array_equal(gb.y[:n_out].cpu().numpy(), _scaled(lin.numpy().reshape(-1).astype(np.int64), moduli, S))


def test_full_size_batched_map_layer_feeds_gadget():
    """The 3x3x64 layer of the 16x64x56x56 batched map, then the scaling
    gadget on its 3.2M outputs: every output decodes to floor((conv + r)/s)."""
    w = WL.BATCHED
    _shape, _ks, _wt, X, Y, Zo, offsets = _run_full_layer(w)
    del X
    torch.cuda.empty_cache()
    n_in = int(np.prod(w.in_shape))
    gp = B.make_params(w.moduli, w.scale_idx, w.n, w.seed, n_in)
    gb = B.Buffers(gp)
    B.redash_garble_scale_given(gp, gb.offsets, Zo, gb.out_zero, gb.tables, gb.work)
    B.redash_eval_scale(gp, Y, gb.tables, gb.out_labels, gb.work)
    B.redash_decode(gp, gb.out_labels, gb.out_zero, gb.offsets, gb.y, gb.bad)
    torch.cuda.synchronize()
    assert np.array_equal(H.to_u32(gb.offsets), H.to_u32(offsets))
    assert int(gb.bad.item()) == 0
    assert np.array_equal(gb.y.cpu().numpy(), _scaled(WL.make_inputs(w), w.moduli, w.scale_idx))
