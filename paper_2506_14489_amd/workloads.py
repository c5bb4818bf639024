"""Seeded synthetic workloads for the scaling gadget.

This module holds only configuration data and seeded input generators; it
contains none of the gadget's arithmetic.  It is shared by the tests, the
benchmark and the oracle-side checks, and is the only code the HIP path and
the oracle have in common.

Activations are signed integers x in the signed range of Z_P.  The paper
measures on CIFAR-10 CNNs with trained weights (Sec. 4, Table 3); those are
not available, and the gadget's cost does not depend on the values, so the
workloads are synthetic with the shapes and value ranges of CNN layers:

* tiny     : 1,024 values uniform in [-P/2, P/2), P = 2310, s = 11
* dense    : 4,096 values uniform in the signed range of Z_{P/19},
             P = 9,699,690, s = 19 (outputs of a previous P/19-scaled layer)
* conv     : 64x32x32 outputs of an exact integer 3x3x64 convolution of int8
             activations with int8 weights (stride 1, zero padding 1),
             10 primes, s = 23*29
* batched  : the same recipe over a 16x64x56x56 map, 12 primes, s = 37
* resnet18 : one gadget after each of the 21 conv/fc layers of a ResNet-18 at
             224x224 (stem, 16 block convs, 3 downsample convs, fc), each
             layer's output drawn from int8 inputs and weights of that layer's
             shape; s cycles 37, 31*37, 29; per-layer seeds 10..30

The short and power-of-two bases of Sec. 4, each scaled by its power of two
(ScaleQuant+ with s = 2^l), with 2^14 values uniform in the signed range of
Z_P (the size of the paper's gadget micro-benchmark); P/(2s) is not an
integer for any of them:

* cpm8-8, cpm8-32 : the first 8 primes with 2 replaced by 2^3 or 2^5
                    (the micro-benchmark bases), seeds 40, 41
* short-f         : (32, 167, 173), the short base of model f, seed 42
* short-F         : (32, 97, 107), the short base of model F, seed 43
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

PRIMES_12 = [2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37]


@dataclass(frozen=True)
class Workload:
    name: str
    moduli: tuple
    scale_idx: tuple
    n: int
    seed: int
    kind: str                      # "uniform" | "conv" | "fc"
    low: int = 0                   # uniform: inclusive low
    high: int = 0                  # uniform: exclusive high
    in_shape: tuple = ()           # conv: NCHW input shape; fc: (batch, in)
    w_shape: tuple = ()            # conv: (out, in, kh, kw); fc: (out, in)
    stride: int = 1
    pad: int = 0
    out_shape: tuple = field(default=())

    @property
    def P(self) -> int:
        P = 1
        for m in self.moduli:
            P *= m
        return P

    @property
    def s(self) -> int:
        s = 1
        for i in self.scale_idx:
            s *= self.moduli[i]
        return s


def _conv(name, moduli, scale_idx, seed, in_shape, cout, ksize, stride, pad):
    n_, c_, h_, w_ = in_shape
    ho = (h_ + 2 * pad - ksize) // stride + 1
    wo = (w_ + 2 * pad - ksize) // stride + 1
    out_shape = (n_, cout, ho, wo)
    return Workload(name, tuple(moduli), tuple(scale_idx), n_ * cout * ho * wo, seed, "conv",
                    in_shape=tuple(in_shape), w_shape=(cout, c_, ksize, ksize), stride=stride,
                    pad=pad, out_shape=out_shape)


TINY = Workload("tiny", tuple(PRIMES_12[:5]), (4,), 1024, 0, "uniform", -1155, 1155)
DENSE = Workload("dense", tuple(PRIMES_12[:8]), (7,), 4096, 1, "uniform", -255255, 255255)
CONV = _conv("conv", PRIMES_12[:10], (8, 9), 2, (1, 64, 32, 32), 64, 3, 1, 1)
BATCHED = _conv("batched", PRIMES_12, (11,), 3, (16, 64, 56, 56), 64, 3, 1, 1)

CONFIGS = [TINY, DENSE, CONV, BATCHED]


def _signed_uniform(name, moduli, scale_idx, n, seed):
    P = 1
    for m in moduli:
        P *= m
    return Workload(name, tuple(moduli), tuple(scale_idx), n, seed, "uniform", -(P // 2), P - P // 2)


CPM8_8 = _signed_uniform("cpm8-8", (3, 5, 7, 8, 11, 13, 17, 19), (3,), 1 << 14, 40)
CPM8_32 = _signed_uniform("cpm8-32", (3, 5, 7, 11, 13, 17, 19, 32), (7,), 1 << 14, 41)
SHORT_F = _signed_uniform("short-f", (32, 167, 173), (0,), 1 << 14, 42)
SHORT_BIG_F = _signed_uniform("short-F", (32, 97, 107), (0,), 1 << 14, 43)

SHORT_BASES = [CPM8_8, CPM8_32, SHORT_F, SHORT_BIG_F]


def at_size(w: Workload, n: int) -> Workload:
    """A uniform workload with n values instead of w.n (same base, seed and range)."""
    if w.kind != "uniform":
        raise ValueError("only uniform workloads can be resized")
    return Workload(w.name, w.moduli, w.scale_idx, n, w.seed, w.kind, w.low, w.high)


def resnet18_layers():
    """The 21 scaled layers of a ResNet-18 at 224x224, batch 1, in forward
    order, with per-layer seeds 10..30 and s cycling 37, 31*37, 29."""
    scale_cycle = [(11,), (10, 11), (9,)]
    specs = [("stem", (1, 3, 224, 224), 64, 7, 2, 3)]
    c, hw = 64, 56
    for stage, cout in enumerate([64, 128, 256, 512]):
        first_stride = 1 if stage == 0 else 2
        hw_out = hw // first_stride
        specs.append((f"l{stage + 1}.0.a", (1, c, hw, hw), cout, 3, first_stride, 1))
        specs.append((f"l{stage + 1}.0.b", (1, cout, hw_out, hw_out), cout, 3, 1, 1))
        if stage > 0:
            specs.append((f"l{stage + 1}.0.down", (1, c, hw, hw), cout, 1, 2, 0))
        specs.append((f"l{stage + 1}.1.a", (1, cout, hw_out, hw_out), cout, 3, 1, 1))
        specs.append((f"l{stage + 1}.1.b", (1, cout, hw_out, hw_out), cout, 3, 1, 1))
        c, hw = cout, hw_out
    layers = []
    for ell, (name, ins, cout, ks, st, pd) in enumerate(specs):
        layers.append(_conv(f"resnet18.{name}", PRIMES_12, scale_cycle[ell % 3], 10 + ell, ins, cout,
                            ks, st, pd))
    ell = len(specs)
    layers.append(Workload("resnet18.fc", tuple(PRIMES_12), scale_cycle[ell % 3], 1000, 10 + ell, "fc",
                           in_shape=(1, 512), w_shape=(1000, 512), out_shape=(1, 1000)))
    return layers


RESNET18 = resnet18_layers()


def by_name(name: str) -> Workload:
    for w in CONFIGS + RESNET18 + SHORT_BASES:
        if w.name == name:
            return w
    raise KeyError(name)


def _exact_conv_int8(a: np.ndarray, w: np.ndarray, stride: int, pad: int) -> np.ndarray:
    """Exact integer convolution (no bias) via im2col and a float64 product.
    All partial sums are integers below 2^53, so float64 is exact in any
    summation order."""
    import torch

    at = torch.from_numpy(a.astype(np.float64))
    wt = torch.from_numpy(w.astype(np.float64))
    n, c, h, wd = a.shape
    cout, _, kh, kw = w.shape
    cols = torch.nn.functional.unfold(at, (kh, kw), padding=pad, stride=stride)  # n, c*kh*kw, L
    out = torch.matmul(wt.reshape(cout, -1), cols)                             # n, cout, L
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (wd + 2 * pad - kw) // stride + 1
    res = out.reshape(n, cout, ho, wo).numpy()
    xi = np.rint(res).astype(np.int64)
    assert np.array_equal(xi.astype(np.float64), res)
    return xi


def layer_operands(w: Workload):
    """The int8 input activations (in_shape) and int8 weights (w_shape) of a
    conv or fc workload: the operands of the linear layer whose outputs are
    the workload's activations."""
    if w.kind not in ("conv", "fc"):
        raise ValueError("only conv and fc workloads come from a layer")
    rng = np.random.default_rng(w.seed)
    a = rng.integers(-128, 128, size=w.in_shape, dtype=np.int8)
    wt = rng.integers(-128, 128, size=w.w_shape, dtype=np.int8)
    return a, wt


def make_inputs(w: Workload) -> np.ndarray:
    """The activations x (int64, flattened NCHW) of a workload."""
    rng = np.random.default_rng(w.seed)
    if w.kind == "uniform":
        x = rng.integers(w.low, w.high, size=w.n, dtype=np.int64)
    elif w.kind == "conv":
        a, wt = layer_operands(w)
        x = _exact_conv_int8(a, wt, w.stride, w.pad).reshape(-1)
    elif w.kind == "fc":
        a, wt = layer_operands(w)
        x = (a.astype(np.int64) @ wt.astype(np.int64).T).reshape(-1)
    else:  # pragma: no cover
        raise ValueError(w.kind)
    assert x.shape == (w.n,)
    half = w.P // 2
    # wrap into the signed range of Z_P (no value of these recipes needs it)
    x = ((x + half) % w.P) - half
    return x.astype(np.int64)
