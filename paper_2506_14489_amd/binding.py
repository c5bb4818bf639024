"""Python binding of libredash.so (the C ABI in include/redash.h).

Argument marshalling only: every step of garbling, evaluation, encoding and
decoding runs in the library's HIP kernels.  PyTorch supplies device memory
(int32 CUDA tensors holding the uint32 words, int64 tensors for values) and
the stream (torch's current stream unless one is given).

There is no fallback: if the library is not built, or a call returns an
error, a ``RedashError`` is raised.
"""

from __future__ import annotations

import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libredash.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "redash.h")

REDASH_OK = 0
REDASH_E_PARAM = -1
REDASH_E_NULL = -2
REDASH_E_HIP = -3
REDASH_E_LABEL = -4
REDASH_E_SIZE = -5
NOALLOC_WORK_WORDS = 16 << 20  # REDASH_NOALLOC_WORK_WORDS


class RedashError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {strerror(code)} ({code})")
        self.code = code


class Params(ctypes.Structure):
    """Mirror of ``redash_params``."""

    _fields_ = [
        ("k", ctypes.c_uint32),
        ("moduli", ctypes.c_uint32 * 16),
        ("t", ctypes.c_uint32),
        ("scale_idx", ctypes.c_uint32 * 16),
        ("n", ctypes.c_uint64),
        ("seed", ctypes.c_uint64),
        ("a0", ctypes.c_uint64),
    ]


class Sizes(ctypes.Structure):
    """Mirror of ``redash_sizes``."""

    _fields_ = [
        ("label_words", ctypes.c_uint64),
        ("table_words", ctypes.c_uint64),
        ("offset_words", ctypes.c_uint32),
        ("gates", ctypes.c_uint32),
        ("work_words", ctypes.c_uint64),
    ]


def make_params(moduli, scale_idx, n: int, seed: int, a0: int = 0) -> Params:
    p = Params()
    p.k = len(moduli)
    for i, m in enumerate(moduli):
        p.moduli[i] = int(m)
    p.t = len(scale_idx)
    for i, s in enumerate(scale_idx):
        p.scale_idx[i] = int(s)
    p.n = int(n)
    p.seed = int(seed)
    p.a0 = int(a0)
    return p


class LinearParams(ctypes.Structure):
    """Mirror of ``redash_linear_params``."""

    _fields_ = [
        ("k", ctypes.c_uint32),
        ("moduli", ctypes.c_uint32 * 16),
        ("batch", ctypes.c_uint32),
        ("c_in", ctypes.c_uint32),
        ("h_in", ctypes.c_uint32),
        ("w_in", ctypes.c_uint32),
        ("c_out", ctypes.c_uint32),
        ("kh", ctypes.c_uint32),
        ("kw", ctypes.c_uint32),
        ("stride", ctypes.c_uint32),
        ("pad", ctypes.c_uint32),
    ]


class LinearSizes(ctypes.Structure):
    """Mirror of ``redash_linear_sizes``."""

    _fields_ = [
        ("in_label_words", ctypes.c_uint64),
        ("out_label_words", ctypes.c_uint64),
        ("prepared_bytes", ctypes.c_uint64),
        ("work_bytes", ctypes.c_uint64),
        ("h_out", ctypes.c_uint32),
        ("w_out", ctypes.c_uint32),
        ("offset_words", ctypes.c_uint32),
    ]


def make_linear_params(moduli, batch, c_in, h_in, w_in, c_out, kh=1, kw=1, stride=1, pad=0) -> LinearParams:
    """A conv2d layer (NCHW input, OIHW weights); a dense layer is
    h_in = w_in = kh = kw = 1."""
    p = LinearParams()
    p.k = len(moduli)
    for i, m in enumerate(moduli):
        p.moduli[i] = int(m)
    p.batch, p.c_in, p.h_in, p.w_in = int(batch), int(c_in), int(h_in), int(w_in)
    p.c_out, p.kh, p.kw, p.stride, p.pad = int(c_out), int(kh), int(kw), int(stride), int(pad)
    return p


_lib = None


def lib() -> ctypes.CDLL:
    """Load libredash.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2506_14489_amd.build` "
                "(there is no fallback implementation)")
        L = ctypes.CDLL(LIB_PATH)
        vp = ctypes.c_void_p
        pp = ctypes.POINTER(Params)
        L.redash_plan.argtypes = [pp, ctypes.POINTER(Sizes)]
        L.redash_garble_scale.argtypes = [pp, vp, vp, vp, vp, vp, vp]
        L.redash_garble_scale_given.argtypes = [pp, vp, vp, vp, vp, vp, vp]
        L.redash_encode.argtypes = [pp, vp, vp, vp, vp, vp]
        L.redash_eval_scale.argtypes = [pp, vp, vp, vp, vp, vp]
        L.redash_eval_scale_noalloc.argtypes = [pp, vp, vp, vp, vp]
        L.redash_decode.argtypes = [pp, vp, vp, vp, vp, vp, vp]
        L.redash_hash_labels.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64, vp, ctypes.c_uint32,
                                         vp, vp, vp]
        L.redash_aes_ctr.argtypes = [ctypes.c_uint64, ctypes.c_uint64, vp, vp]
        L.redash_aes_ctr_bitsliced.argtypes = [ctypes.c_uint64, ctypes.c_uint64, vp, vp]
        L.redash_strerror.argtypes = [ctypes.c_int]
        L.redash_strerror.restype = ctypes.c_char_p
        lp = ctypes.POINTER(LinearParams)
        L.redash_linear_plan.argtypes = [lp, ctypes.POINTER(LinearSizes)]
        L.redash_linear_prepare.argtypes = [lp, vp, vp, vp]
        L.redash_linear_eval.argtypes = [lp, vp, vp, vp, vp, vp]
        L.redash_linear_garble.argtypes = [lp, vp, vp, vp, vp, vp, vp, vp]
        for name in ("redash_plan", "redash_garble_scale", "redash_garble_scale_given", "redash_encode", "redash_eval_scale",
                     "redash_eval_scale_noalloc", "redash_decode",
                     "redash_hash_labels", "redash_aes_ctr", "redash_aes_ctr_bitsliced", "redash_linear_plan", "redash_linear_prepare", "redash_linear_eval",
                     "redash_linear_garble"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def declared_symbols() -> list[str]:
    """Names of the entry points declared in include/redash.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\s*\*|int)\s*(redash_\w+)\s*\(", text, re.M)))


def strerror(code: int) -> str:
    return lib().redash_strerror(int(code)).decode()


def _check(rc: int, what: str):
    if rc != REDASH_OK:
        raise RedashError(rc, what)


def _ptr(t, dtype, min_numel: int, what: str):
    """Device pointer of a contiguous CUDA tensor of the given dtype and size."""
    if t is None:
        return None
    import torch

    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{what}: expected a CUDA tensor")
    if t.dtype != dtype:
        raise TypeError(f"{what}: expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what}: tensor must be contiguous")
    if t.numel() < min_numel:
        raise ValueError(f"{what}: needs {min_numel} elements, has {t.numel()}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def redash_plan(params: Params) -> dict:
    s = Sizes()
    _check(lib().redash_plan(ctypes.byref(params), ctypes.byref(s)), "redash_plan")
    return {"label_words": s.label_words, "table_words": s.table_words, "offset_words": s.offset_words,
            "gates": s.gates, "work_words": s.work_words}


def plan_rc(params: Params) -> int:
    """Return code of redash_plan (no exception), for validation tests."""
    s = Sizes()
    return lib().redash_plan(ctypes.byref(params), ctypes.byref(s))


def redash_garble_scale(params, offsets, in_zero, out_zero, tables, work, stream=None):
    import torch

    sz = redash_plan(params)
    _check(lib().redash_garble_scale(
        ctypes.byref(params), _ptr(offsets, torch.int32, sz["offset_words"], "offsets"),
        _ptr(in_zero, torch.int32, sz["label_words"], "in_zero"),
        _ptr(out_zero, torch.int32, sz["label_words"], "out_zero"),
        _ptr(tables, torch.int32, sz["table_words"], "tables"),
        _ptr(work, torch.int32, sz["work_words"], "work"), _stream(stream)), "redash_garble_scale")


def redash_garble_scale_given(params, offsets, in_zero, out_zero, tables, work, stream=None):
    """Garble on the caller's input zero-labels (read only), e.g. a garbled
    linear layer's output zero-labels built on the same seed's offsets."""
    import torch

    sz = redash_plan(params)
    _check(lib().redash_garble_scale_given(
        ctypes.byref(params), _ptr(offsets, torch.int32, sz["offset_words"], "offsets"),
        _ptr(in_zero, torch.int32, sz["label_words"], "in_zero"),
        _ptr(out_zero, torch.int32, sz["label_words"], "out_zero"),
        _ptr(tables, torch.int32, sz["table_words"], "tables"),
        _ptr(work, torch.int32, sz["work_words"], "work"), _stream(stream)), "redash_garble_scale_given")


def redash_encode(params, x, in_zero, offsets, in_labels, stream=None):
    import torch

    sz = redash_plan(params)
    _check(lib().redash_encode(
        ctypes.byref(params), _ptr(x, torch.int64, params.n, "x"),
        _ptr(in_zero, torch.int32, sz["label_words"], "in_zero"),
        _ptr(offsets, torch.int32, sz["offset_words"], "offsets"),
        _ptr(in_labels, torch.int32, sz["label_words"], "in_labels"), _stream(stream)), "redash_encode")


def redash_eval_scale(params, in_labels, tables, out_labels, work, stream=None):
    import torch

    sz = redash_plan(params)
    _check(lib().redash_eval_scale(
        ctypes.byref(params), _ptr(in_labels, torch.int32, sz["label_words"], "in_labels"),
        _ptr(tables, torch.int32, sz["table_words"], "tables"),
        _ptr(out_labels, torch.int32, sz["label_words"], "out_labels"),
        _ptr(work, torch.int32, sz["work_words"], "work"), _stream(stream)), "redash_eval_scale")


def redash_eval_scale_noalloc(params, in_labels, tables, out_labels, stream=None):
    """redash_eval_scale on the library's fixed working buffer (no d_work)."""
    import torch

    sz = redash_plan(params)
    _check(lib().redash_eval_scale_noalloc(
        ctypes.byref(params), _ptr(in_labels, torch.int32, sz["label_words"], "in_labels"),
        _ptr(tables, torch.int32, sz["table_words"], "tables"),
        _ptr(out_labels, torch.int32, sz["label_words"], "out_labels"), _stream(stream)),
        "redash_eval_scale_noalloc")


def redash_decode(params, out_labels, out_zero, offsets, y, bad_count, stream=None):
    import torch

    sz = redash_plan(params)
    _check(lib().redash_decode(
        ctypes.byref(params), _ptr(out_labels, torch.int32, sz["label_words"], "out_labels"),
        _ptr(out_zero, torch.int32, sz["label_words"], "out_zero"),
        _ptr(offsets, torch.int32, sz["offset_words"], "offsets"), _ptr(y, torch.int64, params.n, "y"),
        _ptr(bad_count, torch.int64, 1, "bad_count"), _stream(stream)), "redash_decode")


def redash_hash_labels(q, m, count, labels, gadget_id, tau, out, stream=None):
    import torch

    wq, wm = label_words_of(q), label_words_of(m)
    _check(lib().redash_hash_labels(
        int(q), int(m), int(count), _ptr(labels, torch.int32, wq * count, "labels"), int(gadget_id) & 0xFFFFFFFF,
        _ptr(tau, torch.int64, count, "tau"), _ptr(out, torch.int32, wm * count, "out"), _stream(stream)),
        "redash_hash_labels")


def redash_aes_ctr(count, c0, out, stream=None):
    """AES-128 under the hash key in counter mode (the device's AES rate)."""
    import torch

    _check(lib().redash_aes_ctr(int(count), int(c0), _ptr(out, torch.int32, 4 * count, "out"), _stream(stream)),
           "redash_aes_ctr")


def redash_aes_ctr_bitsliced(count, c0, out, stream=None):
    """redash_aes_ctr from the bitsliced AES (the device's AES rate without tables)."""
    import torch

    _check(lib().redash_aes_ctr_bitsliced(int(count), int(c0), _ptr(out, torch.int32, 4 * count, "out"),
                                          _stream(stream)), "redash_aes_ctr_bitsliced")


def redash_linear_plan(params: LinearParams) -> dict:
    s = LinearSizes()
    _check(lib().redash_linear_plan(ctypes.byref(params), ctypes.byref(s)), "redash_linear_plan")
    return {"in_label_words": s.in_label_words, "out_label_words": s.out_label_words,
            "prepared_bytes": s.prepared_bytes, "work_bytes": s.work_bytes, "h_out": s.h_out, "w_out": s.w_out,
            "offset_words": s.offset_words}


def linear_plan_rc(params: LinearParams) -> int:
    """Return code of redash_linear_plan (no exception), for validation tests."""
    s = LinearSizes()
    return lib().redash_linear_plan(ctypes.byref(params), ctypes.byref(s))


def redash_linear_prepare(params, weights, prepared, stream=None):
    import torch

    sz = redash_linear_plan(params)
    nw = params.c_out * params.c_in * params.kh * params.kw
    _check(lib().redash_linear_prepare(
        ctypes.byref(params), _ptr(weights, torch.int32, nw, "weights"),
        _ptr(prepared, torch.uint8, sz["prepared_bytes"], "prepared"), _stream(stream)), "redash_linear_prepare")


def redash_linear_eval(params, in_labels, prepared, work, out_labels, stream=None):
    import torch

    sz = redash_linear_plan(params)
    _check(lib().redash_linear_eval(
        ctypes.byref(params), _ptr(in_labels, torch.int32, sz["in_label_words"], "in_labels"),
        _ptr(prepared, torch.uint8, sz["prepared_bytes"], "prepared"),
        _ptr(work, torch.uint8, sz["work_bytes"], "work"),
        _ptr(out_labels, torch.int32, sz["out_label_words"], "out_labels"), _stream(stream)), "redash_linear_eval")


def redash_linear_garble(params, in_zero, prepared, bias, offsets, work, out_zero, stream=None):
    import torch

    sz = redash_linear_plan(params)
    _check(lib().redash_linear_garble(
        ctypes.byref(params), _ptr(in_zero, torch.int32, sz["in_label_words"], "in_zero"),
        _ptr(prepared, torch.uint8, sz["prepared_bytes"], "prepared"),
        _ptr(bias, torch.int64, params.c_out, "bias"),
        _ptr(offsets, torch.int32, sz["offset_words"], "offsets"),
        _ptr(work, torch.uint8, sz["work_bytes"], "work"),
        _ptr(out_zero, torch.int32, sz["out_label_words"], "out_zero"), _stream(stream)), "redash_linear_garble")


def label_words_of(m: int) -> int:
    """W_m, read off redash_plan: the base (2, m) holds W_2 = 4 words (128
    one-bit residues) plus W_m; an even m is paired with 251 instead."""
    if m == 2:
        return 4
    if m % 2:
        return redash_plan(make_params([2, m], [1], 1, 0))["offset_words"] - 4
    return redash_plan(make_params([m, 251], [1], 1, 0))["offset_words"] - label_words_of(251)


class Buffers:
    """Device buffers of one gadget call, sized from redash_plan (int32 words)."""

    def __init__(self, params: Params, device="cuda", tables: bool = True):
        import torch

        sz = redash_plan(params)
        self.sizes = sz
        i32 = torch.int32
        self.offsets = torch.empty(sz["offset_words"], dtype=i32, device=device)
        self.in_zero = torch.empty(sz["label_words"], dtype=i32, device=device)
        self.out_zero = torch.empty(sz["label_words"], dtype=i32, device=device)
        self.in_labels = torch.empty(sz["label_words"], dtype=i32, device=device)
        self.out_labels = torch.empty(sz["label_words"], dtype=i32, device=device)
        self.tables = torch.empty(max(sz["table_words"], 1), dtype=i32, device=device) if tables else None
        self.work = torch.empty(max(sz["work_words"], 1), dtype=i32, device=device)
        self.y = torch.empty(max(params.n, 1), dtype=torch.int64, device=device)
        self.bad = torch.zeros(1, dtype=torch.int64, device=device)
