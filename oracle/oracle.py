"""ctypes wrapper of the plain C oracle ``gc_oracle.c``.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module.  It never loads the
HIP library and the HIP library never loads it.

The wrapper only marshals numpy arrays; every step of the garbling,
evaluation and decoding arithmetic is in ``gc_oracle.c``.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "gc_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

MAXLAMBDA = 128


def build(force: bool = False) -> str:
    """Compile gc_oracle.c into liboracle.so (plain gcc, no tuning flags)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-shared", "-fPIC", "-o", tmp, SRC])
        os.replace(tmp, LIB)
    return LIB


class Params(ctypes.Structure):
    _fields_ = [
        ("k", ctypes.c_uint32),
        ("moduli", ctypes.c_uint32 * 16),
        ("t", ctypes.c_uint32),
        ("scale_idx", ctypes.c_uint32 * 16),
        ("n", ctypes.c_uint64),
        ("seed", ctypes.c_uint64),
    ]


def make_params(moduli, scale_idx, n, seed) -> Params:
    p = Params()
    p.k = len(moduli)
    for i, m in enumerate(moduli):
        p.moduli[i] = m
    p.t = len(scale_idx)
    for i, s in enumerate(scale_idx):
        p.scale_idx[i] = s
    p.n = n
    p.seed = seed
    return p


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build())
        u32p = ctypes.POINTER(ctypes.c_uint32)
        _lib.orc_lambda.restype = ctypes.c_uint32
        _lib.orc_words.restype = ctypes.c_uint32
        _lib.orc_hash.argtypes = [ctypes.c_uint32, ctypes.c_uint32, u32p, ctypes.c_uint32,
                                  ctypes.c_uint64, u32p]
        _lib.orc_hash_parts.argtypes = [ctypes.c_uint32, ctypes.c_uint32, u32p, ctypes.c_uint32,
                                        ctypes.c_uint64, u32p, u32p, u32p]
        _lib.orc_prg_value.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64, u32p]
        _lib.orc_prg_label.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64,
                                       ctypes.c_uint32, ctypes.c_int, u32p]
        _lib.orc_frac_digits.argtypes = [u32p, ctypes.c_int, u32p, ctypes.c_int, u32p]
        _lib.orc_garble.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64, ctypes.c_uint64,
                                    u32p, u32p, u32p, u32p]
        _lib.orc_garble_given.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64, ctypes.c_uint64,
                                          u32p, u32p, u32p, u32p]
        _lib.orc_encode.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64,
                                    ctypes.POINTER(ctypes.c_int64), u32p, u32p, u32p]
        _lib.orc_eval.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64, ctypes.c_uint64,
                                  u32p, u32p, u32p]
        _lib.orc_decode.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64, u32p, u32p, u32p,
                                    ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_uint8)]
        _lib.orc_trace.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64, ctypes.c_int64] + [u32p] * 11
        _lib.orc_sizes.argtypes = [ctypes.POINTER(Params), ctypes.c_uint64,
                                   ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint64),
                                   ctypes.POINTER(ctypes.c_uint32), ctypes.POINTER(ctypes.c_uint32)]
        _lib.orc_gate_list.argtypes = [ctypes.POINTER(Params)] + [u32p] * 5
    return _lib


def _p(a: np.ndarray, ctype=ctypes.c_uint32):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ctype))


class OracleError(RuntimeError):
    pass


def _check(rc: int):
    if rc != 0:
        raise OracleError(f"oracle returned {rc}")


def lam(m: int) -> int:
    return lib().orc_lambda(m)


def words(m: int) -> int:
    return lib().orc_words(m)


def sizes(params: Params, n: int):
    lw, tw = ctypes.c_uint64(), ctypes.c_uint64()
    g, ow = ctypes.c_uint32(), ctypes.c_uint32()
    _check(lib().orc_sizes(ctypes.byref(params), n, ctypes.byref(lw), ctypes.byref(tw),
                           ctypes.byref(g), ctypes.byref(ow)))
    return {"label_words": lw.value, "table_words": tw.value, "gates": g.value, "offset_words": ow.value}


def check_params(params: Params) -> int:
    return lib().orc_check_params(ctypes.byref(params))


def gate_list(params: Params):
    G = sizes(params, 1)["gates"]
    arrs = [np.zeros(G, np.uint32) for _ in range(5)]
    _check(lib().orc_gate_list(ctypes.byref(params), *[_p(a) for a in arrs]))
    return [tuple(int(a[g]) for a in arrs) for g in range(G)]


def aes128(key: bytes, block: bytes) -> bytes:
    out = (ctypes.c_uint8 * 16)()
    lib().orc_aes128((ctypes.c_uint8 * 16)(*key), (ctypes.c_uint8 * 16)(*block), out)
    return bytes(out)


def aes128_key_expansion(key: bytes) -> bytes:
    out = (ctypes.c_uint8 * 176)()
    lib().orc_aes128_key_expansion((ctypes.c_uint8 * 16)(*key), out)
    return bytes(out)


def sbox() -> bytes:
    out = (ctypes.c_uint8 * 256)()
    lib().orc_sbox(out)
    return bytes(out)


def frac_digits(V_limbs, radices):
    V = np.array(V_limbs, dtype=np.uint32)
    r = np.array(radices, dtype=np.uint32)
    out = np.zeros(len(r), np.uint32)
    lib().orc_frac_digits(_p(V), len(V), _p(r), len(r), _p(out))
    return out


def pk32_pack(m: int, res) -> np.ndarray:
    r = np.zeros(MAXLAMBDA, np.uint32)
    r[: len(res)] = res
    w = np.zeros(MAXLAMBDA, np.uint32)
    lib().orc_pk32_pack(ctypes.c_uint32(m), _p(r), _p(w))
    return w[: words(m)].copy()


def pk32_unpack(m: int, wrds) -> np.ndarray:
    w = np.zeros(MAXLAMBDA, np.uint32)
    w[: len(wrds)] = wrds
    r = np.zeros(MAXLAMBDA, np.uint32)
    lib().orc_pk32_unpack(ctypes.c_uint32(m), _p(w), _p(r))
    return r[: lam(m)].copy()


def hash_label(q: int, m: int, A, gadget_id: int, tau: int) -> np.ndarray:
    a = np.zeros(MAXLAMBDA, np.uint32)
    a[: len(A)] = A
    out = np.zeros(MAXLAMBDA, np.uint32)
    lib().orc_hash(q, m, _p(a), gadget_id, tau, _p(out))
    return out[: lam(m)].copy()


def hash_parts(q: int, m: int, A, gadget_id: int, tau: int):
    """(x, u, V) of the hash: the fold of the packed label (4 lanes), sigma of
    it (4 lanes) and the hash value before digit extraction (8 limbs; the top
    4 are 0 when m = 2)."""
    a = np.zeros(MAXLAMBDA, np.uint32)
    a[: len(A)] = A
    x, u, V = np.zeros(4, np.uint32), np.zeros(4, np.uint32), np.zeros(8, np.uint32)
    lib().orc_hash_parts(q, m, _p(a), gadget_id, tau, _p(x), _p(u), _p(V))
    return x, u, V


def prg_value(seed: int, stream: int, idx: int) -> np.ndarray:
    """rho(stream, idx) of the garbler PRG as 8 little-endian 32-bit limbs."""
    V = np.zeros(8, np.uint32)
    lib().orc_prg_value(seed, stream, idx, _p(V))
    return V


def prg_label(seed: int, stream: int, idx: int, m: int, first_minus_one: bool) -> np.ndarray:
    out = np.zeros(MAXLAMBDA, np.uint32)
    lib().orc_prg_label(seed, stream, idx, m, int(first_minus_one), _p(out))
    return out[: lam(m)].copy()


def garble(params: Params, a_begin: int, count: int, with_tables: bool = True):
    """Returns (offsets, in_zero, out_zero, tables or None), stride = count."""
    sz = sizes(params, count)
    offsets = np.zeros(sz["offset_words"], np.uint32)
    zin = np.zeros(sz["label_words"], np.uint32)
    zout = np.zeros(sz["label_words"], np.uint32)
    tables = np.zeros(max(sz["table_words"], 1), np.uint32) if with_tables else None
    _check(lib().orc_garble(ctypes.byref(params), a_begin, count, _p(offsets), _p(zin), _p(zout),
                            _p(tables)))
    return offsets, zin, zout, tables


def garble_given(params: Params, a_begin: int, count: int, in_zero: np.ndarray, with_tables: bool = True):
    """Garble on the given input zero-labels (stride = count).  Returns
    (offsets, out_zero, tables or None)."""
    sz = sizes(params, count)
    offsets = np.zeros(sz["offset_words"], np.uint32)
    zin = np.ascontiguousarray(in_zero, dtype=np.uint32)
    assert len(zin) == sz["label_words"]
    zout = np.zeros(sz["label_words"], np.uint32)
    tables = np.zeros(max(sz["table_words"], 1), np.uint32) if with_tables else None
    _check(lib().orc_garble_given(ctypes.byref(params), a_begin, count, _p(offsets), _p(zin), _p(zout),
                                  _p(tables)))
    return offsets, zout, tables


def encode(params: Params, x: np.ndarray, zero: np.ndarray, offsets: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.int64)
    out = np.zeros_like(zero)
    _check(lib().orc_encode(ctypes.byref(params), len(x), _p(x, ctypes.c_int64), _p(zero),
                            _p(offsets), _p(out)))
    return out


def evaluate(params: Params, a_begin: int, count: int, in_labels: np.ndarray, tables: np.ndarray):
    out = np.zeros_like(in_labels)
    _check(lib().orc_eval(ctypes.byref(params), a_begin, count, _p(in_labels), _p(tables), _p(out)))
    return out


def decode(params: Params, out_labels: np.ndarray, out_zero: np.ndarray, offsets: np.ndarray):
    k = params.k
    W = sum(words(params.moduli[i]) for i in range(k))
    count = len(out_labels) // W
    y = np.zeros(count, np.int64)
    bad = np.zeros(count, np.uint8)
    _check(lib().orc_decode(ctypes.byref(params), count, _p(out_labels), _p(out_zero), _p(offsets),
                            _p(y, ctypes.c_int64), _p(bad, ctypes.c_uint8)))
    return y, bad


def trace(params: Params, a: int, x: int):
    k = params.k
    G = sizes(params, 1)["gates"]
    L = MAXLAMBDA
    t = {
        "offsets": np.zeros((k, L), np.uint32),
        "gb_slots": np.zeros((G + 1, k, L), np.uint32),
        "ev_slots": np.zeros((G + 1, k, L), np.uint32),
        "gb_in": np.zeros((G, L), np.uint32),
        "ev_in": np.zeros((G, L), np.uint32),
        "gb_out": np.zeros((G, L), np.uint32),
        "ev_out": np.zeros((G, L), np.uint32),
        "gb_outR": np.zeros((k, L), np.uint32),
        "ev_outR": np.zeros((k, L), np.uint32),
        "gb_final": np.zeros((k, L), np.uint32),
        "ev_final": np.zeros((k, L), np.uint32),
    }
    order = ["offsets", "gb_slots", "ev_slots", "gb_in", "ev_in", "gb_out", "ev_out", "gb_outR",
             "ev_outR", "gb_final", "ev_final"]
    _check(lib().orc_trace(ctypes.byref(params), a, x, *[_p(t[n]) for n in order]))
    return t


def label_view(buf: np.ndarray, params: Params, count: int, i: int) -> np.ndarray:
    """Words of modulus i of a label tensor with stride ``count``: shape (W_i, count)."""
    off = 0
    for j in range(i):
        off += words(params.moduli[j]) * count
    W = words(params.moduli[i])
    return buf[off: off + W * count].reshape(W, count)
