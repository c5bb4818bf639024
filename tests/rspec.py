"""A second statement of the garbling hash and PRG, in Python integers, for
the tests that pin the C oracle's ``hash_label`` and ``prg_label``.

The paper fixes the algebra of the projection gates (Sec. 2.3) but no hash,
PRG, tweak or bit convention; the library and the oracle follow one
specification of their own.  This module restates that specification
directly on integers, with AES-128 taken from the system libcrypto (an
implementation that shares nothing with the oracle's FIPS-197 code):

* labels over Z_q are packed PK32: residue i at bit b*(i mod g) of word
  i // g, b = bit length of q-1, g = 32 // b;
* fold: word w of the packed label is XORed into 32-bit lane w mod 4 of a
  128-bit integer X (lane 0 = bits 0-31);
* sigma(X) = ((X_hi xor X_lo) << 64) | X_hi with X_lo, X_hi the low and high
  64-bit halves (the linear orthomorphism of Guo, Katz, Wang and Yu, 2020);
* tweak T_j = gadget_id * 2^96 + ((4 tau + j) mod 2^64), j < n, n = 1 for an
  output modulus 2 and 2 otherwise;
* U_j = AES_K(u xor T_j) xor u xor T_j with K = 00 01 ... 0f, 128-bit integers
  entering AES as 16 little-endian bytes;
* V = sum_j U_j 2^(128 j); the output label is the first lambda_m base-m
  digits of the fraction V / 2^(128 n);
* PRG: K_seed = the 64-bit seed as 16 little-endian bytes,
  rho(stream, idx) = AES(C_0) + 2^128 AES(C_1),
  C_h = stream * 2^120 + ((2 idx + h) mod 2^64).

Nothing here is imported by the library or by the oracle.
"""

from __future__ import annotations

import ctypes
import ctypes.util

M64 = (1 << 64) - 1
M128 = (1 << 128) - 1
HASH_KEY = bytes(range(16))


class LibCrypto:
    """AES-128 in ECB mode through libcrypto's EVP interface."""

    def __init__(self):
        name = ctypes.util.find_library("crypto")
        if not name:
            raise OSError("libcrypto not found")
        lc = ctypes.CDLL(name)
        lc.EVP_CIPHER_CTX_new.restype = ctypes.c_void_p
        lc.EVP_aes_128_ecb.restype = ctypes.c_void_p
        lc.EVP_EncryptInit_ex.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_char_p, ctypes.c_char_p]
        lc.EVP_CIPHER_CTX_set_padding.argtypes = [ctypes.c_void_p, ctypes.c_int]
        lc.EVP_EncryptUpdate.argtypes = [ctypes.c_void_p, ctypes.c_char_p, ctypes.POINTER(ctypes.c_int),
                                         ctypes.c_char_p, ctypes.c_int]
        lc.EVP_CIPHER_CTX_free.argtypes = [ctypes.c_void_p]
        self.lc = lc

    def encrypt(self, key: bytes, block: bytes) -> bytes:
        lc = self.lc
        ctx = lc.EVP_CIPHER_CTX_new()
        try:
            assert lc.EVP_EncryptInit_ex(ctx, lc.EVP_aes_128_ecb(), None, key, None) == 1
            lc.EVP_CIPHER_CTX_set_padding(ctx, 0)
            out = ctypes.create_string_buffer(32)
            n = ctypes.c_int(0)
            assert lc.EVP_EncryptUpdate(ctx, out, ctypes.byref(n), block, 16) == 1
            return out.raw[:16]
        finally:
            lc.EVP_CIPHER_CTX_free(ctx)

    def aes_int(self, key: bytes, x: int) -> int:
        """AES_K of a 128-bit integer given as little-endian bytes."""
        return int.from_bytes(self.encrypt(key, (x & M128).to_bytes(16, "little")), "little")


def lam(m: int) -> int:
    """Least lambda with m^lambda >= 2^128."""
    lam_, p = 0, 1
    while p < (1 << 128):
        p *= m
        lam_ += 1
    return lam_


def pack(m: int, residues) -> list[int]:
    b = (m - 1).bit_length()
    g = 32 // b
    W = -(-lam(m) // g)
    words = [0] * W
    for i, r in enumerate(residues):
        words[i // g] |= int(r) << (b * (i % g))
    return words


def fold(words) -> int:
    lanes = [0, 0, 0, 0]
    for w, v in enumerate(words):
        lanes[w % 4] ^= int(v)
    return sum(l << (32 * i) for i, l in enumerate(lanes))


def sigma(x: int) -> int:
    lo, hi = x & M64, x >> 64
    return ((hi ^ lo) << 64) | hi


def tweak(gadget_id: int, tau: int, j: int) -> int:
    return (gadget_id << 96) | ((4 * tau + j) & M64)


def hash_value(aes: LibCrypto, q: int, m: int, residues, gadget_id: int, tau: int) -> int:
    u = sigma(fold(pack(q, residues)))
    n = 1 if m == 2 else 2
    V = 0
    for j in range(n):
        t = tweak(gadget_id, tau, j)
        V |= (aes.aes_int(HASH_KEY, u ^ t) ^ u ^ t) << (128 * j)
    return V


def frac_digits(V: int, bits: int, radices) -> list[int]:
    """Digits of the fraction V / 2^bits in the given radices, most
    significant first."""
    out = []
    for r in radices:
        V *= r
        out.append(V >> bits)
        V &= (1 << bits) - 1
    return out


def hash_label(aes: LibCrypto, q: int, m: int, residues, gadget_id: int, tau: int) -> list[int]:
    n = 1 if m == 2 else 2
    V = hash_value(aes, q, m, residues, gadget_id, tau)
    return frac_digits(V, 128 * n, [m] * lam(m))


def prg_value(aes: LibCrypto, seed: int, stream: int, idx: int) -> int:
    key = (seed & M64).to_bytes(16, "little")
    V = 0
    for h in range(2):
        c = (stream << 120) | ((2 * idx + h) & M64)
        V |= aes.aes_int(key, c) << (128 * h)
    return V


def is_pow2(m: int) -> bool:
    return m >= 2 and m & (m - 1) == 0


def offset(aes: LibCrypto, seed: int, i: int, m: int) -> list[int]:
    """R_m of base modulus index i: digits of rho(1, i) in the radices
    (r0, m, m, ...), then residue 0 mapped to a unit of Z_m (d + 1 with
    r0 = m - 1 for a prime, 2d + 1 with r0 = m / 2 for a power of two above 2)."""
    pw = is_pow2(m) and m > 2
    r0 = m // 2 if pw else m - 1
    d = frac_digits(prg_value(aes, seed, 1, i), 256, [r0] + [m] * (lam(m) - 1))
    d[0] = 2 * d[0] + 1 if pw else d[0] + 1
    return d


def zero_label(aes: LibCrypto, seed: int, a: int, i: int, k: int, m: int) -> list[int]:
    """Input zero-label of base modulus index i of gadget a: digits of
    rho(2, a k + i) in radix m."""
    return frac_digits(prg_value(aes, seed, 2, a * k + i), 256, [m] * lam(m))
