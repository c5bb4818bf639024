// Device helpers for gfx950: AES-128 on LDS round tables, the projection-gate
// hash, base-m digit extraction into packed labels, and residue arithmetic on
// packed 32-bit words.  All per-modulus quantities come from a ModConst that
// is uniform across the wavefront (it lives in the kernel argument block).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "aes_tables.hpp"
#include "plan.hpp"

namespace redash {

// The four round tables, copied into LDS by every block.
__device__ const Words1024 g_round_tables = kRoundTables;

constexpr int kTableWords = 1024;
constexpr int kMaxW = 6;  // largest W over moduli 2..255 (m = 3, 5, 17, 19)

__device__ __forceinline__ void stage_round_tables(uint32_t *lds_tables, int tid, int nthreads) {
    for (int i = tid; i < kTableWords; i += nthreads) lds_tables[i] = g_round_tables.v[i];
}

// ---------------------------------------------------------------------------
// AES-128 encryption of one block held as four little-endian column words.
// Rounds 1..9 use TE0..TE3; the last round takes each S-box byte from the
// table in which it already sits at the right byte position.
// ---------------------------------------------------------------------------
template <typename KeyFn>
__device__ __forceinline__ void aes128_encrypt(const uint32_t *__restrict__ T, uint32_t &s0, uint32_t &s1,
                                               uint32_t &s2, uint32_t &s3, KeyFn rk) {
    s0 ^= rk(0);
    s1 ^= rk(1);
    s2 ^= rk(2);
    s3 ^= rk(3);
#pragma unroll
    for (int r = 1; r < 10; ++r) {
        uint32_t t0 = T[s0 & 255] ^ T[256 + ((s1 >> 8) & 255)] ^ T[512 + ((s2 >> 16) & 255)] ^ T[768 + (s3 >> 24)];
        uint32_t t1 = T[s1 & 255] ^ T[256 + ((s2 >> 8) & 255)] ^ T[512 + ((s3 >> 16) & 255)] ^ T[768 + (s0 >> 24)];
        uint32_t t2 = T[s2 & 255] ^ T[256 + ((s3 >> 8) & 255)] ^ T[512 + ((s0 >> 16) & 255)] ^ T[768 + (s1 >> 24)];
        uint32_t t3 = T[s3 & 255] ^ T[256 + ((s0 >> 8) & 255)] ^ T[512 + ((s1 >> 16) & 255)] ^ T[768 + (s2 >> 24)];
        s0 = t0 ^ rk(4 * r);
        s1 = t1 ^ rk(4 * r + 1);
        s2 = t2 ^ rk(4 * r + 2);
        s3 = t3 ^ rk(4 * r + 3);
    }
    // S(x) sits in byte 0 of TE2/TE3, byte 1 of TE0/TE3, byte 2 of TE0/TE1, byte 3 of TE1/TE2.
    uint32_t o0 = (T[512 + (s0 & 255)] & 0xffu) | (T[768 + ((s1 >> 8) & 255)] & 0xff00u) |
                  (T[(s2 >> 16) & 255] & 0xff0000u) | (T[256 + (s3 >> 24)] & 0xff000000u);
    uint32_t o1 = (T[512 + (s1 & 255)] & 0xffu) | (T[768 + ((s2 >> 8) & 255)] & 0xff00u) |
                  (T[(s3 >> 16) & 255] & 0xff0000u) | (T[256 + (s0 >> 24)] & 0xff000000u);
    uint32_t o2 = (T[512 + (s2 & 255)] & 0xffu) | (T[768 + ((s3 >> 8) & 255)] & 0xff00u) |
                  (T[(s0 >> 16) & 255] & 0xff0000u) | (T[256 + (s1 >> 24)] & 0xff000000u);
    uint32_t o3 = (T[512 + (s3 & 255)] & 0xffu) | (T[768 + ((s0 >> 8) & 255)] & 0xff00u) |
                  (T[(s1 >> 16) & 255] & 0xff0000u) | (T[256 + (s2 >> 24)] & 0xff000000u);
    s0 = o0 ^ rk(40);
    s1 = o1 ^ rk(41);
    s2 = o2 ^ rk(42);
    s3 = o3 ^ rk(43);
}

struct HashKey {
    __device__ __forceinline__ uint32_t operator()(int i) const { return kHashKey.w[i]; }
};

struct ArgKey {
    const uint32_t *w;
    __device__ __forceinline__ uint32_t operator()(int i) const { return w[i]; }
};

// ---------------------------------------------------------------------------
// Residue arithmetic (all operands already reduced below m).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t div_m(uint32_t x, const ModConst &mc) {
    uint32_t t = __umulhi(x, mc.divM);
    if (mc.div_fix) return (t + ((x - t) >> 1)) >> mc.divS;
    return t >> mc.divS;
}

__device__ __forceinline__ uint32_t add_mod(uint32_t a, uint32_t b, uint32_t m) {
    uint32_t s = a + b;
    return min(s, s - m);  // s - m wraps above s exactly when s < m
}

__device__ __forceinline__ uint32_t sub_mod(uint32_t a, uint32_t b, uint32_t m) {
    uint32_t d = a - b;
    return min(d, d + m);  // d wraps when a < b; d + m then lands in [0, m)
}

__device__ __forceinline__ uint32_t mul_mod(uint32_t c, uint32_t a, const ModConst &mc) {
    uint32_t p = __umul24(c, a);  // both < 256
    return p - __umul24(div_m(p, mc), mc.m);
}

__device__ __forceinline__ uint32_t field(uint32_t word, uint32_t pos, const ModConst &mc) {
    return (word >> (mc.b * pos)) & mc.mask;
}

// Residues in word w of a label over Z_m.
__device__ __forceinline__ uint32_t residues_in_word(uint32_t w, const ModConst &mc) {
    return (w + 1 == mc.W) ? mc.glast : mc.g;
}

// y + c x, residue by residue, for one packed word (m > 2).
__device__ __forceinline__ uint32_t word_axpy(uint32_t y, uint32_t x, uint32_t c, uint32_t nres, const ModConst &mc) {
    uint32_t out = 0;
    for (uint32_t j = 0; j < nres; ++j) {
        uint32_t r = add_mod(field(y, j, mc), mul_mod(c, field(x, j, mc), mc), mc.m);
        out |= r << (mc.b * j);
    }
    return out;
}

// y - x, residue by residue (m > 2).
__device__ __forceinline__ uint32_t word_sub(uint32_t y, uint32_t x, uint32_t nres, const ModConst &mc) {
    uint32_t out = 0;
    for (uint32_t j = 0; j < nres; ++j) out |= sub_mod(field(y, j, mc), field(x, j, mc), mc.m) << (mc.b * j);
    return out;
}

// c (y - x), residue by residue (m > 2).
__device__ __forceinline__ uint32_t word_scaled_sub(uint32_t y, uint32_t x, uint32_t c, uint32_t nres,
                                                    const ModConst &mc) {
    uint32_t out = 0;
    for (uint32_t j = 0; j < nres; ++j)
        out |= mul_mod(c, sub_mod(field(y, j, mc), field(x, j, mc), mc.m), mc) << (mc.b * j);
    return out;
}

// Generic word operations including m = 2, where a label is a bit vector and
// every operation is an XOR (c is 0 or 1 mod 2).
__device__ __forceinline__ uint32_t label_axpy(uint32_t y, uint32_t x, uint32_t c, uint32_t w, const ModConst &mc) {
    if (mc.m == 2) return (c & 1u) ? (y ^ x) : y;
    return word_axpy(y, x, c, residues_in_word(w, mc), mc);
}
__device__ __forceinline__ uint32_t label_sub(uint32_t y, uint32_t x, uint32_t w, const ModConst &mc) {
    if (mc.m == 2) return y ^ x;
    return word_sub(y, x, residues_in_word(w, mc), mc);
}
__device__ __forceinline__ uint32_t label_scaled_sub(uint32_t y, uint32_t x, uint32_t c, uint32_t w,
                                                     const ModConst &mc) {
    if (mc.m == 2) return (c & 1u) ? (y ^ x) : 0u;
    return word_scaled_sub(y, x, c, residues_in_word(w, mc), mc);
}

// ---------------------------------------------------------------------------
// Digits of the fraction V / 2^256 (V in 8 little-endian limbs): the next
// `nres` base-m digits, most significant first, packed into one word.
// Multiplying by pw = m^nres yields them at once as the carry out of the top
// limb; V keeps the fractional part.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t frac_mul_carry(uint32_t (&V)[8], uint32_t pw) {
    uint64_t carry = 0;
#pragma unroll
    for (int l = 0; l < 8; ++l) {
        uint64_t t = static_cast<uint64_t>(V[l]) * pw + carry;
        V[l] = static_cast<uint32_t>(t);
        carry = t >> 32;
    }
    return static_cast<uint32_t>(carry);
}

__device__ __forceinline__ uint32_t digits_word(uint32_t (&V)[8], uint32_t w, const ModConst &mc) {
    const bool last = (w + 1 == mc.W);
    const uint32_t nres = last ? mc.glast : mc.g;
    uint32_t D = frac_mul_carry(V, last ? mc.pw_last : mc.pw_g);
    uint32_t out = 0;
    for (uint32_t j = nres; j-- > 1;) {
        uint32_t q = div_m(D, mc);
        out |= (D - q * mc.m) << (mc.b * j);
        D = q;
    }
    return out | D;  // the most significant digit is residue 0 of the word
}

// For m = 2 (128-bit fraction in V[0..3]) digit r is bit 127 - r of V, so
// word w is the bit reversal of limb 3 - w.
__device__ __forceinline__ uint32_t bits_word(const uint32_t (&V)[8], uint32_t w) {
    uint32_t limb = (w == 0) ? V[3] : (w == 1) ? V[2] : (w == 2) ? V[1] : V[0];
    return __brev(limb);
}

// ---------------------------------------------------------------------------
// Projection-gate hash, first half: fold the input label's packed words,
// apply sigma and run n AES blocks (n = 2, or 1 when the output modulus is 2).
// Result: V (8 limbs; only V[0..3] meaningful when n = 1).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void hash_fraction(const uint32_t *T, uint32_t x0, uint32_t x1, uint32_t x2, uint32_t x3,
                                              uint64_t tau, uint32_t gid, bool two_blocks, uint32_t (&V)[8]) {
    // sigma(x) = ((x_hi ^ x_lo) << 64) | x_hi with x_lo = lanes 0-1, x_hi = lanes 2-3.
    const uint32_t u0 = x2, u1 = x3, u2 = x2 ^ x0, u3 = x3 ^ x1;
    const uint64_t tw = tau * 4u;
    {
        const uint32_t k0 = static_cast<uint32_t>(tw), k1 = static_cast<uint32_t>(tw >> 32);
        uint32_t s0 = u0 ^ k0, s1 = u1 ^ k1, s2 = u2, s3 = u3 ^ gid;
        const uint32_t i0 = s0, i1 = s1, i2 = s2, i3 = s3;
        aes128_encrypt(T, s0, s1, s2, s3, HashKey{});
        V[0] = s0 ^ i0;
        V[1] = s1 ^ i1;
        V[2] = s2 ^ i2;
        V[3] = s3 ^ i3;
    }
    if (two_blocks) {
        const uint64_t tw1 = tw + 1u;
        const uint32_t k0 = static_cast<uint32_t>(tw1), k1 = static_cast<uint32_t>(tw1 >> 32);
        uint32_t s0 = u0 ^ k0, s1 = u1 ^ k1, s2 = u2, s3 = u3 ^ gid;
        const uint32_t i0 = s0, i1 = s1, i2 = s2, i3 = s3;
        aes128_encrypt(T, s0, s1, s2, s3, HashKey{});
        V[4] = s0 ^ i0;
        V[5] = s1 ^ i1;
        V[6] = s2 ^ i2;
        V[7] = s3 ^ i3;
    } else {
        V[4] = V[5] = V[6] = V[7] = 0;
    }
}

// Pad word w of the hash output over Z_m (words must be produced in order
// w = 0, 1, ... because V is consumed).
__device__ __forceinline__ uint32_t pad_word(uint32_t (&V)[8], uint32_t w, const ModConst &mc) {
    return (mc.m == 2) ? bits_word(V, w) : digits_word(V, w, mc);
}

// Garbler PRG block pair rho(stream, idx): AES_{K_seed}(C_0) || AES_{K_seed}(C_1),
// C_h = stream * 2^120 + 2 idx + h.
__device__ __forceinline__ void prg_fraction(const uint32_t *T, const uint32_t *seed_rk, uint32_t stream, uint64_t idx,
                                             uint32_t (&V)[8]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint64_t c = idx * 2u + static_cast<uint64_t>(h);
        uint32_t s0 = static_cast<uint32_t>(c), s1 = static_cast<uint32_t>(c >> 32), s2 = 0, s3 = stream << 24;
        aes128_encrypt(T, s0, s1, s2, s3, ArgKey{seed_rk});
        V[4 * h] = s0;
        V[4 * h + 1] = s1;
        V[4 * h + 2] = s2;
        V[4 * h + 3] = s3;
    }
}

// Digits of V / 2^256 in radix m for every residue of a label, packed (any m).
// For m = 2 this also takes the fraction digit by digit (radix 2 over 256 bits),
// which differs from the hash's 128-bit layout; it is used by the PRG only.
__device__ __forceinline__ uint32_t prg_word(uint32_t (&V)[8], uint32_t w, const ModConst &mc) {
    if (mc.m != 2) return digits_word(V, w, mc);
    // radix 2: the next 32 digits are the top 32 bits of the 256-bit fraction,
    // most significant first, i.e. the bit reversal of the top limb; then shift.
    uint32_t top = V[7];
#pragma unroll
    for (int l = 7; l > 0; --l) V[l] = V[l - 1];
    V[0] = 0;
    return __brev(top);
}

}  // namespace redash
