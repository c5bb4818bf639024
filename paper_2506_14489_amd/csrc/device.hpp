// Device helpers for gfx950: AES-128 on LDS round tables, the projection-gate
// hash, base-m digit extraction into packed labels, and residue arithmetic on
// packed 32-bit words.  All per-modulus quantities come from a ModConst that
// is uniform across the wavefront (it lives in the kernel argument block).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

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

// Calls f(std::integral_constant<int, J>{}) for J = 0 .. N-1: every index is
// a compile-time constant, so arrays indexed by it stay in registers.
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (N > 0) {
        static_for<N - 1>(f);
        f(std::integral_constant<int, N - 1>{});
    }
}

// Takes the first word of a small register array and shifts the rest down:
// a rolled loop can walk the array while every index stays a constant (a
// runtime index would move the array to scratch memory).
template <int N>
__device__ __forceinline__ uint32_t next_word(uint32_t (&a)[N]) {
    const uint32_t v = a[0];
#pragma unroll
    for (int j = 0; j + 1 < N; ++j) a[j] = a[j + 1];
    return v;
}

// The value itself, through an empty asm statement that the optimizer cannot
// see into (no instruction is emitted).  Used on the digit x - q m: if it is
// merged into the following arithmetic, the compiler rewrites the product q m
// as one it cannot prove to be 24-bit and emits a quarter-rate multiply.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
    asm("" : "+v"(v));
    return v;
}

// A wave-uniform value masked to 24 bits in the calling block.  Instruction
// selection only uses v_mul_u32_u24 when it sees both operands' 24-bit bound
// in the same basic block; a mask hoisted out of the block (as the compiler
// does with a plain expression) is invisible to it, and the multiply becomes
// the quarter-rate 32-bit one.  The empty volatile asm keeps the mask here.
__device__ __forceinline__ uint32_t uniform24(uint32_t v) {
    asm volatile("" : "+s"(v));
    return v & 0xffffffu;
}

// 24 x 24 -> low 32 bits (v_mul_u32_u24), as an unsigned value: HIP's
// __umul24 returns int, and a right shift of that would be arithmetic.
__device__ __forceinline__ uint32_t mul24(uint32_t a, uint32_t b) {
    return static_cast<uint32_t>(__umul24(a, b));
}

__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);  // truth table of a ^ b ^ c
}

__device__ __forceinline__ uint32_t rotl8(uint32_t x) { return __builtin_amdgcn_alignbit(x, x, 24); }

// Round-table access policies.  column(w0, w1, w2, w3, K, i) is one column
// of a middle round, TE0[byte 0 of w0] ^ TE1[byte 1 of w1] ^ TE2[byte 2 of
// w2] ^ TE3[byte 3 of w3] ^ K(i); last_column(...) is the last round's
// column (S(byte 0 of w0), S(byte 1 of w1), S(byte 2 of w2), S(byte 3 of
// w3)) ^ K(i).  TEt[x] = rotl(TE0[x], 8t), TE0[x] = (2S(x), S(x), S(x), 3S(x))
// as bytes 0..3.
//
// FourTables: TE0..TE3 back to back (1024 words); each S-box byte is taken
// from the table in which it already sits at the right byte position.
struct FourTables {
    const uint32_t *T;
    __device__ __forceinline__ uint32_t te(int t, uint32_t w, int k) const {
        return T[256 * t + ((w >> (8 * k)) & 255u)];
    }
    template <typename Key>
    __device__ __forceinline__ uint32_t column(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, const Key &K,
                                               int i) const {
        return xor3(xor3(te(0, w0, 0), te(1, w1, 1), te(2, w2, 2)), te(3, w3, 3), K(i));
    }
    template <typename Key>
    __device__ __forceinline__ uint32_t last_column(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, const Key &K,
                                                    int i) const {
        // S(x) is byte 0 of TE2, byte 1 of TE3, byte 2 of TE0, byte 3 of TE1
        return ((T[512 + (w0 & 255u)] & 0xffu) | (T[768 + ((w1 >> 8) & 255u)] & 0xff00u) |
                (T[(w2 >> 16) & 255u] & 0xff0000u) | (T[256 + (w3 >> 24)] & 0xff000000u)) ^
               K(i);
    }
};

// PermTE02: TE0 and TE2 in 32 copies each, in 256 LDS rows of 256 bytes: row
// x holds TE0[x] in its lower 128 bytes and TE2[x] in its upper 128 bytes,
// copy c at byte 4c of each half.  Lane l reads copy l mod 32, which sits in
// bank l mod 32: a wavefront's lookups never conflict, whatever the indices.
// One v_perm_b32 builds the address 256 x + 4 (l mod 32) (+ 128 for TE2)
// straight from the state word.  Since TE1 = rotl8 TE0 and TE3 = rotl8 TE2,
// a column is TE0[a] ^ TE2[c] ^ rotl8(TE0[b] ^ TE2[d] ^ rotr8(k)): two
// three-input XORs and one rotation.
constexpr int kReplicas = 32;
constexpr uint32_t kTableRowBytes = 256;
constexpr uint32_t kTableRegionBytes = 256 * kTableRowBytes;  // 64 KiB

// The table region must start at LDS address 0: the kernels that use it
// declare no static LDS, so their dynamic LDS array begins there, and the
// absolute address then needs no base addition per lookup.
typedef __attribute__((address_space(3))) const uint32_t lds_u32;
typedef __attribute__((address_space(3))) uint32_t lds_u32_rw;

__device__ __forceinline__ uint32_t lds_read(uint32_t addr) {
    return *reinterpret_cast<lds_u32 *>(static_cast<uintptr_t>(addr));
}

typedef __attribute__((address_space(3))) const uint8_t lds_u8;
__device__ __forceinline__ uint32_t lds_read_u8(uint32_t addr) {
    return *reinterpret_cast<lds_u8 *>(static_cast<uintptr_t>(addr));
}

struct PermTE02 {
    uint32_t off0, off2;  // 4 (lane mod 32), and that + 128
    // address bytes: [offset, byte k of w, 0, 0]
    __device__ __forceinline__ static uint32_t at(uint32_t w, uint32_t off, int k) {
        return lds_read(__builtin_amdgcn_perm(w, off, 0x0c0c0000u | ((4u + k) << 8)));
    }
    template <typename Key>
    __device__ __forceinline__ uint32_t column(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, const Key &K,
                                               int i) const {
        return xor3(at(w0, off0, 0), at(w2, off2, 2), rotl8(xor3(at(w1, off0, 1), at(w3, off2, 3), K.rot(i))));
    }
    template <typename Key>
    __device__ __forceinline__ uint32_t last_column(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, const Key &K,
                                                    int i) const {
        // S(x) is byte 1 and byte 2 of TE0[x], byte 0 and byte 3 of TE2[x]
        const uint32_t lo = __builtin_amdgcn_perm(at(w1, off0, 1), at(w0, off2, 0), 0x0c0c0500u);
        const uint32_t hi = __builtin_amdgcn_perm(at(w3, off2, 3), at(w2, off0, 2), 0x07020c0cu);
        return xor3(lo, hi, K(i));
    }
};

__device__ __forceinline__ void stage_perm_te02(uint32_t *lds, int tid, int nthreads) {
    // word 64 x + c: TE0[x] for c < 32, TE2[x] for 32 <= c < 64
    for (int i = tid; i < 256 * 2 * kReplicas; i += nthreads) {
        const int x = i >> 6, half = (i >> 5) & 1;
        lds[i] = g_round_tables.v[512 * half + x];
    }
}

__device__ __forceinline__ PermTE02 perm_te02() {
    const uint32_t off = 4u * (threadIdx.x % kReplicas);
    return PermTE02{off, off + 128u};
}

// NB independent blocks encrypted round by round, so that the table reads of
// all blocks are in flight together.
//
// The wave's priority is raised for the rounds and lowered after them: when
// several waves of a SIMD have an instruction ready, one in its AES rounds
// (which keep the LDS pipe busy with table reads) issues before one in other
// work (mostly VALU), so the two pipes stay busy together.
template <int NB, bool PAIRED = false, typename Tab, typename Key>
__device__ __forceinline__ void aes128_encrypt_n(const Tab &T, uint32_t (&s)[NB][4], const Key &K) {
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int c = 0; c < 4; ++c) s[b][c] ^= K(c);
    // Rounds 1..9 stay a loop (the round keys are uniform loads): the
    // instruction cache holds the whole gate loop that way.  A round's new
    // state needs registers of its own while the old one is read, so a loop
    // of one round per pass copies the state back at the end of every pass.
    // PAIRED takes two rounds per pass, the state going to t and back to s,
    // without the copies; it holds more values live, which pays only where
    // the kernel has registers to spare.
    auto round_to = [&](const uint32_t(&in)[NB][4], uint32_t(&o)[NB][4], int r) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            o[b][0] = T.column(in[b][0], in[b][1], in[b][2], in[b][3], K, 4 * r);
            o[b][1] = T.column(in[b][1], in[b][2], in[b][3], in[b][0], K, 4 * r + 1);
            o[b][2] = T.column(in[b][2], in[b][3], in[b][0], in[b][1], K, 4 * r + 2);
            o[b][3] = T.column(in[b][3], in[b][0], in[b][1], in[b][2], K, 4 * r + 3);
        }
    };
    auto last_round = [&](const uint32_t(&in)[NB][4]) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const uint32_t s0 = in[b][0], s1 = in[b][1], s2 = in[b][2], s3 = in[b][3];
            s[b][0] = T.last_column(s0, s1, s2, s3, K, 40);
            s[b][1] = T.last_column(s1, s2, s3, s0, K, 41);
            s[b][2] = T.last_column(s2, s3, s0, s1, K, 42);
            s[b][3] = T.last_column(s3, s0, s1, s2, K, 43);
        }
    };
    if constexpr (PAIRED) {
        uint32_t t[NB][4];
#pragma unroll 1
        for (int r = 1; r < 9; r += 2) {
            round_to(s, t, r);
            round_to(t, s, r + 1);
        }
        round_to(s, t, 9);
        last_round(t);
    } else {
#pragma unroll 1
        for (int r = 1; r < 10; ++r) {
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const uint32_t s0 = s[b][0], s1 = s[b][1], s2 = s[b][2], s3 = s[b][3];
                s[b][0] = T.column(s0, s1, s2, s3, K, 4 * r);
                s[b][1] = T.column(s1, s2, s3, s0, K, 4 * r + 1);
                s[b][2] = T.column(s2, s3, s0, s1, K, 4 * r + 2);
                s[b][3] = T.column(s3, s0, s1, s2, K, 4 * r + 3);
            }
        }
        last_round(s);
    }
    __builtin_amdgcn_s_setprio(0);
}

// One block held as four little-endian column words, on the four tables.
template <typename Key>
__device__ __forceinline__ void aes128_encrypt(const uint32_t *__restrict__ T, uint32_t &s0, uint32_t &s1,
                                               uint32_t &s2, uint32_t &s3, const Key &rk) {
    uint32_t s[1][4] = {{s0, s1, s2, s3}};
    aes128_encrypt_n<1>(FourTables{T}, s, rk);
    s0 = s[0][0];
    s1 = s[0][1];
    s2 = s[0][2];
    s3 = s[0][3];
}

__constant__ RoundKeys c_hash_key = kHashKey;

// Key policies: K(i) is round-key word i, K.rot(i) the same word rotated
// right by 8 bits (the form the two-table column takes).
__device__ __forceinline__ uint32_t rotr8(uint32_t x) { return __builtin_amdgcn_alignbit(x, x, 8); }

struct HashKey {
    __device__ __forceinline__ uint32_t operator()(int i) const { return c_hash_key.w[i]; }
    __device__ __forceinline__ uint32_t rot(int i) const { return rotr8(c_hash_key.w[i]); }
};

// Round keys held in LDS (every lane reads the same word, a broadcast):
// unlike scalar loads, LDS reads complete in order with the table reads, so
// the wait counters never have to drain inside the round loop.  The 44 words
// are followed by their rotated forms.
constexpr int kLdsKeyWords = 88;
struct LdsKey {
    const uint32_t *w;
    __device__ __forceinline__ uint32_t operator()(int i) const { return w[i]; }
    __device__ __forceinline__ uint32_t rot(int i) const { return w[44 + i]; }
};

__device__ __forceinline__ void stage_hash_key(uint32_t *lds, int tid, int nthreads) {
    for (int i = tid; i < 44; i += nthreads) {
        lds[i] = c_hash_key.w[i];
        lds[44 + i] = rotr8(c_hash_key.w[i]);
    }
}

struct ArgKey {
    const uint32_t *w;
    __device__ __forceinline__ uint32_t operator()(int i) const { return w[i]; }
    __device__ __forceinline__ uint32_t rot(int i) const { return rotr8(w[i]); }
};

// ---------------------------------------------------------------------------
// Residue arithmetic (all operands already reduced below m).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t div_m(uint32_t x, const ModConst &mc) {
    uint32_t t = __umulhi(x, mc.divM);
    if (mc.div_fix) return (t + ((x - t) >> 1)) >> mc.divS;
    return t >> mc.divS;
}

// By value (a reference-returning min would make the compiler keep its
// operands in scratch memory).
__device__ __forceinline__ uint32_t umin(uint32_t a, uint32_t b) { return a < b ? a : b; }

__device__ __forceinline__ uint32_t add_mod(uint32_t a, uint32_t b, uint32_t m) {
    uint32_t s = a + b;
    return umin(s, s - m);  // s - m wraps above s exactly when s < m
}

__device__ __forceinline__ uint32_t sub_mod(uint32_t a, uint32_t b, uint32_t m) {
    uint32_t d = a - b;
    return umin(d, d + m);  // d wraps when a < b; d + m then lands in [0, m)
}

__device__ __forceinline__ uint32_t mul_mod(uint32_t c, uint32_t a, const ModConst &mc) {
    uint32_t p = mul24(c, a);  // both < 256
    return p - mul24(div_m(p, mc), mc.m);
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

// The same with pw = 0 standing for 2^32 (m = 4, 16): the carry is the top
// limb and the limbs move up by one.
__device__ __forceinline__ uint32_t frac_carry_any(uint32_t (&V)[8], uint32_t pw) {
    if (pw) return frac_mul_carry(V, pw);
    const uint32_t top = V[7];
#pragma unroll
    for (int l = 7; l > 0; --l) V[l] = V[l - 1];
    V[0] = 0;
    return top;
}

__device__ __forceinline__ uint32_t digits_word(uint32_t (&V)[8], uint32_t w, const ModConst &mc) {
    const bool last = (w + 1 == mc.W);
    const uint32_t nres = last ? mc.glast : mc.g;
    uint32_t D = frac_carry_any(V, last ? mc.pw_last : mc.pw_g);
    uint32_t out = 0;
    for (uint32_t j = nres; j-- > 1;) {
        uint32_t q = div_m(D, mc);
        out |= (D - q * mc.m) << (mc.b * j);
        D = q;
    }
    return out | D;  // the most significant digit is residue 0 of the word
}

// floor(x / d) for a 32-bit x with constants from division_constants().
__device__ __forceinline__ uint32_t div_const(uint32_t x, uint32_t M, uint32_t s, uint32_t fix) {
    const uint32_t t = __umulhi(x, M);
    return fix ? (t + ((x - t) >> 1)) >> s : t >> s;
}

// Evaluator fast path for one packed word over Z_m (m > 2, mc.fast set).
// D holds the word's nres pad digits as a base-m number (residue 0 the most
// significant digit).  For each residue j, with pad digit p, row residue r
// and label residue l:
//   sub gate (ACC = false): l <- c (l - p - r)      computed as c (l + 2m - p - r) < 3 m^2
//   acc gate (ACC = true):  l <- l + c (p + r)      computed unreduced, < 2 m^2
// followed by one multiply-shift reduction.  D is first split as
// hi * m^nlo + lo so that every further digit division works on < 2^24.
template <bool ACC>
__device__ __forceinline__ uint32_t fast_word(uint32_t D, uint32_t nres, uint32_t nlo, uint32_t lo_M, uint32_t lo_s,
                                              uint32_t pw_lo, uint32_t rw, uint32_t l, uint32_t c,
                                              const ModConst &mc) {
    const uint32_t m = mc.m, b = mc.b, mask = mc.mask;
    uint32_t hi = D, lo = 0;
    if (nlo) {
        hi = __umulhi(D, lo_M) >> lo_s;
        lo = D - mul24(hi, pw_lo);
    }
    // mc.two_m (= 2m) is a separate field on purpose: were the compiler to
    // see it as 2 * m, it would fold "+ 2m - (x - q m)" into (q + 2) m, a
    // product it cannot prove to be 24-bit (quarter-rate multiply).
    auto residue = [&](uint32_t p, uint32_t j) -> uint32_t {
        const uint32_t r = (rw >> (b * j)) & mask;
        const uint32_t lj = (l >> (b * j)) & mask;
        const uint32_t v = ACC ? lj + mul24(c, p + r) : mul24(c, lj + mc.two_m - p - r);
        const uint32_t q = __umulhi(v, mc.red_M);
        return (v - mul24(q, m)) << (b * j);
    };
    uint32_t res = 0;
    const uint32_t nhi = nres - nlo;
    // low part: positions nres-1 down to nhi (least significant digit first)
    uint32_t x = lo;
    for (uint32_t j = nres - 1; j > nhi; --j) {
        const uint32_t q = mul24(x, mc.sd_M) >> mc.sd_s;
        res |= residue(opaque(x - mul24(q, m)), j);
        x = q;
    }
    if (nlo) res |= residue(x, nhi);
    // high part: positions nhi-1 down to 0
    x = hi;
    for (uint32_t j = nhi - 1; j > 0; --j) {
        const uint32_t q = mul24(x, mc.sd_M) >> mc.sd_s;
        res |= residue(opaque(x - mul24(q, m)), j);
        x = q;
    }
    res |= residue(x, 0);
    return res;
}

// The ND base-m digits of x < m^ND (with (m^ND)^2 < 2^32), most significant
// first, handed to f(digit, integral_constant<J0 + k>) for k = 0..ND-1:
// F = x C mod 2^32 with C = floor(2^32 / m^ND) + 1 approximates the fraction
// x / m^ND from above by less than 2^-32 x, so each umulhi(F, m) is the next
// digit exactly, and F m mod 2^32 the remaining fraction.
template <int ND, int J0, typename Fn>
__device__ __forceinline__ void frac_digits(uint32_t x, uint32_t C, uint32_t m, Fn &&f) {
    if constexpr (ND > 0) {
        uint32_t F = x * C;
        static_for<ND>([&](auto k) {
            constexpr int kk = decltype(k)::value;
            f(__umulhi(F, m), std::integral_constant<int, J0 + kk>{});
            if constexpr (kk + 1 < ND) F *= m;
        });
    }
}

// fast_word with the residue count and field width known at compile time:
// every loop unrolled, every shift an immediate.
//
// With TAB, the product c (v mod m) mod m comes from the gate's byte table in
// LDS (v < 3m, see free_op_table): tk is the table's LDS address, plus 2m for
// a sub gate, so the sub gate's byte address is lj + tk - p - r.
//
// The digits of each part come from fraction multiplication (ModConst::fd):
// two full-rate multiplies per digit instead of a division step.
template <bool ACC, int NRES, int B, bool TAB>
__device__ __forceinline__ uint32_t fast_word_c(uint32_t D, uint32_t lo_M, uint32_t lo_s, uint32_t pw_lo,
                                                uint32_t c_hi, uint32_t c_lo, uint32_t rw, uint32_t l, uint32_t c,
                                                const ModConst &mc, uint32_t tk) {
    constexpr int NLO = NRES / 2, NHI = NRES - NLO;
    constexpr uint32_t MASK = (1u << B) - 1u;
    const uint32_t m = uniform24(mc.m);
    c = uniform24(c);
    uint32_t hi = D, lo = 0;
    if constexpr (NLO > 0) {
        hi = __umulhi(D, lo_M) >> lo_s;
        lo = D - mul24(hi, pw_lo);
    }
    uint32_t res = 0;
    // Every multiply below must see both operands' 24-bit bound in this block
    // (v_mul_u32_u24): shifted quotients and the sub gate's difference go
    // through a bit-field extract of width 24 or 16, whose bound the
    // instruction selector always sees (one op, like the shift it replaces).
    auto residue = [&](uint32_t p, auto jc) {
        constexpr int j = decltype(jc)::value;
        const uint32_t r = (rw >> (B * j)) & MASK;
        const uint32_t lj = (l >> (B * j)) & MASK;
        if constexpr (TAB) {
            if constexpr (ACC) {
                const uint32_t x = lj + lds_read_u8(tk + p + r);  // < 2m
                res |= umin(x, x - m) << (B * j);
            } else {
                res |= lds_read_u8(lj + tk - p - r) << (B * j);
            }
        } else {
            const uint32_t v = ACC ? lj + mul24(c, __builtin_amdgcn_ubfe(p + r, 0, 16))
                                   : mul24(c, __builtin_amdgcn_ubfe(lj + mc.two_m - p - r, 0, 16));
            const uint32_t q = __umulhi(v, mc.red_M);
            // (opaque: a shift folded into the product would widen its operand)
            res |= opaque(v - mul24(q, m)) << (B * j);
        }
    };
    // high part: residues 0..NHI-1; low part: NHI..NRES-1 (most significant first)
    frac_digits<NHI, 0>(hi, c_hi, mc.m, residue);
    frac_digits<NLO, NHI>(lo, c_lo, mc.m, residue);
    return res;
}

// Dispatch on (residues in the word, bits per residue): the combinations
// of the primes up to 37 and of the short bases' moduli (8, 32, 97, 107,
// 128, 167, 173) are unrolled, anything else takes the loops.
template <bool ACC, bool TAB>
__device__ __forceinline__ uint32_t fast_word_any(uint32_t D, uint32_t nres, uint32_t nlo, uint32_t lo_M,
                                                  uint32_t lo_s, uint32_t pw_lo, uint32_t c_hi, uint32_t c_lo,
                                                  uint32_t rw, uint32_t l, uint32_t c, const ModConst &mc,
                                                  uint32_t tk) {
    if (!mc.fd) return fast_word<ACC>(D, nres, nlo, lo_M, lo_s, pw_lo, rw, l, c, mc);
    switch (nres | (mc.b << 8)) {
#define REDASH_FW(NR, BB)        \
    case (NR) | ((BB) << 8): \
        return fast_word_c<ACC, NR, BB, TAB>(D, lo_M, lo_s, pw_lo, c_hi, c_lo, rw, l, c, mc, tk);
        REDASH_FW(16, 2) REDASH_FW(1, 2) REDASH_FW(10, 3) REDASH_FW(6, 3) REDASH_FW(8, 4) REDASH_FW(6, 4)
        REDASH_FW(3, 4) REDASH_FW(6, 5) REDASH_FW(5, 5) REDASH_FW(3, 5) REDASH_FW(2, 5) REDASH_FW(1, 5)
        REDASH_FW(5, 6) REDASH_FW(3, 3) REDASH_FW(4, 7) REDASH_FW(3, 7) REDASH_FW(4, 8) REDASH_FW(2, 8)
#undef REDASH_FW
        default: return fast_word<ACC>(D, nres, nlo, lo_M, lo_s, pw_lo, rw, l, c, mc);
    }
}

// Garbler rows: for one packed word over Z_m (m > 2, fast constants), the
// residues (b_j - p_j) mod m, where p_j are the word's pad digits held in D
// as a base-m number (residue 0 the most significant digit) and b_j the
// residues of the packed word bw.
template <int NRES, int B>
__device__ __forceinline__ uint32_t row_word_c(uint32_t D, uint32_t lo_M, uint32_t lo_s, uint32_t pw_lo, uint32_t c_hi,
                                               uint32_t c_lo, uint32_t bw, const ModConst &mc) {
    constexpr int NLO = NRES / 2, NHI = NRES - NLO;
    constexpr uint32_t MASK = (1u << B) - 1u;
    const uint32_t m = uniform24(mc.m);
    uint32_t hi = D, lo = 0;
    if constexpr (NLO > 0) {
        hi = __umulhi(D, lo_M) >> lo_s;
        lo = D - mul24(hi, pw_lo);
    }
    uint32_t res = 0;
    auto residue = [&](uint32_t p, auto jc) {
        constexpr int j = decltype(jc)::value;
        const uint32_t d = ((bw >> (B * j)) & MASK) - p;
        res |= umin(d, d + m) << (B * j);
    };
    frac_digits<NHI, 0>(hi, c_hi, mc.m, residue);
    frac_digits<NLO, NHI>(lo, c_lo, mc.m, residue);
    return res;
}

// row_word_c for any word shape; shapes outside the unrolled list of
// fast_word_any take the generic digit loop.
__device__ __forceinline__ uint32_t row_word_any(uint32_t D, uint32_t nres, uint32_t lo_M, uint32_t lo_s,
                                                 uint32_t pw_lo, uint32_t c_hi, uint32_t c_lo, uint32_t bw,
                                                 const ModConst &mc) {
    switch (mc.fd ? nres | (mc.b << 8) : 0u) {
#define REDASH_RW(NR, BB) \
    case (NR) | ((BB) << 8): return row_word_c<NR, BB>(D, lo_M, lo_s, pw_lo, c_hi, c_lo, bw, mc);
        REDASH_RW(16, 2) REDASH_RW(1, 2) REDASH_RW(10, 3) REDASH_RW(6, 3) REDASH_RW(8, 4) REDASH_RW(6, 4)
        REDASH_RW(3, 4) REDASH_RW(6, 5) REDASH_RW(5, 5) REDASH_RW(3, 5) REDASH_RW(2, 5) REDASH_RW(1, 5)
        REDASH_RW(5, 6) REDASH_RW(3, 3) REDASH_RW(4, 7) REDASH_RW(3, 7) REDASH_RW(4, 8) REDASH_RW(2, 8)
#undef REDASH_RW
        default: {
            uint32_t res = 0;
            for (uint32_t j = nres; j-- > 0;) {
                uint32_t p = D;
                if (j) {
                    const uint32_t q = div_m(D, mc);
                    p = D - q * mc.m;
                    D = q;
                }
                res |= sub_mod(field(bw, j, mc), p, mc.m) << (mc.b * j);
            }
            return res;
        }
    }
}

// (x + u) mod m in every field of one packed word (m > 2) at once, with u
// given as its even fields ue and its odd fields shifted down, uo (see
// ModConst::sw_even): sums of two residues stay below 2m <= 2^(b+1) in a
// field with b free bits above it, adding 2^b - m sets bit b exactly where
// the sum is at least m, and m times that bit is subtracted.
__device__ __forceinline__ uint32_t swar_add(uint32_t x, uint32_t ue, uint32_t uo, const ModConst &mc) {
    const uint32_t se = (x & mc.sw_even) + ue;
    const uint32_t so = ((x >> mc.b) & mc.sw_even) + uo;
    const uint32_t ce = ((se + mc.sw_k) >> mc.b) & mc.sw_ones;
    const uint32_t co = ((so + mc.sw_k) >> mc.b) & mc.sw_ones;
    return (se - ce * mc.m) | ((so - co * mc.m) << mc.b);
}

// (x + u) mod m residue by residue for one packed word (any m; m = 2 is XOR).
__device__ __forceinline__ uint32_t word_add(uint32_t x, uint32_t u, uint32_t nres, const ModConst &mc) {
    if (mc.m == 2) return x ^ u;
    uint32_t out = 0;
    for (uint32_t j = 0; j < nres; ++j) out |= add_mod(field(x, j, mc), field(u, j, mc), mc.m) << (mc.b * j);
    return out;
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
    // (scalars rather than array stores inside the branch, which the
    // compiler would otherwise route through scratch memory)
    uint32_t h0 = 0, h1 = 0, h2 = 0, h3 = 0;
    if (two_blocks) {
        const uint64_t tw1 = tw + 1u;
        const uint32_t k0 = static_cast<uint32_t>(tw1), k1 = static_cast<uint32_t>(tw1 >> 32);
        uint32_t s0 = u0 ^ k0, s1 = u1 ^ k1, s2 = u2, s3 = u3 ^ gid;
        const uint32_t i0 = s0, i1 = s1, i2 = s2, i3 = s3;
        aes128_encrypt(T, s0, s1, s2, s3, HashKey{});
        h0 = s0 ^ i0;
        h1 = s1 ^ i1;
        h2 = s2 ^ i2;
        h3 = s3 ^ i3;
    }
    V[4] = h0;
    V[5] = h1;
    V[6] = h2;
    V[7] = h3;
}

// The hash fractions of NG gates that share one input label (folded into
// x0..x3): gate j uses tweak tau + j and two blocks (a gate whose output
// modulus is 2 only reads V[j][0..3]).
template <int NG, bool PAIRED = false, typename Tab, typename Key>
__device__ __forceinline__ void hash_fraction_n(const Tab &T, const Key &rk, uint32_t x0, uint32_t x1, uint32_t x2,
                                                uint32_t x3, uint64_t tau, uint32_t gid, uint32_t (&V)[NG][8]) {
    const uint32_t u0 = x2, u1 = x3, u2 = x2 ^ x0, u3 = x3 ^ x1;
    uint32_t s[2 * NG][4];
#pragma unroll
    for (int j = 0; j < NG; ++j) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint64_t tw = (tau + static_cast<uint64_t>(j)) * 4u + static_cast<uint64_t>(h);
            s[2 * j + h][0] = u0 ^ static_cast<uint32_t>(tw);
            s[2 * j + h][1] = u1 ^ static_cast<uint32_t>(tw >> 32);
            s[2 * j + h][2] = u2;
            s[2 * j + h][3] = u3 ^ gid;
        }
    }
    aes128_encrypt_n<2 * NG, PAIRED>(T, s, rk);
    // Matyas-Meyer-Oseas feed-forward of the block input u ^ T.  The inputs
    // are formed again from x and tau rather than kept through the rounds
    // (opaque keeps the compiler from reusing the earlier values): six
    // registers live across the AES instead of up to twelve.
    const uint32_t y0 = opaque(x0), y1 = opaque(x1), y2 = opaque(x2), y3 = opaque(x3);
    const uint64_t tau2 = (static_cast<uint64_t>(opaque(static_cast<uint32_t>(tau >> 32))) << 32) |
                          opaque(static_cast<uint32_t>(tau));
#pragma unroll
    for (int j = 0; j < NG; ++j) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint64_t tw = (tau2 + static_cast<uint64_t>(j)) * 4u + static_cast<uint64_t>(h);
            V[j][4 * h + 0] = s[2 * j + h][0] ^ y2 ^ static_cast<uint32_t>(tw);
            V[j][4 * h + 1] = s[2 * j + h][1] ^ y3 ^ static_cast<uint32_t>(tw >> 32);
            V[j][4 * h + 2] = s[2 * j + h][2] ^ y2 ^ y0;
            V[j][4 * h + 3] = s[2 * j + h][3] ^ y3 ^ y1 ^ gid;
        }
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
