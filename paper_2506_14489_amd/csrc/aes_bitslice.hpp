// Bitsliced AES-128 under the hash key, 32 blocks per 32-bit word: bit i of
// slice [j][b] is bit b of byte j of block i.  No table lookups: SubBytes is
// the depth-16 S-box circuit of Boyar and Peralta ("A depth-16 circuit for
// the AES S-box", 2012: 32 AND, 81 XOR/XNOR gates), MixColumns is xtime on
// bit slices, ShiftRows a renaming of the byte index, AddRoundKey a
// complement of the slices whose round-key bit is 1 (the key is a
// compile-time constant).
#pragma once

#include <stdint.h>

#include "aes_tables.hpp"

#if defined(__HIPCC__)
#define REDASH_HD __host__ __device__ __forceinline__
#else
#define REDASH_HD inline
#endif

namespace redash {

// S(x) on 32 bytes at once; x[b] holds bit b (b = 0 the least significant)
// of the 32 bytes, replaced by the bits of S(x).  The circuit's inputs
// U0..U7 and outputs S0..S7 count from the most significant bit.
REDASH_HD void sbox_bs(uint32_t (&x)[8]) {
    const uint32_t U0 = x[7], U1 = x[6], U2 = x[5], U3 = x[4], U4 = x[3], U5 = x[2], U6 = x[1], U7 = x[0];
    // top linear layer
    const uint32_t T1 = U0 ^ U3, T2 = U0 ^ U5, T3 = U0 ^ U6, T4 = U3 ^ U5, T5 = U4 ^ U6;
    const uint32_t T6 = T1 ^ T5, T7 = U1 ^ U2, T8 = U7 ^ T6, T9 = U7 ^ T7, T10 = T6 ^ T7;
    const uint32_t T11 = U1 ^ U5, T12 = U2 ^ U5, T13 = T3 ^ T4, T14 = T6 ^ T11, T15 = T5 ^ T11;
    const uint32_t T16 = T5 ^ T12, T17 = T9 ^ T16, T18 = U3 ^ U7, T19 = T7 ^ T18, T20 = T1 ^ T19;
    const uint32_t T21 = U6 ^ U7, T22 = T7 ^ T21, T23 = T2 ^ T22, T24 = T2 ^ T10, T25 = T20 ^ T17;
    const uint32_t T26 = T3 ^ T16, T27 = T1 ^ T12;
    const uint32_t D = U7;
    // nonlinear middle
    const uint32_t M1 = T13 & T6, M2 = T23 & T8, M3 = T14 ^ M1, M4 = T19 & D, M5 = M4 ^ M1;
    const uint32_t M6 = T3 & T16, M7 = T22 & T9, M8 = T26 ^ M6, M9 = T20 & T17, M10 = M9 ^ M6;
    const uint32_t M11 = T1 & T15, M12 = T4 & T27, M13 = M12 ^ M11, M14 = T2 & T10, M15 = M14 ^ M11;
    const uint32_t M16 = M3 ^ M2, M17 = M5 ^ T24, M18 = M8 ^ M7, M19 = M10 ^ M15, M20 = M16 ^ M13;
    const uint32_t M21 = M17 ^ M15, M22 = M18 ^ M13, M23 = M19 ^ T25, M24 = M22 ^ M23, M25 = M22 & M20;
    const uint32_t M26 = M21 ^ M25, M27 = M20 ^ M21, M28 = M23 ^ M25, M29 = M28 & M27, M30 = M26 & M24;
    const uint32_t M31 = M20 & M23, M32 = M27 & M31, M33 = M27 ^ M25, M34 = M21 & M22, M35 = M24 & M34;
    const uint32_t M36 = M24 ^ M25, M37 = M21 ^ M29, M38 = M32 ^ M33, M39 = M23 ^ M30, M40 = M35 ^ M36;
    const uint32_t M41 = M38 ^ M40, M42 = M37 ^ M39, M43 = M37 ^ M38, M44 = M39 ^ M40, M45 = M42 ^ M41;
    const uint32_t M46 = M44 & T6, M47 = M40 & T8, M48 = M39 & D, M49 = M43 & T16, M50 = M38 & T9;
    const uint32_t M51 = M37 & T17, M52 = M42 & T15, M53 = M45 & T27, M54 = M41 & T10, M55 = M44 & T13;
    const uint32_t M56 = M40 & T23, M57 = M39 & T19, M58 = M43 & T3, M59 = M38 & T22, M60 = M37 & T20;
    const uint32_t M61 = M42 & T1, M62 = M45 & T4, M63 = M41 & T2;
    // bottom linear layer
    const uint32_t L0 = M61 ^ M62, L1 = M50 ^ M56, L2 = M46 ^ M48, L3 = M47 ^ M55, L4 = M54 ^ M58;
    const uint32_t L5 = M49 ^ M61, L6 = M62 ^ L5, L7 = M46 ^ L3, L8 = M51 ^ M59, L9 = M52 ^ M53;
    const uint32_t L10 = M53 ^ L4, L11 = M60 ^ L2, L12 = M48 ^ M51, L13 = M50 ^ L0, L14 = M52 ^ M61;
    const uint32_t L15 = M55 ^ L1, L16 = M56 ^ L0, L17 = M57 ^ L1, L18 = M58 ^ L8, L19 = M63 ^ L4;
    const uint32_t L20 = L0 ^ L1, L21 = L1 ^ L7, L22 = L3 ^ L12, L23 = L18 ^ L2, L24 = L15 ^ L9;
    const uint32_t L25 = L6 ^ L10, L26 = L7 ^ L9, L27 = L8 ^ L10, L28 = L11 ^ L14, L29 = L11 ^ L17;
    x[7] = L6 ^ L24;      // S0
    x[6] = ~(L16 ^ L26);  // S1
    x[5] = ~(L19 ^ L28);  // S2
    x[4] = L6 ^ L21;      // S3
    x[3] = L20 ^ L22;     // S4
    x[2] = L25 ^ L29;     // S5
    x[1] = ~(L13 ^ L27);  // S6
    x[0] = ~(L6 ^ L23);   // S7
}

// xtime on one bit-sliced byte (multiplication by x modulo x^8 + x^4 + x^3 + x + 1)
REDASH_HD void xtime_bs(const uint32_t (&a)[8], uint32_t (&y)[8]) {
    y[0] = a[7];
    y[1] = a[0] ^ a[7];
    y[2] = a[1];
    y[3] = a[2] ^ a[7];
    y[4] = a[3] ^ a[7];
    y[5] = a[4];
    y[6] = a[5];
    y[7] = a[6];
}

// One AES-128 encryption of 32 blocks under the hash key.  st[j][b]: byte j
// (byte j of the block is byte j mod 4 of its little-endian word j / 4, i.e.
// row j mod 4 of column j / 4 of the state), bit b.
REDASH_HD void aes128_bs(uint32_t (&st)[16][8]) {
    auto add_round_key = [&](int r) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const uint32_t kb = (kHashKey.w[4 * r + j / 4] >> (8 * (j % 4))) & 255u;
#pragma unroll
            for (int b = 0; b < 8; ++b)
                if ((kb >> b) & 1u) st[j][b] = ~st[j][b];
        }
    };
    add_round_key(0);
#pragma unroll
    for (int r = 1; r <= 10; ++r) {
#pragma unroll
        for (int j = 0; j < 16; ++j) sbox_bs(st[j]);
        // ShiftRows: row i of column c takes row i of column c + i
        uint32_t t[16][8];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int row = j % 4, col = j / 4;
            const int from = row + 4 * ((col + row) % 4);
#pragma unroll
            for (int b = 0; b < 8; ++b) t[j][b] = st[from][b];
        }
        if (r < 10) {
            // MixColumns: out_i = 2 a_i + 3 a_{i+1} + a_{i+2} + a_{i+3} = a_i + s + xtime(a_i + a_{i+1})
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                uint32_t sum[8];
#pragma unroll
                for (int b = 0; b < 8; ++b) sum[b] = t[4 * c][b] ^ t[4 * c + 1][b] ^ t[4 * c + 2][b] ^ t[4 * c + 3][b];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    uint32_t u[8], x2[8];
#pragma unroll
                    for (int b = 0; b < 8; ++b) u[b] = t[4 * c + i][b] ^ t[4 * c + (i + 1) % 4][b];
                    xtime_bs(u, x2);
#pragma unroll
                    for (int b = 0; b < 8; ++b) st[4 * c + i][b] = t[4 * c + i][b] ^ sum[b] ^ x2[b];
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < 16; ++j)
#pragma unroll
                for (int b = 0; b < 8; ++b) st[j][b] = t[j][b];
        }
        add_round_key(r);
    }
}

// Transposes a 32 x 32 bit matrix in place: bit i of a[q] <-> bit q of a[i].
REDASH_HD void transpose32(uint32_t (&a)[32]) {
    uint32_t m = 0x0000ffffu;
#pragma unroll
    for (int s = 16; s >= 1; s >>= 1, m ^= m << s) {
#pragma unroll
        for (int k = 0; k < 32; k = ((k | s) + 1) & ~s) {
            const uint32_t t = ((a[k] >> s) ^ a[k | s]) & m;
            a[k | s] ^= t;
            a[k] ^= t << s;
        }
    }
}

}  // namespace redash
