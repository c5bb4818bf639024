// Compile-time AES-128 constants (FIPS-197), generated from the field
// arithmetic rather than typed in:
//   * S-box: multiplicative inverse in GF(2^8) modulo x^8+x^4+x^3+x+1
//     (0 maps to 0), followed by the affine map
//     b ^ rotl(b,1) ^ rotl(b,2) ^ rotl(b,3) ^ rotl(b,4) ^ 0x63   (Sec. 5.1.1)
//   * round tables for the column-major little-endian formulation: a state
//     column is one 32-bit word whose low byte is row 0.  TE0[x] is the
//     MixColumns column of the S-box output of x placed in row 0, i.e. the
//     bytes (2 S(x), S(x), S(x), 3 S(x)) from low to high; TE1..TE3 are its
//     byte rotations for rows 1..3                                 (Sec. 5.1.3)
//   * key expansion for Nk = 4, Nr = 10                             (Sec. 5.2)
#pragma once

#include <stdint.h>

namespace redash {

struct Bytes256 {
    uint8_t v[256];
};
struct Words1024 {
    uint32_t v[1024];
};
struct RoundKeys {
    uint32_t w[44];  // w[4 r + c]: column c of round key r, row 0 in the low byte
};

constexpr uint8_t gf_xtime(uint8_t a) {
    return static_cast<uint8_t>((a << 1) ^ ((a & 0x80) ? 0x1b : 0x00));
}

constexpr uint8_t gf_mul(uint8_t a, uint8_t b) {
    uint8_t p = 0;
    for (int i = 0; i < 8; ++i) {
        if (b & 1) p = static_cast<uint8_t>(p ^ a);
        a = gf_xtime(a);
        b = static_cast<uint8_t>(b >> 1);
    }
    return p;
}

// a^254 = a^{-1} for a != 0 in GF(2^8) (the multiplicative group has order 255).
constexpr uint8_t gf_inv(uint8_t a) {
    uint8_t r = 1, base = a;
    int e = 254;
    while (e) {
        if (e & 1) r = gf_mul(r, base);
        base = gf_mul(base, base);
        e >>= 1;
    }
    return a ? r : 0;
}

constexpr uint8_t rotl8(uint8_t x, int r) {
    return static_cast<uint8_t>((x << r) | (x >> (8 - r)));
}

constexpr Bytes256 make_sbox() {
    Bytes256 s{};
    for (int x = 0; x < 256; ++x) {
        uint8_t b = gf_inv(static_cast<uint8_t>(x));
        s.v[x] = static_cast<uint8_t>(b ^ rotl8(b, 1) ^ rotl8(b, 2) ^ rotl8(b, 3) ^ rotl8(b, 4) ^ 0x63);
    }
    return s;
}

constexpr uint32_t rotl32(uint32_t x, int r) {
    return (x << r) | (x >> (32 - r));
}

// TE0..TE3 back to back: word 256 j + x is TEj[x].
constexpr Words1024 make_round_tables() {
    Words1024 t{};
    Bytes256 s = make_sbox();
    for (int x = 0; x < 256; ++x) {
        uint32_t sx = s.v[x];
        uint32_t s2 = gf_mul(static_cast<uint8_t>(sx), 2);
        uint32_t s3 = gf_mul(static_cast<uint8_t>(sx), 3);
        uint32_t t0 = s2 | (sx << 8) | (sx << 16) | (s3 << 24);
        t.v[x] = t0;
        t.v[256 + x] = rotl32(t0, 8);
        t.v[512 + x] = rotl32(t0, 16);
        t.v[768 + x] = rotl32(t0, 24);
    }
    return t;
}

constexpr RoundKeys expand_key(const uint8_t key[16]) {
    RoundKeys rk{};
    Bytes256 s = make_sbox();
    for (int i = 0; i < 4; ++i)
        rk.w[i] = static_cast<uint32_t>(key[4 * i]) | (static_cast<uint32_t>(key[4 * i + 1]) << 8) |
                  (static_cast<uint32_t>(key[4 * i + 2]) << 16) | (static_cast<uint32_t>(key[4 * i + 3]) << 24);
    uint8_t rcon = 1;
    for (int i = 4; i < 44; ++i) {
        uint32_t tmp = rk.w[i - 1];
        if (i % 4 == 0) {
            // RotWord moves byte 1 to byte 0 (row 0 is the low byte), then SubWord, then Rcon on row 0.
            tmp = (tmp >> 8) | (tmp << 24);
            tmp = static_cast<uint32_t>(s.v[tmp & 0xff]) | (static_cast<uint32_t>(s.v[(tmp >> 8) & 0xff]) << 8) |
                  (static_cast<uint32_t>(s.v[(tmp >> 16) & 0xff]) << 16) |
                  (static_cast<uint32_t>(s.v[tmp >> 24]) << 24);
            tmp ^= rcon;
            rcon = gf_xtime(rcon);
        }
        rk.w[i] = rk.w[i - 4] ^ tmp;
    }
    return rk;
}

// The fixed hash key of the projection gates: bytes 00 01 .. 0f.
constexpr RoundKeys make_hash_round_keys() {
    uint8_t key[16] = {};
    for (int i = 0; i < 16; ++i) key[i] = static_cast<uint8_t>(i);
    return expand_key(key);
}

// Garbler PRG key: the 64-bit seed as 16 little-endian bytes.
constexpr RoundKeys make_seed_round_keys(uint64_t seed) {
    uint8_t key[16] = {};
    for (int i = 0; i < 8; ++i) key[i] = static_cast<uint8_t>(seed >> (8 * i));
    return expand_key(key);
}

inline constexpr Bytes256 kSbox = make_sbox();
inline constexpr Words1024 kRoundTables = make_round_tables();
inline constexpr RoundKeys kHashKey = make_hash_round_keys();

// FIPS-197 Appendix C.1 checks the constant generator at compile time.
static_assert(kSbox.v[0x00] == 0x63 && kSbox.v[0x01] == 0x7c && kSbox.v[0x53] == 0xed && kSbox.v[0xff] == 0x16,
              "S-box");
// Round-10 key of Appendix C.1: 13111d7f e3944a17 f307a78b 4d2b30c5.
static_assert(kHashKey.w[40] == 0x7f1d1113u && kHashKey.w[43] == 0xc5302b4du, "key expansion of 00..0f");

}  // namespace redash
