// Host check of the bitsliced AES (paper_2506_14489_amd/csrc/aes_bitslice.hpp),
// built with g++ under the address and undefined-behaviour sanitizers by
// tests/test_sanitizers.py:
//  * the S-box circuit on all 256 inputs against S(x) = affine(x^-1) computed
//    here from GF(2^8) arithmetic;
//  * aes128_bs on 32 random blocks (and the FIPS-197 C.1 plaintext) against a
//    byte-oriented AES-128 written here from FIPS-197 over the same round keys,
//    and the C.1 ciphertext;
//  * the 32 x 32 bit transpose on random words.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "../paper_2506_14489_amd/csrc/aes_bitslice.hpp"

using namespace redash;

static uint8_t gmul(uint8_t a, uint8_t b) {
    uint8_t p = 0;
    while (b) {
        if (b & 1) p ^= a;
        const uint8_t h = a & 0x80;
        a = static_cast<uint8_t>(a << 1);
        if (h) a ^= 0x1b;
        b >>= 1;
    }
    return p;
}

static uint8_t SB[256];

static void make_ref_sbox() {
    for (int x = 0; x < 256; ++x) {
        uint8_t inv = 0;
        for (int y = 1; x && y < 256; ++y)
            if (gmul(static_cast<uint8_t>(x), static_cast<uint8_t>(y)) == 1) inv = static_cast<uint8_t>(y);
        uint8_t s = inv, r = 0x63;
        for (int i = 0; i < 5; ++i) {
            r ^= s;
            s = static_cast<uint8_t>((s << 1) | (s >> 7));
        }
        SB[x] = r;
    }
}

static uint8_t key_byte(int r, int j) { return static_cast<uint8_t>(kHashKey.w[4 * r + j / 4] >> (8 * (j % 4))); }

static void ref_aes(const uint8_t in[16], uint8_t out[16]) {
    uint8_t s[16], t[16];
    for (int j = 0; j < 16; ++j) s[j] = in[j] ^ key_byte(0, j);
    for (int r = 1; r <= 10; ++r) {
        for (int j = 0; j < 16; ++j) s[j] = SB[s[j]];
        for (int j = 0; j < 16; ++j) t[j] = s[j % 4 + 4 * ((j / 4 + j % 4) % 4)];
        if (r < 10) {
            for (int c = 0; c < 4; ++c)
                for (int i = 0; i < 4; ++i)
                    s[4 * c + i] = gmul(t[4 * c + i], 2) ^ gmul(t[4 * c + (i + 1) % 4], 3) ^ t[4 * c + (i + 2) % 4] ^
                                   t[4 * c + (i + 3) % 4];
        } else {
            memcpy(s, t, 16);
        }
        for (int j = 0; j < 16; ++j) s[j] ^= key_byte(r, j);
    }
    memcpy(out, s, 16);
}

int main() {
    make_ref_sbox();
    long bad = 0;
    // S-box: 256 inputs in 8 words of 32 lanes
    for (int g = 0; g < 8; ++g) {
        uint32_t x[8] = {};
        for (int i = 0; i < 32; ++i)
            for (int b = 0; b < 8; ++b)
                if (((g * 32 + i) >> b) & 1) x[b] |= 1u << i;
        sbox_bs(x);
        for (int i = 0; i < 32; ++i) {
            int o = 0;
            for (int b = 0; b < 8; ++b) o |= static_cast<int>((x[b] >> i) & 1u) << b;
            if (o != SB[g * 32 + i]) ++bad;
        }
    }
    printf("sbox: %ld mismatches\n", bad);
    // FIPS-197 C.1 through the reference
    const uint8_t pt[16] = {0x00, 0x11, 0x22, 0x33, 0x44, 0x55, 0x66, 0x77,
                            0x88, 0x99, 0xaa, 0xbb, 0xcc, 0xdd, 0xee, 0xff};
    const uint8_t c1[16] = {0x69, 0xc4, 0xe0, 0xd8, 0x6a, 0x7b, 0x04, 0x30,
                            0xd8, 0xcd, 0xb7, 0x80, 0x70, 0xb4, 0xc5, 0x5a};
    uint8_t ct[16];
    ref_aes(pt, ct);
    if (memcmp(ct, c1, 16)) ++bad;
    // 32 blocks bitsliced against the reference
    uint8_t blk[32][16];
    uint64_t r = 88172645463325252ull;
    auto next = [&]() {
        r ^= r << 13;
        r ^= r >> 7;
        r ^= r << 17;
        return r;
    };
    for (int i = 0; i < 32; ++i)
        for (int j = 0; j < 16; ++j) blk[i][j] = static_cast<uint8_t>(next());
    memcpy(blk[5], pt, 16);
    uint32_t st[16][8] = {};
    for (int i = 0; i < 32; ++i)
        for (int j = 0; j < 16; ++j)
            for (int b = 0; b < 8; ++b)
                if ((blk[i][j] >> b) & 1) st[j][b] |= 1u << i;
    aes128_bs(st);
    long aes_bad = 0;
    for (int i = 0; i < 32; ++i) {
        uint8_t want[16];
        ref_aes(blk[i], want);
        for (int j = 0; j < 16; ++j) {
            int o = 0;
            for (int b = 0; b < 8; ++b) o |= static_cast<int>((st[j][b] >> i) & 1u) << b;
            if (o != want[j]) ++aes_bad;
            if (i == 5 && o != c1[j]) ++aes_bad;
        }
    }
    bad += aes_bad;
    printf("aes128_bs: %ld mismatching bytes\n", aes_bad);
    // transpose
    long tr_bad = 0;
    for (int rep = 0; rep < 100; ++rep) {
        uint32_t a[32], b0[32];
        for (int q = 0; q < 32; ++q) a[q] = b0[q] = static_cast<uint32_t>(next());
        transpose32(a);
        for (int q = 0; q < 32; ++q)
            for (int i = 0; i < 32; ++i)
                if (((a[i] >> q) & 1u) != ((b0[q] >> i) & 1u)) ++tr_bad;
    }
    bad += tr_bad;
    printf("transpose32: %ld mismatches\n", tr_bad);
    printf("aes bitslice check: %ld failures\n", bad);
    return bad ? 1 : 0;
}
