/*
 * gc_oracle.c -- plain, slow CPU oracle for the garbled ReDASH scaling gadget.
 *
 * TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and the CPU
 * baseline leg of bench.py may load this library.  It shares no code, header,
 * table or constant generator with the HIP library: it carries its own AES,
 * its own label packing, its own gate list and its own layouts, all written
 * from the definitions below.
 *
 * What it follows:
 *   - wire labels l_a = l_0 + a*R over Z_m, free addition and free
 *     multiplication by public constants                       (Sec. 2.3)
 *   - projection gates with p-1 ciphertexts (row reduction)    (Sec. 2.3)
 *   - ShiftUp by P/2, division by s (Sec. 3.2), generalized base
 *     extension (Sec. 3.3, Eq. rns_to_mrs with the corrected missing-residue
 *     formula), ShiftDown by P/(2s)                             (Sec. 3.4)
 *     READING where P/2 or P/(2s) is not an integer (odd P, or a power-of-two
 *     modulus that is also scaled by, Sec. 4's 2^l bases): ShiftUp by
 *     U = floor(P/2), ShiftDown by floor(U/s); the gadget then returns
 *     floor((x + (U mod s)) / s), which is floor(x/s) whenever P/(2s) is an
 *     integer.
 *   - moduli: primes, or one power of two (the 2^l moduli of Sec. 4),
 *     pairwise coprime
 *   - garbler offline / evaluator online roles                 (Sec. 2.1)
 *
 * The paper does not fix the label hash, the label length, the PRG, the
 * tweaks, the table layout or any bit convention.  The concrete choices
 * ("R-spec v1") are written out in the design notes and restated at each
 * function below.  The paper does not pin the exact label BITS; the tests
 * pin them by the invariants (every wire label equals its zero-label plus
 * value times the offset; decode equals floor(x/s)), by FIPS-197 for AES,
 * and step by step against a second statement of the hash and the PRG on
 * Python integers and libcrypto's AES (fold lanes, sigma as a linear
 * orthomorphism, tweak words, feed-forward, digits, PRG counters), plus
 * known-answer files derived from it.
 *
 * Plain C99 + unsigned __int128 (gcc).  Single-threaded.  No tuning.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_MAXK 16
#define ORC_MAXLAMBDA 128
#define ORC_MAXGATES 256

#define ORC_OK 0
#define ORC_EPARAM -1
#define ORC_ENULL -2

typedef struct {
    uint32_t k;
    uint32_t moduli[16];
    uint32_t t;
    uint32_t scale_idx[16];
    uint64_t n;
    uint64_t seed;
} orc_params;

/* ======================================================================
 * AES-128, written from FIPS-197 (Sections 5.1 and 5.2).
 * ====================================================================== */

static uint8_t SBOX[256];
static int sbox_ready = 0;

static uint8_t xtime(uint8_t a) { return (uint8_t)((a << 1) ^ ((a & 0x80) ? 0x1b : 0x00)); }

static uint8_t gf_mul(uint8_t a, uint8_t b) {
    uint8_t p = 0;
    while (b) {
        if (b & 1) p ^= a;
        a = xtime(a);
        b >>= 1;
    }
    return p;
}

static uint8_t rotl8(uint8_t x, int r) { return (uint8_t)((x << r) | (x >> (8 - r))); }

/* S-box: multiplicative inverse in GF(2^8) (0 -> 0) followed by the affine
 * transformation b ^ rotl(b,1) ^ rotl(b,2) ^ rotl(b,3) ^ rotl(b,4) ^ 0x63. */
static void build_sbox(void) {
    for (int x = 0; x < 256; ++x) {
        uint8_t inv = 0;
        if (x) {
            for (int y = 1; y < 256; ++y)
                if (gf_mul((uint8_t)x, (uint8_t)y) == 1) { inv = (uint8_t)y; break; }
        }
        SBOX[x] = (uint8_t)(inv ^ rotl8(inv, 1) ^ rotl8(inv, 2) ^ rotl8(inv, 3) ^ rotl8(inv, 4) ^ 0x63);
    }
    sbox_ready = 1;
}

static void ensure_sbox(void) { if (!sbox_ready) build_sbox(); }

/* Key expansion for Nk = 4, Nr = 10: 44 words w[i], stored as 176 bytes. */
static void key_expansion(const uint8_t key[16], uint8_t w[176]) {
    ensure_sbox();
    memcpy(w, key, 16);
    uint8_t rcon = 0x01;
    for (int i = 4; i < 44; ++i) {
        uint8_t t[4];
        memcpy(t, w + 4 * (i - 1), 4);
        if (i % 4 == 0) {
            uint8_t r0 = t[0];           /* RotWord */
            t[0] = t[1]; t[1] = t[2]; t[2] = t[3]; t[3] = r0;
            for (int j = 0; j < 4; ++j) t[j] = SBOX[t[j]]; /* SubWord */
            t[0] ^= rcon;
            rcon = xtime(rcon);
        }
        for (int j = 0; j < 4; ++j) w[4 * i + j] = (uint8_t)(w[4 * (i - 4) + j] ^ t[j]);
    }
}

/* Cipher(): state s[r][c] = in[r + 4c]. */
static void aes_encrypt(const uint8_t rk[176], const uint8_t in[16], uint8_t out[16]) {
    uint8_t s[4][4], u[4][4];
    for (int c = 0; c < 4; ++c)
        for (int r = 0; r < 4; ++r) s[r][c] = in[r + 4 * c];
    for (int c = 0; c < 4; ++c)
        for (int r = 0; r < 4; ++r) s[r][c] ^= rk[4 * c + r];
    for (int round = 1; round <= 10; ++round) {
        for (int r = 0; r < 4; ++r)            /* SubBytes */
            for (int c = 0; c < 4; ++c) s[r][c] = SBOX[s[r][c]];
        for (int r = 0; r < 4; ++r)            /* ShiftRows */
            for (int c = 0; c < 4; ++c) u[r][c] = s[r][(c + r) % 4];
        memcpy(s, u, sizeof s);
        if (round != 10) {                     /* MixColumns */
            for (int c = 0; c < 4; ++c) {
                uint8_t a0 = s[0][c], a1 = s[1][c], a2 = s[2][c], a3 = s[3][c];
                s[0][c] = (uint8_t)(gf_mul(a0, 2) ^ gf_mul(a1, 3) ^ a2 ^ a3);
                s[1][c] = (uint8_t)(a0 ^ gf_mul(a1, 2) ^ gf_mul(a2, 3) ^ a3);
                s[2][c] = (uint8_t)(a0 ^ a1 ^ gf_mul(a2, 2) ^ gf_mul(a3, 3));
                s[3][c] = (uint8_t)(gf_mul(a0, 3) ^ a1 ^ a2 ^ gf_mul(a3, 2));
            }
        }
        for (int c = 0; c < 4; ++c)            /* AddRoundKey */
            for (int r = 0; r < 4; ++r) s[r][c] ^= rk[16 * round + 4 * c + r];
    }
    for (int c = 0; c < 4; ++c)
        for (int r = 0; r < 4; ++r) out[r + 4 * c] = s[r][c];
}

/* 128-bit integers travel as 4 little-endian 32-bit lanes; the AES input byte
 * in_j is byte (j mod 4) of lane j/4 (i.e. in_0 = X mod 256). */
static void lanes_to_bytes(const uint32_t x[4], uint8_t b[16]) {
    for (int j = 0; j < 16; ++j) b[j] = (uint8_t)(x[j / 4] >> (8 * (j % 4)));
}
static void bytes_to_lanes(const uint8_t b[16], uint32_t x[4]) {
    for (int l = 0; l < 4; ++l)
        x[l] = (uint32_t)b[4 * l] | ((uint32_t)b[4 * l + 1] << 8) |
               ((uint32_t)b[4 * l + 2] << 16) | ((uint32_t)b[4 * l + 3] << 24);
}

/* ======================================================================
 * Number theory and label sizes
 * ====================================================================== */

static int is_prime_u32(uint32_t n) {
    if (n < 2) return 0;
    for (uint32_t d = 2; d * d <= n; ++d)
        if (n % d == 0) return 0;
    return 1;
}

static int is_pow2_u32(uint32_t n) { return n >= 2 && (n & (n - 1)) == 0; }

static uint32_t gcd_u32(uint32_t a, uint32_t b) {
    while (b) {
        uint32_t t = a % b;
        a = b;
        b = t;
    }
    return a;
}

/* Radix of the first offset digit: R_m[0] is drawn from it and mapped to a
 * unit of Z_m (d + 1 for a prime m, 2d + 1 for m = 2^l, l >= 2). */
static uint32_t offset_first_radix(uint32_t m) { return (is_pow2_u32(m) && m > 2) ? m / 2 : m - 1; }
static uint32_t offset_first_unit(uint32_t m, uint32_t d) { return (is_pow2_u32(m) && m > 2) ? 2 * d + 1 : d + 1; }

static uint32_t inv_mod(uint32_t a, uint32_t m) {
    a %= m;
    for (uint32_t x = 1; x < m; ++x)
        if ((a * x) % m == 1) return x;
    return 0;
}

/* lambda_m = min{ lambda : m^lambda >= 2^128 } (integer test). */
static uint32_t lambda_of(uint32_t m) {
    const unsigned __int128 MAX = ~(unsigned __int128)0; /* 2^128 - 1 */
    unsigned __int128 p = 1;
    uint32_t lam = 0;
    for (;;) {
        if (p > MAX / m) return lam + 1; /* p*m > 2^128 - 1 */
        p *= m;
        ++lam;
    }
}

static uint32_t bits_of(uint32_t m) { /* bit length of m-1 */
    uint32_t b = 0, v = m - 1;
    while (v) { ++b; v >>= 1; }
    return b;
}
static uint32_t per_word(uint32_t m) { return 32u / bits_of(m); }
static uint32_t words_of(uint32_t m) { return (lambda_of(m) + per_word(m) - 1) / per_word(m); }

/* PK32: residue i lives in word i / g at bit offset b * (i mod g). */
static void pk32_pack(uint32_t m, const uint32_t *res, uint32_t *words) {
    uint32_t lam = lambda_of(m), b = bits_of(m), g = per_word(m), W = words_of(m);
    for (uint32_t w = 0; w < W; ++w) words[w] = 0;
    for (uint32_t i = 0; i < lam; ++i) words[i / g] |= res[i] << (b * (i % g));
}
static void pk32_unpack(uint32_t m, const uint32_t *words, uint32_t *res) {
    uint32_t lam = lambda_of(m), b = bits_of(m), g = per_word(m);
    uint32_t mask = (b == 32) ? 0xffffffffu : ((1u << b) - 1u);
    for (uint32_t i = 0; i < lam; ++i) res[i] = (words[i / g] >> (b * (i % g))) & mask;
}

/* Digits of the fraction V / 2^(32*nl) in the radices given:
 * h_i = floor(V_i * r_i / 2^(32 nl)),  V_{i+1} = V_i * r_i mod 2^(32 nl).
 * V is little-endian 32-bit limbs and is consumed. */
static void frac_digits(uint32_t *V, int nl, const uint32_t *radix, int count, uint32_t *out) {
    for (int i = 0; i < count; ++i) {
        uint64_t carry = 0;
        for (int l = 0; l < nl; ++l) {
            uint64_t t = (uint64_t)V[l] * radix[i] + carry;
            V[l] = (uint32_t)t;
            carry = t >> 32;
        }
        out[i] = (uint32_t)carry;
    }
}

/* Fixed hash key K = 00 01 02 ... 0f (the FIPS-197 Appendix C.1 key). */
static uint8_t HASH_RK[176];
static int hash_rk_ready = 0;
static const uint8_t *hash_round_keys(void) {
    if (!hash_rk_ready) {
        uint8_t key[16];
        for (int i = 0; i < 16; ++i) key[i] = (uint8_t)i;
        key_expansion(key, HASH_RK);
        hash_rk_ready = 1;
    }
    return HASH_RK;
}

/* The 128 n-bit value behind H_m(A, tau) (n = 1 if m == 2 else 2), with the
 * intermediate values the tests pin one by one:
 *   x = fold(PK32(A)): word w is XORed into 32-bit lane (w mod 4)
 *   u = sigma(x) = ((x_hi ^ x_lo) << 64) | x_hi   (linear orthomorphism;
 *       x_lo = lanes 0-1, x_hi = lanes 2-3)
 *   T_j = gadget_id * 2^96 + ((tau * 4 + j) mod 2^64)   (j < n; bits 64-95 zero)
 *   U_j = AES_K(u ^ T_j) ^ u ^ T_j                (Matyas-Meyer-Oseas)
 *   V = sum_j U_j 2^(128 j), returned as 4 n little-endian limbs. */
static void hash_value(uint32_t q, uint32_t m, const uint32_t *A, uint32_t gadget_id, uint64_t tau,
                       uint32_t x[4], uint32_t u[4], uint32_t V[8]) {
    const uint8_t *rk = hash_round_keys();
    uint32_t words[ORC_MAXLAMBDA];
    pk32_pack(q, A, words);
    for (int l = 0; l < 4; ++l) x[l] = 0;
    for (uint32_t w = 0; w < words_of(q); ++w) x[w % 4] ^= words[w];
    u[0] = x[2];
    u[1] = x[3];
    u[2] = x[2] ^ x[0];
    u[3] = x[3] ^ x[1];
    int n = (m == 2) ? 1 : 2;
    for (int l = 0; l < 8; ++l) V[l] = 0;
    for (int j = 0; j < n; ++j) {
        uint64_t tw = tau * 4u + (uint64_t)j;
        uint32_t T[4] = {(uint32_t)tw, (uint32_t)(tw >> 32), 0u, gadget_id};
        uint32_t in[4], ct[4];
        uint8_t ib[16], ob[16];
        for (int l = 0; l < 4; ++l) in[l] = u[l] ^ T[l];
        lanes_to_bytes(in, ib);
        aes_encrypt(rk, ib, ob);
        bytes_to_lanes(ob, ct);
        for (int l = 0; l < 4; ++l) V[4 * j + l] = ct[l] ^ u[l] ^ T[l];
    }
}

/* H_m(A, tau): A is a label over Z_q (lambda_q residues); the result is a
 * label over Z_m (lambda_m residues): the first lambda_m base-m digits of the
 * fraction V / 2^(128 n), V from hash_value(). */
static void hash_label(uint32_t q, uint32_t m, const uint32_t *A, uint32_t gadget_id, uint64_t tau,
                       uint32_t *out) {
    uint32_t x[4], u[4], V[8];
    hash_value(q, m, A, gadget_id, tau, x, u, V);
    int n = (m == 2) ? 1 : 2;
    uint32_t lam = lambda_of(m);
    uint32_t radix[ORC_MAXLAMBDA];
    for (uint32_t i = 0; i < lam; ++i) radix[i] = m;
    frac_digits(V, 4 * n, radix, (int)lam, out);
}

/* Garbler PRG: K_seed = seed as 16 little-endian bytes;
 * rho(stream, idx) = AES_{K_seed}(C_0) + 2^128 AES_{K_seed}(C_1),
 * C_h = stream * 2^120 + ((idx * 2 + h) mod 2^64), returned as 8
 * little-endian limbs. */
static void prg_value(const uint8_t rk_seed[176], uint32_t stream, uint64_t idx, uint32_t V[8]) {
    for (int h = 0; h < 2; ++h) {
        uint64_t lo = idx * 2u + (uint64_t)h;
        uint32_t C[4] = {(uint32_t)lo, (uint32_t)(lo >> 32), 0u, stream << 24};
        uint8_t ib[16], ob[16];
        uint32_t ct[4];
        lanes_to_bytes(C, ib);
        aes_encrypt(rk_seed, ib, ob);
        bytes_to_lanes(ob, ct);
        for (int l = 0; l < 4; ++l) V[4 * h + l] = ct[l];
    }
}

/* A label read off rho(stream, idx) as fraction digits; the first radix is
 * offset_first_radix(m) when first_minus_one is set (offsets). */
static void prg_label(const uint8_t rk_seed[176], uint32_t stream, uint64_t idx, uint32_t m,
                      int first_minus_one, uint32_t *out) {
    uint32_t V[8];
    prg_value(rk_seed, stream, idx, V);
    uint32_t lam = lambda_of(m);
    uint32_t radix[ORC_MAXLAMBDA];
    for (uint32_t i = 0; i < lam; ++i) radix[i] = m;
    if (first_minus_one) radix[0] = offset_first_radix(m);
    frac_digits(V, 8, radix, (int)lam, out);
}

static void seed_round_keys(uint64_t seed, uint8_t rk[176]) {
    uint8_t key[16];
    for (int i = 0; i < 16; ++i) key[i] = (i < 8) ? (uint8_t)(seed >> (8 * i)) : 0;
    key_expansion(key, rk);
}

/* ======================================================================
 * Parameters, gate list, layouts
 * ====================================================================== */

typedef struct {
    uint32_t src, dst, kind, coeff; /* kind 0: sub (L <- coeff (L - E)), 1: acc (A <- A + coeff E) */
    uint32_t phase;                 /* 0 = A, 1 = B */
} orc_gate;

typedef struct {
    uint32_t k, t, u;
    uint32_t m[ORC_MAXK];
    uint32_t S[ORC_MAXK], R[ORC_MAXK];
    uint32_t is_scale[ORC_MAXK];
    uint32_t lam[ORC_MAXK], W[ORC_MAXK];
    uint64_t P, s;
    uint32_t G;
    orc_gate gate[ORC_MAXGATES];
} orc_plan;

static int make_plan(const orc_params *p, orc_plan *pl) {
    if (!p || !pl) return ORC_ENULL;
    if (p->k < 2 || p->k > 15) return ORC_EPARAM;
    if (p->t < 1 || p->t > p->k - 1) return ORC_EPARAM;
    memset(pl, 0, sizeof *pl);
    pl->k = p->k;
    pl->t = p->t;
    unsigned __int128 P = 1;
    for (uint32_t i = 0; i < p->k; ++i) {
        uint32_t m = p->moduli[i];
        if (m < 2 || m > 255 || !(is_prime_u32(m) || is_pow2_u32(m))) return ORC_EPARAM;
        if (i > 0 && m <= p->moduli[i - 1]) return ORC_EPARAM;
        for (uint32_t j = 0; j < i; ++j)
            if (gcd_u32(m, p->moduli[j]) != 1) return ORC_EPARAM;
        pl->m[i] = m;
        pl->lam[i] = lambda_of(m);
        pl->W[i] = words_of(m);
        P *= m;
    }
    if (P >= ((unsigned __int128)1 << 63)) return ORC_EPARAM;
    uint64_t s = 1;
    for (uint32_t a = 0; a < p->t; ++a) {
        uint32_t si = p->scale_idx[a];
        if (si >= p->k) return ORC_EPARAM;
        if (a > 0 && si <= p->scale_idx[a - 1]) return ORC_EPARAM;
        pl->S[a] = si;
        pl->is_scale[si] = 1;
        s *= p->moduli[si];
    }
    pl->P = (uint64_t)P;
    pl->s = s;
    pl->u = 0;
    for (uint32_t i = 0; i < p->k; ++i)
        if (!pl->is_scale[i]) pl->R[pl->u++] = i;
    /* Gate list: Phase A over S (targets: later S, then R); Phase B over R
     * (targets: later R, then S with MRS weights). */
    uint32_t G = 0;
    for (uint32_t a = 0; a < pl->t; ++a) {
        uint32_t src = pl->S[a];
        uint32_t tg[ORC_MAXK], nt = 0;
        for (uint32_t b = a + 1; b < pl->t; ++b) tg[nt++] = pl->S[b];
        for (uint32_t b = 0; b < pl->u; ++b) tg[nt++] = pl->R[b];
        for (uint32_t j = 0; j < nt; ++j) {
            orc_gate *g = &pl->gate[G++];
            g->src = src; g->dst = tg[j]; g->kind = 0; g->phase = 0;
            g->coeff = inv_mod(pl->m[src], pl->m[tg[j]]);
        }
    }
    for (uint32_t b = 0; b < pl->u; ++b) {
        uint32_t src = pl->R[b];
        for (uint32_t c = b + 1; c < pl->u; ++c) {
            orc_gate *g = &pl->gate[G++];
            g->src = src; g->dst = pl->R[c]; g->kind = 0; g->phase = 1;
            g->coeff = inv_mod(pl->m[src], pl->m[pl->R[c]]);
        }
        for (uint32_t a = 0; a < pl->t; ++a) {
            uint32_t dst = pl->S[a], md = pl->m[dst];
            uint32_t w = 1;
            for (uint32_t c = 0; c < b; ++c) w = (w * (pl->m[pl->R[c]] % md)) % md;
            orc_gate *g = &pl->gate[G++];
            g->src = src; g->dst = dst; g->kind = 1; g->phase = 1; g->coeff = w;
        }
    }
    pl->G = G;
    return ORC_OK;
}

/* Label tensor layout: for modulus i, a block of W_i * n words; word w of
 * gadget a at block + w * n + a.  Offsets: one PK32 label per modulus,
 * concatenated.  Tables: gate blocks in gate order; gate g (input modulus q,
 * output modulus m) holds n * (q-1) * W_m words, row of colour c (1..q-1) of
 * gadget a at ((a * (q-1) + (c-1)) * W_m + w). */
static uint64_t label_block(const orc_plan *pl, uint32_t i, uint64_t n) {
    uint64_t off = 0;
    for (uint32_t j = 0; j < i; ++j) off += (uint64_t)pl->W[j] * n;
    return off;
}
static uint32_t offset_block(const orc_plan *pl, uint32_t i) {
    uint32_t off = 0;
    for (uint32_t j = 0; j < i; ++j) off += pl->W[j];
    return off;
}
static uint64_t table_block(const orc_plan *pl, uint32_t g, uint64_t n) {
    uint64_t off = 0;
    for (uint32_t h = 0; h < g; ++h) {
        const orc_gate *gt = &pl->gate[h];
        off += n * (uint64_t)(pl->m[gt->src] - 1) * pl->W[gt->dst];
    }
    return off;
}

static void read_label(const orc_plan *pl, const uint32_t *buf, uint32_t i, uint64_t n, uint64_t a,
                       uint32_t *res) {
    uint32_t words[ORC_MAXLAMBDA];
    uint64_t base = label_block(pl, i, n);
    for (uint32_t w = 0; w < pl->W[i]; ++w) words[w] = buf[base + (uint64_t)w * n + a];
    pk32_unpack(pl->m[i], words, res);
}
static void write_label(const orc_plan *pl, uint32_t *buf, uint32_t i, uint64_t n, uint64_t a,
                        const uint32_t *res) {
    uint32_t words[ORC_MAXLAMBDA];
    pk32_pack(pl->m[i], res, words);
    uint64_t base = label_block(pl, i, n);
    for (uint32_t w = 0; w < pl->W[i]; ++w) buf[base + (uint64_t)w * n + a] = words[w];
}

/* Componentwise label arithmetic over Z_m. */
static void lab_axpy(uint32_t m, uint32_t lam, uint32_t *y, const uint32_t *x, uint32_t c) {
    for (uint32_t i = 0; i < lam; ++i) y[i] = (uint32_t)((y[i] + (uint64_t)c * x[i]) % m);
}
static void lab_sub_scale(uint32_t m, uint32_t lam, uint32_t *y, const uint32_t *e, uint32_t c) {
    for (uint32_t i = 0; i < lam; ++i) y[i] = (uint32_t)(((uint64_t)c * ((y[i] + m - e[i]) % m)) % m);
}

/* ======================================================================
 * Public entry points
 * ====================================================================== */

int orc_check_params(const orc_params *p) {
    orc_plan pl;
    return make_plan(p, &pl);
}

int orc_sizes(const orc_params *p, uint64_t n, uint64_t *label_words, uint64_t *table_words,
              uint32_t *gates, uint32_t *offset_words) {
    orc_plan pl;
    int rc = make_plan(p, &pl);
    if (rc) return rc;
    if (label_words) *label_words = label_block(&pl, pl.k, n);
    if (table_words) *table_words = table_block(&pl, pl.G, n);
    if (gates) *gates = pl.G;
    if (offset_words) *offset_words = offset_block(&pl, pl.k);
    return ORC_OK;
}

/* Gate list export: arrays of length G. */
int orc_gate_list(const orc_params *p, uint32_t *src, uint32_t *dst, uint32_t *kind, uint32_t *coeff,
                  uint32_t *phase) {
    orc_plan pl;
    int rc = make_plan(p, &pl);
    if (rc) return rc;
    for (uint32_t g = 0; g < pl.G; ++g) {
        src[g] = pl.gate[g].src;
        dst[g] = pl.gate[g].dst;
        kind[g] = pl.gate[g].kind;
        coeff[g] = pl.gate[g].coeff;
        phase[g] = pl.gate[g].phase;
    }
    return ORC_OK;
}

uint32_t orc_lambda(uint32_t m) { return lambda_of(m); }
uint32_t orc_words(uint32_t m) { return words_of(m); }

void orc_sbox(uint8_t *out) {
    ensure_sbox();
    memcpy(out, SBOX, 256);
}

void orc_aes128(const uint8_t *key, const uint8_t *in, uint8_t *out) {
    uint8_t rk[176];
    key_expansion(key, rk);
    aes_encrypt(rk, in, out);
}

void orc_aes128_key_expansion(const uint8_t *key, uint8_t *w176) { key_expansion(key, w176); }

void orc_frac_digits(uint32_t *V, int nl, const uint32_t *radix, int count, uint32_t *out) {
    frac_digits(V, nl, radix, count, out);
}

void orc_pk32_pack(uint32_t m, const uint32_t *res, uint32_t *words) { pk32_pack(m, res, words); }
void orc_pk32_unpack(uint32_t m, const uint32_t *words, uint32_t *res) { pk32_unpack(m, words, res); }

/* Hash of one label given as residues; out gets lambda_m residues. */
void orc_hash(uint32_t q, uint32_t m, const uint32_t *A, uint32_t gadget_id, uint64_t tau, uint32_t *out) {
    hash_label(q, m, A, gadget_id, tau, out);
}

/* The intermediate values of the hash (fold x, sigma u, and the 128 n-bit
 * value V before its digits are taken), for the tests that pin each step. */
void orc_hash_parts(uint32_t q, uint32_t m, const uint32_t *A, uint32_t gadget_id, uint64_t tau, uint32_t *x,
                    uint32_t *u, uint32_t *V) {
    hash_value(q, m, A, gadget_id, tau, x, u, V);
}

/* rho(stream, idx) under the seed's key, as 8 little-endian limbs. */
void orc_prg_value(uint64_t seed, uint32_t stream, uint64_t idx, uint32_t *V) {
    uint8_t rk[176];
    seed_round_keys(seed, rk);
    prg_value(rk, stream, idx, V);
}

void orc_prg_label(uint64_t seed, uint32_t stream, uint64_t idx, uint32_t m, int first_minus_one,
                   uint32_t *out) {
    uint8_t rk[176];
    seed_round_keys(seed, rk);
    prg_label(rk, stream, idx, m, first_minus_one, out);
}

/* Offsets R_m: digits of rho(1, i) with radices (r0, m, ..., m), then R_m[0]
 * mapped to a unit of Z_m so that the m colours of a wire are distinct:
 * r0 = m-1 and R_m[0] = d+1 for a prime m; r0 = m/2 and R_m[0] = 2d+1 for
 * m = 2^l, l >= 2. */
static void make_offsets(const orc_plan *pl, const uint8_t rk_seed[176], uint32_t R[ORC_MAXK][ORC_MAXLAMBDA]) {
    for (uint32_t i = 0; i < pl->k; ++i) {
        prg_label(rk_seed, 1u, i, pl->m[i], 1, R[i]);
        R[i][0] = offset_first_unit(pl->m[i], R[i][0]);
    }
}

/* Garble (or trace) gadget a.  All labels as residue arrays.
 *   zin  : k input zero-labels Z_{a,i}
 *   zout : k output zero-labels O^0_{a,i}
 *   tables/n/a_local : where rows go (tables may be NULL)
 *   trace_* : optional per-gate records (NULL to skip) */
typedef struct {
    uint32_t *slots;   /* (G+1) x k x ORC_MAXLAMBDA: garbler zero-labels of the k slots */
    uint32_t *gate_in; /* G x ORC_MAXLAMBDA: A^0 (zero-label of the digit wire)        */
    uint32_t *gate_out;/* G x ORC_MAXLAMBDA: B^0 (zero-label of the projected output)  */
    uint32_t *out_R;   /* k x ORC_MAXLAMBDA: zero-labels of the R outputs after Phase A */
} orc_gtrace;

static void garble_one(const orc_plan *pl, uint32_t gadget_id, uint64_t a, uint32_t R[ORC_MAXK][ORC_MAXLAMBDA],
                       uint32_t zin[ORC_MAXK][ORC_MAXLAMBDA], uint32_t zout[ORC_MAXK][ORC_MAXLAMBDA],
                       uint32_t *tables, uint64_t n, uint64_t a_local, orc_gtrace *tr) {
    const uint32_t k = pl->k;
    uint32_t Wl[ORC_MAXK][ORC_MAXLAMBDA];
    uint32_t outR[ORC_MAXK][ORC_MAXLAMBDA];
    uint64_t half = pl->P / 2, down = half / pl->s; /* floor(P/2), floor(floor(P/2)/s) */
    /* ShiftUp: G^0_i = Z_i - (floor(P/2) mod m_i) R_i. */
    for (uint32_t i = 0; i < k; ++i) {
        uint32_t m = pl->m[i];
        uint32_t c = (uint32_t)((m - half % m) % m);
        memcpy(Wl[i], zin[i], sizeof Wl[i]);
        lab_axpy(m, pl->lam[i], Wl[i], R[i], c);
    }
    int phaseB = 0;
    for (uint32_t g = 0; g < pl->G; ++g) {
        const orc_gate *gt = &pl->gate[g];
        if (gt->phase == 1 && !phaseB) {
            phaseB = 1;
            for (uint32_t b = 0; b < pl->u; ++b) memcpy(outR[pl->R[b]], Wl[pl->R[b]], sizeof outR[0]);
            for (uint32_t a2 = 0; a2 < pl->t; ++a2) memset(Wl[pl->S[a2]], 0, sizeof Wl[0]);
        }
        if (tr && tr->slots)
            for (uint32_t i = 0; i < k; ++i)
                memcpy(tr->slots + ((uint64_t)g * k + i) * ORC_MAXLAMBDA, Wl[i], sizeof Wl[i]);
        uint32_t src = gt->src, dst = gt->dst;
        uint32_t q = pl->m[src], m = pl->m[dst];
        uint32_t lq = pl->lam[src], lm = pl->lam[dst];
        uint64_t tau = a * (uint64_t)pl->G + g;
        const uint32_t *A0 = Wl[src];
        /* v0: the value whose input label has colour 0. */
        uint32_t v0 = (uint32_t)(((uint64_t)(q - A0[0] % q) % q) * inv_mod(R[src][0], q) % q);
        uint32_t Av[ORC_MAXLAMBDA], H[ORC_MAXLAMBDA], B0[ORC_MAXLAMBDA];
        memcpy(Av, A0, sizeof Av);
        lab_axpy(q, lq, Av, R[src], v0);
        hash_label(q, m, Av, gadget_id, tau, H);
        /* Row reduction: B^0 = H(A_{v0}) - (v0 mod m) R_m. */
        memcpy(B0, H, sizeof B0);
        lab_axpy(m, lm, B0, R[dst], (m - v0 % m) % m);
        if (tables) {
            uint64_t blk = table_block(pl, g, n);
            for (uint32_t v = 0; v < q; ++v) {
                if (v == v0) continue;
                uint32_t c = (uint32_t)((A0[0] + (uint64_t)v * R[src][0]) % q);
                uint32_t Ax[ORC_MAXLAMBDA], Hx[ORC_MAXLAMBDA], row[ORC_MAXLAMBDA], words[ORC_MAXLAMBDA];
                memcpy(Ax, A0, sizeof Ax);
                lab_axpy(q, lq, Ax, R[src], v);
                hash_label(q, m, Ax, gadget_id, tau, Hx);
                /* row[c] = B^0 + (v mod m) R_m - H(A_v) */
                memcpy(row, B0, sizeof row);
                lab_axpy(m, lm, row, R[dst], v % m);
                for (uint32_t i = 0; i < lm; ++i) row[i] = (row[i] + m - Hx[i]) % m;
                pk32_pack(m, row, words);
                uint64_t at = blk + ((a_local * (q - 1) + (c - 1)) * (uint64_t)pl->W[dst]);
                for (uint32_t w = 0; w < pl->W[dst]; ++w) tables[at + w] = words[w];
            }
        }
        if (tr && tr->gate_in) memcpy(tr->gate_in + (uint64_t)g * ORC_MAXLAMBDA, A0, sizeof Av);
        if (tr && tr->gate_out) memcpy(tr->gate_out + (uint64_t)g * ORC_MAXLAMBDA, B0, sizeof B0);
        if (gt->kind == 0) lab_sub_scale(m, lm, Wl[dst], B0, gt->coeff);
        else lab_axpy(m, lm, Wl[dst], B0, gt->coeff);
    }
    if (tr && tr->slots)
        for (uint32_t i = 0; i < k; ++i)
            memcpy(tr->slots + ((uint64_t)pl->G * k + i) * ORC_MAXLAMBDA, Wl[i], sizeof Wl[i]);
    if (tr && tr->out_R)
        for (uint32_t b = 0; b < pl->u; ++b)
            memcpy(tr->out_R + (uint64_t)pl->R[b] * ORC_MAXLAMBDA, outR[pl->R[b]], sizeof outR[0]);
    /* Outputs: R wires from the end of Phase A, S wires from the accumulators;
     * ShiftDown: O^0_i = out_i + (P/(2s) mod m_i) R_i. */
    for (uint32_t i = 0; i < k; ++i) {
        uint32_t m = pl->m[i];
        memcpy(zout[i], pl->is_scale[i] ? Wl[i] : outR[i], sizeof zout[i]);
        lab_axpy(m, pl->lam[i], zout[i], R[i], (uint32_t)(down % m));
    }
}

/* Garble gadgets a_begin .. a_begin+count-1.  Buffers use n = count as the
 * structure-of-arrays stride.  offsets: sum W words.  in_zero/out_zero:
 * label tensors.  tables: may be NULL (zero-label path only: one hash per
 * gate, which yields the output zero-labels without any row). */
int orc_garble(const orc_params *p, uint64_t a_begin, uint64_t count, uint32_t *offsets, uint32_t *in_zero,
               uint32_t *out_zero, uint32_t *tables) {
    orc_plan pl;
    int rc = make_plan(p, &pl);
    if (rc) return rc;
    if (!offsets || !in_zero || !out_zero) return ORC_ENULL;
    uint8_t rk_seed[176];
    seed_round_keys(p->seed, rk_seed);
    uint32_t gadget_id = (uint32_t)p->seed;
    static uint32_t R[ORC_MAXK][ORC_MAXLAMBDA];
    memset(R, 0, sizeof R);
    make_offsets(&pl, rk_seed, R);
    for (uint32_t i = 0; i < pl.k; ++i) {
        uint32_t words[ORC_MAXLAMBDA];
        pk32_pack(pl.m[i], R[i], words);
        memcpy(offsets + offset_block(&pl, i), words, pl.W[i] * sizeof(uint32_t));
    }
    for (uint64_t al = 0; al < count; ++al) {
        uint64_t a = a_begin + al;
        uint32_t zin[ORC_MAXK][ORC_MAXLAMBDA], zout[ORC_MAXK][ORC_MAXLAMBDA];
        memset(zin, 0, sizeof zin);
        for (uint32_t i = 0; i < pl.k; ++i) prg_label(rk_seed, 2u, a * pl.k + i, pl.m[i], 0, zin[i]);
        garble_one(&pl, gadget_id, a, R, zin, zout, tables, count, al, NULL);
        for (uint32_t i = 0; i < pl.k; ++i) {
            write_label(&pl, in_zero, i, count, al, zin[i]);
            write_label(&pl, out_zero, i, count, al, zout[i]);
        }
    }
    return ORC_OK;
}

/* Garble gadgets a_begin .. a_begin+count-1 on input zero-labels the caller
 * gives (the output zero-labels of the layer that feeds the gadget: in a
 * circuit every wire's zero-label comes from the gate that produces it,
 * Sec. 2.3), instead of drawing them from the PRG.  Everything else is as in
 * orc_garble: offsets from the seed, tweaks from the global gadget index. */
int orc_garble_given(const orc_params *p, uint64_t a_begin, uint64_t count, uint32_t *offsets,
                     const uint32_t *in_zero, uint32_t *out_zero, uint32_t *tables) {
    orc_plan pl;
    int rc = make_plan(p, &pl);
    if (rc) return rc;
    if (!offsets || !in_zero || !out_zero) return ORC_ENULL;
    uint8_t rk_seed[176];
    seed_round_keys(p->seed, rk_seed);
    uint32_t gadget_id = (uint32_t)p->seed;
    static uint32_t R[ORC_MAXK][ORC_MAXLAMBDA];
    memset(R, 0, sizeof R);
    make_offsets(&pl, rk_seed, R);
    for (uint32_t i = 0; i < pl.k; ++i) {
        uint32_t words[ORC_MAXLAMBDA];
        pk32_pack(pl.m[i], R[i], words);
        memcpy(offsets + offset_block(&pl, i), words, pl.W[i] * sizeof(uint32_t));
    }
    for (uint64_t al = 0; al < count; ++al) {
        uint64_t a = a_begin + al;
        uint32_t zin[ORC_MAXK][ORC_MAXLAMBDA], zout[ORC_MAXK][ORC_MAXLAMBDA];
        memset(zin, 0, sizeof zin);
        for (uint32_t i = 0; i < pl.k; ++i) read_label(&pl, in_zero, i, count, al, zin[i]);
        garble_one(&pl, gadget_id, a, R, zin, zout, tables, count, al, NULL);
        for (uint32_t i = 0; i < pl.k; ++i) write_label(&pl, out_zero, i, count, al, zout[i]);
    }
    return ORC_OK;
}

/* X_{a,i} = Z_{a,i} + ((x_a mod P) mod m_i) R_i. */
int orc_encode(const orc_params *p, uint64_t count, const int64_t *x, const uint32_t *zero,
               const uint32_t *offsets, uint32_t *labels) {
    orc_plan pl;
    int rc = make_plan(p, &pl);
    if (rc) return rc;
    if (!x || !zero || !offsets || !labels) return ORC_ENULL;
    for (uint64_t a = 0; a < count; ++a) {
        int64_t r = x[a] % (int64_t)pl.P;
        if (r < 0) r += (int64_t)pl.P;
        for (uint32_t i = 0; i < pl.k; ++i) {
            uint32_t m = pl.m[i];
            uint32_t Z[ORC_MAXLAMBDA], Rm[ORC_MAXLAMBDA];
            read_label(&pl, zero, i, count, a, Z);
            pk32_unpack(m, offsets + offset_block(&pl, i), Rm);
            lab_axpy(m, pl.lam[i], Z, Rm, (uint32_t)((uint64_t)r % m));
            write_label(&pl, labels, i, count, a, Z);
        }
    }
    return ORC_OK;
}

/* Evaluate gadget a given its k input labels (residue arrays). */
static void eval_one(const orc_plan *pl, uint32_t gadget_id, uint64_t a, uint32_t L[ORC_MAXK][ORC_MAXLAMBDA],
                     const uint32_t *tables, uint64_t n, uint64_t a_local, uint32_t out[ORC_MAXK][ORC_MAXLAMBDA],
                     orc_gtrace *tr) {
    const uint32_t k = pl->k;
    uint32_t outR[ORC_MAXK][ORC_MAXLAMBDA];
    int phaseB = 0;
    for (uint32_t g = 0; g < pl->G; ++g) {
        const orc_gate *gt = &pl->gate[g];
        if (gt->phase == 1 && !phaseB) {
            phaseB = 1;
            for (uint32_t b = 0; b < pl->u; ++b) memcpy(outR[pl->R[b]], L[pl->R[b]], sizeof outR[0]);
            for (uint32_t a2 = 0; a2 < pl->t; ++a2) memset(L[pl->S[a2]], 0, sizeof L[0]);
        }
        if (tr && tr->slots)
            for (uint32_t i = 0; i < k; ++i)
                memcpy(tr->slots + ((uint64_t)g * k + i) * ORC_MAXLAMBDA, L[i], sizeof L[i]);
        uint32_t src = gt->src, dst = gt->dst;
        uint32_t q = pl->m[src], m = pl->m[dst];
        uint32_t lm = pl->lam[dst];
        uint64_t tau = a * (uint64_t)pl->G + g;
        const uint32_t *A = L[src];
        uint32_t E[ORC_MAXLAMBDA];
        hash_label(q, m, A, gadget_id, tau, E);
        uint32_t c = A[0];
        if (c != 0) {
            uint32_t words[ORC_MAXLAMBDA], row[ORC_MAXLAMBDA];
            uint64_t at = table_block(pl, g, n) + ((a_local * (q - 1) + (c - 1)) * (uint64_t)pl->W[dst]);
            for (uint32_t w = 0; w < pl->W[dst]; ++w) words[w] = tables[at + w];
            pk32_unpack(m, words, row);
            for (uint32_t i = 0; i < lm; ++i) E[i] = (E[i] + row[i]) % m;
        }
        if (tr && tr->gate_in) memcpy(tr->gate_in + (uint64_t)g * ORC_MAXLAMBDA, A, ORC_MAXLAMBDA * 4);
        if (tr && tr->gate_out) memcpy(tr->gate_out + (uint64_t)g * ORC_MAXLAMBDA, E, sizeof E);
        if (gt->kind == 0) lab_sub_scale(m, lm, L[dst], E, gt->coeff);
        else lab_axpy(m, lm, L[dst], E, gt->coeff);
    }
    if (tr && tr->slots)
        for (uint32_t i = 0; i < k; ++i)
            memcpy(tr->slots + ((uint64_t)pl->G * k + i) * ORC_MAXLAMBDA, L[i], sizeof L[i]);
    if (tr && tr->out_R)
        for (uint32_t b = 0; b < pl->u; ++b)
            memcpy(tr->out_R + (uint64_t)pl->R[b] * ORC_MAXLAMBDA, outR[pl->R[b]], sizeof outR[0]);
    for (uint32_t i = 0; i < k; ++i) memcpy(out[i], pl->is_scale[i] ? L[i] : outR[i], sizeof out[i]);
}

/* Evaluate gadgets a_begin .. a_begin+count-1 (stride n = count). */
int orc_eval(const orc_params *p, uint64_t a_begin, uint64_t count, const uint32_t *in_labels,
             const uint32_t *tables, uint32_t *out_labels) {
    orc_plan pl;
    int rc = make_plan(p, &pl);
    if (rc) return rc;
    if (!in_labels || !tables || !out_labels) return ORC_ENULL;
    uint32_t gadget_id = (uint32_t)p->seed;
    for (uint64_t al = 0; al < count; ++al) {
        uint32_t L[ORC_MAXK][ORC_MAXLAMBDA], out[ORC_MAXK][ORC_MAXLAMBDA];
        memset(L, 0, sizeof L);
        for (uint32_t i = 0; i < pl.k; ++i) read_label(&pl, in_labels, i, count, al, L[i]);
        eval_one(&pl, gadget_id, a_begin + al, L, tables, count, al, out, NULL);
        for (uint32_t i = 0; i < pl.k; ++i) write_label(&pl, out_labels, i, count, al, out[i]);
    }
    return ORC_OK;
}

/* Decode: v_i = (Y_i[0] - O_i[0]) R_i[0]^{-1} mod m_i; the label is valid iff
 * Y_i = O_i + v_i R_i componentwise; y = CRT(v) mapped to the signed range
 * [-floor(P/2), ceil(P/2) - 1] (Sec. 2.4; [-P/2, P/2) for even P).  bad[a] = 1
 * for a gadget with any invalid residue label. */
int orc_decode(const orc_params *p, uint64_t count, const uint32_t *out_labels, const uint32_t *out_zero,
               const uint32_t *offsets, int64_t *y, uint8_t *bad) {
    orc_plan pl;
    int rc = make_plan(p, &pl);
    if (rc) return rc;
    if (!out_labels || !out_zero || !offsets || !y || !bad) return ORC_ENULL;
    for (uint64_t a = 0; a < count; ++a) {
        uint32_t v[ORC_MAXK];
        int ok = 1;
        for (uint32_t i = 0; i < pl.k; ++i) {
            uint32_t m = pl.m[i];
            uint32_t Y[ORC_MAXLAMBDA], O[ORC_MAXLAMBDA], Rm[ORC_MAXLAMBDA];
            read_label(&pl, out_labels, i, count, a, Y);
            read_label(&pl, out_zero, i, count, a, O);
            pk32_unpack(m, offsets + offset_block(&pl, i), Rm);
            v[i] = ((Y[0] + m - O[0]) % m) * inv_mod(Rm[0], m) % m;
            for (uint32_t j = 0; j < pl.lam[i]; ++j)
                if (Y[j] != (O[j] + v[i] * Rm[j]) % m) ok = 0;
        }
        /* CRT by incremental search of one coefficient per modulus. */
        unsigned __int128 acc = 0, M = 1;
        for (uint32_t i = 0; i < pl.k; ++i) {
            uint32_t m = pl.m[i];
            for (uint32_t tt = 0; tt < m; ++tt) {
                if ((uint32_t)((acc + (unsigned __int128)tt * M) % m) == v[i]) {
                    acc += (unsigned __int128)tt * M;
                    break;
                }
            }
            M *= m;
        }
        int64_t val = (int64_t)acc;
        if ((uint64_t)val >= (pl.P + 1) / 2) val -= (int64_t)pl.P; /* [-floor(P/2), ceil(P/2) - 1] */
        y[a] = val;
        bad[a] = (uint8_t)!ok;
    }
    return ORC_OK;
}

/* Full trace of one gadget a with signed input x: garbler and evaluator side
 * by side.  Every array is residues with row stride ORC_MAXLAMBDA:
 *   offsets_res  : k rows (R_i)
 *   gb_slots/ev_slots : (G+1) x k rows (slot labels before each gate, final)
 *   gb_in/ev_in  : G rows (A^0 / A of the digit wire)
 *   gb_out/ev_out: G rows (B^0 / E, the projected label)
 *   gb_outR/ev_outR : k rows (R wires after Phase A; S rows unused)
 *   gb_final/ev_final: k rows (O^0 after ShiftDown / evaluator output) */
int orc_trace(const orc_params *p, uint64_t a, int64_t x, uint32_t *offsets_res, uint32_t *gb_slots,
              uint32_t *ev_slots, uint32_t *gb_in, uint32_t *ev_in, uint32_t *gb_out, uint32_t *ev_out,
              uint32_t *gb_outR, uint32_t *ev_outR, uint32_t *gb_final, uint32_t *ev_final) {
    orc_plan pl;
    int rc = make_plan(p, &pl);
    if (rc) return rc;
    uint8_t rk_seed[176];
    seed_round_keys(p->seed, rk_seed);
    uint32_t gadget_id = (uint32_t)p->seed;
    static uint32_t R[ORC_MAXK][ORC_MAXLAMBDA];
    memset(R, 0, sizeof R);
    make_offsets(&pl, rk_seed, R);
    uint32_t zin[ORC_MAXK][ORC_MAXLAMBDA], zout[ORC_MAXK][ORC_MAXLAMBDA];
    memset(zin, 0, sizeof zin);
    for (uint32_t i = 0; i < pl.k; ++i) prg_label(rk_seed, 2u, a * pl.k + i, pl.m[i], 0, zin[i]);
    /* Tables for this single gadget (n = 1). */
    uint64_t tw = table_block(&pl, pl.G, 1);
    uint32_t *tables = (uint32_t *)calloc(tw ? tw : 1, sizeof(uint32_t));
    if (!tables) return ORC_ENULL;
    orc_gtrace gtr = {gb_slots, gb_in, gb_out, gb_outR};
    garble_one(&pl, gadget_id, a, R, zin, zout, tables, 1, 0, &gtr);
    /* Encode x against the input zero-labels, then evaluate. */
    int64_t r = x % (int64_t)pl.P;
    if (r < 0) r += (int64_t)pl.P;
    uint32_t L[ORC_MAXK][ORC_MAXLAMBDA], out[ORC_MAXK][ORC_MAXLAMBDA];
    memset(L, 0, sizeof L);
    for (uint32_t i = 0; i < pl.k; ++i) {
        memcpy(L[i], zin[i], sizeof L[i]);
        lab_axpy(pl.m[i], pl.lam[i], L[i], R[i], (uint32_t)((uint64_t)r % pl.m[i]));
    }
    orc_gtrace etr = {ev_slots, ev_in, ev_out, ev_outR};
    eval_one(&pl, gadget_id, a, L, tables, 1, 0, out, &etr);
    free(tables);
    for (uint32_t i = 0; i < pl.k; ++i) {
        if (offsets_res) memcpy(offsets_res + (uint64_t)i * ORC_MAXLAMBDA, R[i], sizeof R[i]);
        if (gb_final) memcpy(gb_final + (uint64_t)i * ORC_MAXLAMBDA, zout[i], sizeof zout[i]);
        if (ev_final) memcpy(ev_final + (uint64_t)i * ORC_MAXLAMBDA, out[i], sizeof out[i]);
    }
    return ORC_OK;
}
