/*
 * Drives the C oracle (oracle/gc_oracle.c) end to end on small bases so that
 * tests/test_sanitizers.py can run it under the address and
 * undefined-behaviour sanitizers: garble (with and without tables, at the
 * start of the index range and far into it), encode every input of the
 * signed range (or a spread of it), evaluate, decode, trace one gadget, and
 * call the hash and PRG helpers with extreme tweaks and counters.  Exit
 * status 0 when every decode returns floor((x + r)/s), r = floor(P/2) mod s,
 * with every label valid (the value the gadget computes, Sec. 3.2 and 3.4).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    uint32_t k;
    uint32_t moduli[16];
    uint32_t t;
    uint32_t scale_idx[16];
    uint64_t n;
    uint64_t seed;
} orc_params;

int orc_sizes(const orc_params *p, uint64_t n, uint64_t *label_words, uint64_t *table_words, uint32_t *gates,
              uint32_t *offset_words);
int orc_garble(const orc_params *p, uint64_t a_begin, uint64_t count, uint32_t *offsets, uint32_t *in_zero,
               uint32_t *out_zero, uint32_t *tables);
int orc_encode(const orc_params *p, uint64_t count, const int64_t *x, const uint32_t *zero, const uint32_t *offsets,
               uint32_t *labels);
int orc_eval(const orc_params *p, uint64_t a_begin, uint64_t count, const uint32_t *in_labels, const uint32_t *tables,
             uint32_t *out_labels);
int orc_decode(const orc_params *p, uint64_t count, const uint32_t *out_labels, const uint32_t *out_zero,
               const uint32_t *offsets, int64_t *y, uint8_t *bad);
int orc_trace(const orc_params *p, uint64_t a, int64_t x, uint32_t *offsets_res, uint32_t *gb_slots,
              uint32_t *ev_slots, uint32_t *gb_in, uint32_t *ev_in, uint32_t *gb_out, uint32_t *ev_out,
              uint32_t *gb_outR, uint32_t *ev_outR, uint32_t *gb_final, uint32_t *ev_final);
void orc_hash_parts(uint32_t q, uint32_t m, const uint32_t *A, uint32_t gadget_id, uint64_t tau, uint32_t *x,
                    uint32_t *u, uint32_t *V);
void orc_prg_label(uint64_t seed, uint32_t stream, uint64_t idx, uint32_t m, int first_minus_one, uint32_t *out);

#define MAXLAMBDA 128

static int failures = 0;

static int64_t floor_div(int64_t a, int64_t b) {
    int64_t q = a / b;
    if ((a % b != 0) && ((a < 0) != (b < 0))) --q;
    return q;
}

static void run_base(const uint32_t *moduli, uint32_t k, const uint32_t *S, uint32_t t, uint64_t a0, uint64_t seed,
                     uint64_t most) {
    orc_params p;
    memset(&p, 0, sizeof p);
    p.k = k;
    p.t = t;
    p.seed = seed;
    int64_t P = 1, s = 1;
    for (uint32_t i = 0; i < k; ++i) {
        p.moduli[i] = moduli[i];
        P *= moduli[i];
    }
    for (uint32_t i = 0; i < t; ++i) {
        p.scale_idx[i] = S[i];
        s *= moduli[S[i]];
    }
    uint64_t n = (uint64_t)P < most ? (uint64_t)P : most;
    p.n = n;
    uint64_t lw = 0, tw = 0;
    uint32_t G = 0, ow = 0;
    if (orc_sizes(&p, n, &lw, &tw, &G, &ow)) {
        printf("FAIL sizes\n");
        ++failures;
        return;
    }
    uint32_t *offs = calloc(ow, 4), *zin = calloc(lw, 4), *zout = calloc(lw, 4), *tab = calloc(tw, 4);
    uint32_t *X = calloc(lw, 4), *Y = calloc(lw, 4), *zin2 = calloc(lw, 4), *zout2 = calloc(lw, 4);
    int64_t *x = calloc(n, 8), *y = calloc(n, 8);
    uint8_t *bad = calloc(n, 1);
    const int64_t lo = -(P / 2);
    for (uint64_t a = 0; a < n; ++a) x[a] = lo + (int64_t)((a * (uint64_t)(P - 1)) / (n > 1 ? n - 1 : 1));
    int rc = orc_garble(&p, a0, n, offs, zin, zout, tab);
    rc |= orc_garble(&p, a0, n, offs, zin2, zout2, NULL); /* the zero-label path */
    rc |= orc_encode(&p, n, x, zin, offs, X);
    rc |= orc_eval(&p, a0, n, X, tab, Y);
    rc |= orc_decode(&p, n, Y, zout, offs, y, bad);
    if (rc) {
        printf("FAIL rc\n");
        ++failures;
    }
    if (memcmp(zout, zout2, lw * 4) || memcmp(zin, zin2, lw * 4)) {
        printf("FAIL zero-label path differs\n");
        ++failures;
    }
    const int64_t r = (P / 2) % s;
    for (uint64_t a = 0; a < n; ++a) {
        if (bad[a] || y[a] != floor_div(x[a] + r, s)) {
            if (failures++ < 10) printf("FAIL base P=%lld s=%lld x=%lld y=%lld bad=%d\n", (long long)P, (long long)s,
                                        (long long)x[a], (long long)y[a], bad[a]);
        }
    }
    /* one full trace */
    uint32_t *slots = calloc((size_t)(G + 1) * k * MAXLAMBDA, 4), *slots2 = calloc((size_t)(G + 1) * k * MAXLAMBDA, 4);
    uint32_t *gi = calloc((size_t)G * MAXLAMBDA, 4), *ei = calloc((size_t)G * MAXLAMBDA, 4);
    uint32_t *go = calloc((size_t)G * MAXLAMBDA, 4), *eo = calloc((size_t)G * MAXLAMBDA, 4);
    uint32_t *ro = calloc((size_t)k * MAXLAMBDA, 4), *gr = calloc((size_t)k * MAXLAMBDA, 4);
    uint32_t *er = calloc((size_t)k * MAXLAMBDA, 4), *gf = calloc((size_t)k * MAXLAMBDA, 4);
    uint32_t *ef = calloc((size_t)k * MAXLAMBDA, 4);
    if (orc_trace(&p, a0 + 1, x[n / 2], ro, slots, slots2, gi, ei, go, eo, gr, er, gf, ef)) {
        printf("FAIL trace\n");
        ++failures;
    }
    free(slots), free(slots2), free(gi), free(ei), free(go), free(eo), free(ro), free(gr), free(er), free(gf), free(ef);
    free(offs), free(zin), free(zout), free(tab), free(X), free(Y), free(zin2), free(zout2), free(x), free(y), free(bad);
}

int main(void) {
    static const uint32_t b1[] = {2, 3, 5, 7, 11}, s1[] = {4};
    static const uint32_t b2[] = {2, 3, 5, 7}, s2[] = {2, 3};
    static const uint32_t b3[] = {3, 5, 7, 11, 13}, s3[] = {0, 4};
    static const uint32_t b4[] = {3, 4, 5}, s4[] = {1};
    static const uint32_t b5[] = {32, 167, 173}, s5[] = {0};
    static const uint32_t b6[] = {2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37}, s6[] = {11};
    static const uint32_t b7[] = {3, 197, 241}, s7[] = {1};
    run_base(b1, 5, s1, 1, 0, 0, 400);
    run_base(b1, 5, s1, 1, (1ull << 31) + 5, 1ull << 40, 64);
    run_base(b2, 4, s2, 2, 3, 6, 210);
    run_base(b3, 5, s3, 2, 0, 50, 200);
    run_base(b4, 3, s4, 1, 0, 51, 60);
    run_base(b5, 3, s5, 1, 7, 42, 100);
    run_base(b6, 12, s6, 1, 1000, 3, 8);
    run_base(b7, 3, s7, 1, 0, 9, 60);
    uint32_t A[MAXLAMBDA] = {0}, xx[4], u[4], V[8], out[MAXLAMBDA];
    for (int i = 0; i < 128; ++i) A[i] = (uint32_t)(i * 7 + 1) % 251;
    orc_hash_parts(251, 2, A, 0xffffffffu, ~0ull, xx, u, V);
    orc_hash_parts(251, 251, A, 0, 1ull << 63, xx, u, V);
    orc_prg_label(~0ull, 2, ~0ull, 251, 0, out);
    orc_prg_label(0, 1, 0, 128, 1, out);
    printf("oracle check: %d failures\n", failures);
    return failures ? 1 : 0;
}
