// Host check of the per-modulus constants that the plan hands to the kernels:
// every multiply-shift division, digit split and fraction-digit multiplier is
// checked against plain integer division over the whole operand range it is
// used on, for every modulus the library accepts.  tests/test_plan_constants.py
// builds this file with g++ and the address and undefined-behaviour
// sanitizers (together with plan.cpp) and runs it.
//
// For a multiplier that rounds 1/d up (every constant here except the
// fix-up form), x = q d + r gives floor(x M / 2^k) = q + floor((r + x e / 2^k) / d)
// with e = M d - 2^k > 0: for a fixed q the error term grows with r, so the
// first wrong quotient below a bound X is at some x = q d + d - 1 or at
// x = X - 1.  Bounds above 2^22 are checked on exactly those points; smaller
// ones on every x.  (For a power of two the multiplier is exact by
// construction, umulhi(x, 2^(32-e)) = x >> e; it is checked on a sample.)
#include <stdint.h>
#include <stdio.h>

#include "../paper_2506_14489_amd/csrc/plan.hpp"

using namespace redash;

static long fails = 0, checked = 0;

#define CHECK(cond, ...)                                        \
    do {                                                        \
        ++checked;                                              \
        if (!(cond)) {                                          \
            if (fails++ < 20) {                                 \
                printf("FAIL line %d: ", __LINE__);             \
                printf(__VA_ARGS__);                            \
                printf("\n");                                   \
            }                                                   \
        }                                                       \
    } while (0)

static uint32_t umulhi(uint32_t a, uint32_t b) { return static_cast<uint32_t>((static_cast<uint64_t>(a) * b) >> 32); }

// Calls f(x) on every x < bound, or on the points named above.
template <typename F>
static void for_points(uint64_t bound, uint64_t d, F f) {
    if (bound <= (1ull << 22)) {
        for (uint64_t x = 0; x < bound; ++x) f(static_cast<uint32_t>(x));
        return;
    }
    for (uint64_t x = d - 1; x < bound; x += d) f(static_cast<uint32_t>(x));
    for (uint64_t x = 0; x < 4 * d; ++x) f(static_cast<uint32_t>(x));
    f(static_cast<uint32_t>(bound - 1));
}

static uint64_t ipow(uint64_t m, uint32_t e) {
    uint64_t r = 1;
    for (uint32_t i = 0; i < e; ++i) r *= m;
    return r;
}

static void check_modulus(uint32_t m) {
    ModConst mc;
    fill_mod_const(m, &mc);
    // label length: least lambda with m^lambda >= 2^128
    {
        const unsigned __int128 max = ~static_cast<unsigned __int128>(0);  // 2^128 - 1
        unsigned __int128 p = 1;
        bool fits = true;
        for (uint32_t i = 0; i + 1 < mc.lam; ++i) {
            fits = fits && p <= max / m;
            p *= m;
        }
        CHECK(fits, "m=%u lam=%u: m^(lam-1) below 2^128", m, mc.lam);
        // m^lam >= 2^128  <=>  m^(lam-1) > (2^128 - 1) / m
        CHECK(p > max / m, "m=%u lam=%u minimal", m, mc.lam);
    }
    CHECK(mc.b == 32u - static_cast<uint32_t>(__builtin_clz(m - 1)), "m=%u b", m);
    CHECK(mc.g == 32 / mc.b && mc.W == (mc.lam + mc.g - 1) / mc.g && mc.glast == mc.lam - (mc.W - 1) * mc.g,
          "m=%u word shape", m);
    if (m > 2) {
        const uint64_t pg = ipow(m, mc.g), pl = ipow(m, mc.glast);
        CHECK(mc.pw_g == (pg >= (1ull << 32) ? 0u : pg), "m=%u pw_g", m);
        CHECK(mc.pw_last == (pl >= (1ull << 32) ? 0u : pl), "m=%u pw_last", m);
    }
    // the general division: every x below m^g (2^32 when m^g reaches it, or
    // m = 2) and below m^2
    {
        const bool full = m == 2 || ipow(m, mc.g) >= (1ull << 32) || ipow(m, mc.glast) >= (1ull << 32);
        uint64_t bound = full ? (1ull << 32) : ipow(m, mc.g);
        if (static_cast<uint64_t>(m) * m > bound) bound = static_cast<uint64_t>(m) * m;
        if ((m & (m - 1)) == 0) {
            for (uint64_t x = 0; x < bound; x += 4099) {
                CHECK((umulhi(static_cast<uint32_t>(x), mc.divM) >> mc.divS) == x / m, "m=%u div x=%llu", m,
                      static_cast<unsigned long long>(x));
            }
            CHECK((umulhi(0xffffffffu, mc.divM) >> mc.divS) == 0xffffffffu / m, "m=%u div top", m);
        } else if (mc.div_fix) {
            // the fix-up form is exact on all 32-bit x: spot points and the top
            for (uint64_t x = 0; x < (1ull << 32); x += 65537) {
                const uint32_t t = umulhi(static_cast<uint32_t>(x), mc.divM);
                CHECK(((t + ((static_cast<uint32_t>(x) - t) >> 1)) >> mc.divS) == x / m, "m=%u fix x=%llu", m,
                      static_cast<unsigned long long>(x));
            }
        } else {
            for_points(bound, m, [&](uint32_t x) {
                CHECK((umulhi(x, mc.divM) >> mc.divS) == x / m, "m=%u div x=%u", m, x);
            });
        }
    }
    if (m > 2) {
        for (uint32_t a = 1; a < m; ++a) {
            if ((m & 1) == 0 && (a & 1) == 0) continue;  // units of 2^l are the odd residues
            const uint32_t inv = inverse_mod(a, m);
            CHECK(inv < m && (a * inv) % m == 1, "m=%u inverse of %u", m, a);
        }
    }
    if (!mc.fast) return;
    CHECK(m > 2, "m=%u fast", m);
    // one reduction per residue: floor(x/m) = umulhi(x, ceil(2^32/m)) for x < 3 m^2
    for (uint32_t x = 0; x < 3 * m * m; ++x) CHECK(umulhi(x, mc.red_M) == x / m, "m=%u red x=%u", m, x);
    CHECK(mc.two_m == 2 * m, "m=%u two_m", m);
    // the digit split of a word D < m^nres at m^nlo, for full and last words
    uint64_t part = 1;
    for (int k = 0; k < 2; ++k) {
        const uint32_t nres = k ? mc.glast : mc.g;
        const uint32_t nlo = k ? mc.nlo_l : mc.nlo_f, M = k ? mc.lo_M_l : mc.lo_M_f, s = k ? mc.lo_s_l : mc.lo_s_f;
        const uint32_t pw_lo = k ? mc.pw_lo_l : mc.pw_lo_f;
        CHECK(nlo == nres / 2, "m=%u nlo", m);
        const uint64_t d = ipow(m, nlo);
        CHECK(pw_lo == d, "m=%u pw_lo", m);
        if (nlo) {
            for_points(ipow(m, nres), d, [&](uint32_t x) {
                CHECK((umulhi(x, M) >> s) == x / d, "m=%u split nres=%u x=%u", m, nres, x);
            });
        }
        const uint64_t hi = ipow(m, nres - nlo);
        if (hi > part) part = hi;
        if (d > part) part = d;
    }
    // 24-bit multiply-shift digits on the parts
    CHECK(part < (1u << 23) && mc.sd_M < (1u << 24), "m=%u sd bounds", m);
    for (uint32_t x = 0; x < part; ++x) {
        CHECK(static_cast<uint64_t>(x) * mc.sd_M < (1ull << 32), "m=%u sd product x=%u", m, x);
        CHECK(((x * mc.sd_M) >> mc.sd_s) == x / m, "m=%u sd x=%u", m, x);
    }
    if (!mc.fd) return;
    // digits by fraction multiplication: for x < m^n, F = x C mod 2^32 with
    // C = floor(2^32 / m^n) + 1, each digit umulhi(F, m), F <- F m
    for (int k = 0; k < 2; ++k) {
        const uint32_t nres = k ? mc.glast : mc.g;
        const uint32_t nlo = nres / 2, nhi = nres - nlo;
        const uint32_t ch = k ? mc.fc_hi_l : mc.fc_hi_f, cl = k ? mc.fc_lo_l : mc.fc_lo_f;
        for (int part_i = 0; part_i < 2; ++part_i) {
            const uint32_t n = part_i ? nlo : nhi, C = part_i ? cl : ch;
            if (n == 0) continue;
            const uint64_t lim = ipow(m, n);
            for (uint64_t x = 0; x < lim; ++x) {
                uint32_t F = static_cast<uint32_t>(x) * C;
                uint64_t rest = x, scale = lim;
                bool ok = true;
                for (uint32_t j = 0; j < n; ++j) {
                    scale /= m;
                    const uint32_t want = static_cast<uint32_t>(rest / scale);
                    rest %= scale;
                    ok = ok && umulhi(F, m) == want;
                    F *= m;
                }
                CHECK(ok, "m=%u fraction digits n=%u x=%llu", m, n, static_cast<unsigned long long>(x));
            }
        }
    }
}

int main() {
    int accepted = 0, fast = 0;
    for (uint32_t m = 0; m <= 300; ++m) {
        const bool ok = modulus_ok(m);
        bool prime = m >= 2;
        for (uint32_t d = 2; d * d <= m; ++d)
            if (m % d == 0) prime = false;
        const bool pow2 = m >= 2 && (m & (m - 1)) == 0;
        CHECK(ok == (m >= 2 && m <= 255 && (prime || pow2)), "modulus_ok(%u)", m);
        if (!ok) continue;
        ++accepted;
        ModConst mc;
        fill_mod_const(m, &mc);
        fast += mc.fast ? 1 : 0;
        check_modulus(m);
    }
    printf("accepted %d moduli, %d on the fast path, %ld checks, %ld failures\n", accepted, fast, checked, fails);
    // the generic-path moduli, for the record
    printf("generic:");
    for (uint32_t m = 3; m <= 255; ++m) {
        if (!modulus_ok(m)) continue;
        ModConst mc;
        fill_mod_const(m, &mc);
        if (!mc.fast) printf(" %u", m);
    }
    printf("\n");
    return fails ? 1 : 0;
}
