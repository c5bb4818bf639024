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
#include <string.h>

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

// ---------------------------------------------------------------------------
// The evaluator's target-major schedule (build_eval_plan), run on values
// instead of labels: a label over Z_m is replaced by the residue it carries,
// a projection gate q -> m maps digit value v to v mod m, a sub gate is
// L <- c (L - E), an acc gate Acc <- Acc + c E.  Every label is read from the
// place the schedule names (input, output, working storage or slot 0) and
// stored where it says, into buffers that start poisoned, exactly as the
// kernel does.  For every x the outputs must be floor(x_up / s) mod m_i with
// x_up = (x + floor(P/2)) mod P (the ShiftUp is the garbler's; the value the
// evaluator's labels carry), the Phase-B values the mixed-radix digits, and
// every gate must be used exactly once, pairs on consecutive gates.
// ---------------------------------------------------------------------------
static const uint32_t kPoison = 0xdeadbeefu;

static void check_schedule(const uint32_t *moduli, uint32_t k, const uint32_t *S, uint32_t t, uint64_t seed) {
    redash_params p;
    memset(&p, 0, sizeof p);
    p.k = k;
    p.t = t;
    for (uint32_t i = 0; i < k; ++i) p.moduli[i] = moduli[i];
    for (uint32_t a = 0; a < t; ++a) p.scale_idx[a] = S[a];
    p.n = 1;
    Plan P;
    CHECK(build_plan(&p, &P) == REDASH_OK, "plan k=%u t=%u", k, t);
    static EvalPlan E;
    build_eval_plan(P, &E);
    CHECK(sizeof(EvalPlan) <= 4096, "EvalPlan of %zu bytes exceeds the kernel-argument limit", sizeof(EvalPlan));
    // every gate exactly once
    uint32_t used[kMaxGates] = {};
    for (uint32_t st = 0; st < E.nsteps; ++st) {
        const uint32_t s0 = E.step[st];
        used[st_gate(s0)]++;
        if (st_two(s0)) used[st_gate(s0) + 1]++;
    }
    for (uint32_t g = 0; g < P.G; ++g) CHECK(used[g] == 1, "k=%u t=%u gate %u used %u times", k, t, g, used[g]);
    CHECK(E.nblocks <= static_cast<uint32_t>(kMaxBlocks), "blocks %u", E.nblocks);
    // table offsets: running sum of (q-1) W_dst
    uint32_t toff = 0;
    for (uint32_t g = 0; g < P.G; ++g) {
        CHECK(eg_toff(E.egate[g]) == toff, "toff gate %u", g);
        CHECK(eg_dst(E.egate[g]) == gate_dst(P.gate[g]) && eg_kind(E.egate[g]) == gate_kind(P.gate[g]) &&
                  eg_coeff(E.egate[g]) == gate_coeff(P.gate[g]) && eg_tab(E.egate[g]) == gate_tab(P.gate[g]),
              "egate %u", g);
        toff += (P.mod[gate_src(P.gate[g])].m - 1) * P.mod[gate_dst(P.gate[g])].W;
    }
    uint64_t Pv = 1, sv = 1;
    for (uint32_t i = 0; i < k; ++i) Pv *= moduli[i];
    for (uint32_t a = 0; a < t; ++a) sv *= moduli[S[a]];
    uint64_t r = seed * 0x9e3779b97f4a7c15ull + 1;
    for (int trial = 0; trial < 64; ++trial) {
        r ^= r << 13;
        r ^= r >> 7;
        r ^= r << 17;
        const uint64_t x = (trial == 0) ? 0 : (trial == 1) ? Pv - 1 : r % Pv;  // x_up in [0, P)
        const uint64_t y = x / sv;
        uint32_t in[kMaxK], out[kMaxK], work[kMaxK];
        for (uint32_t i = 0; i < k; ++i) {
            in[i] = static_cast<uint32_t>(x % moduli[i]);
            out[i] = kPoison;
            work[i] = kPoison;
        }
        for (uint32_t b = 0; b < E.nblocks; ++b) {
            const uint32_t bd = E.block[b];
            uint32_t slot[2] = {bk_in0(bd) ? in[bk_mod0(bd)] : 0u, 0u};
            uint32_t smod[2] = {bk_mod0(bd), bk_two(bd) ? bk_mod1(bd) : 99u};
            if (bk_two(bd)) slot[1] = bk_in1(bd) ? in[bk_mod1(bd)] : 0u;
            for (uint32_t st = bk_first(bd); st < bk_first(bd) + bk_steps(bd); ++st) {
                const uint32_t sd = E.step[st];
                const uint32_t dm = st_dmod(sd);
                uint32_t v = kPoison;
                switch (st_dloc(sd)) {
                    case kDigIn: v = in[dm]; break;
                    case kDigOut: v = out[dm]; break;
                    case kDigWork: v = work[dm]; break;
                    default: v = (smod[0] == dm) ? slot[0] : kPoison; break;
                }
                CHECK(v < moduli[dm], "k=%u t=%u step %u reads an unset digit label (loc %u)", k, t, st, st_dloc(sd));
                if (v >= moduli[dm]) return;
                const uint32_t ng = st_two(sd) ? 2 : 1;
                for (uint32_t j = 0; j < ng; ++j) {
                    const uint32_t g = st_gate(sd) + j;
                    const uint32_t sl = st_two(sd) ? j : st_slot1(sd);
                    const uint32_t e = E.egate[g];
                    CHECK(gate_src(P.gate[g]) == dm, "step %u gate %u digit modulus", st, g);
                    CHECK(eg_dst(e) == smod[sl], "step %u gate %u goes to slot %u's modulus", st, g, sl);
                    const uint32_t m = moduli[eg_dst(e)];
                    const uint64_t E1 = v % m, c = eg_coeff(e);
                    slot[sl] = eg_kind(e) ? static_cast<uint32_t>((slot[sl] + c * E1) % m)
                                          : static_cast<uint32_t>((c * ((slot[sl] + m - E1) % m)) % m);
                }
                const uint32_t f = st_store(sd);
                if (f & 1u) out[smod[0]] = slot[0];
                if (f & 2u) work[smod[0]] = slot[0];
                if (f & 4u) out[smod[1]] = slot[1];
                if (f & 8u) work[smod[1]] = slot[1];
            }
        }
        for (uint32_t i = 0; i < k; ++i)
            CHECK(out[i] == y % moduli[i], "k=%u t=%u x_up=%llu modulus %u: %u, floor(x_up/s) mod m = %llu", k, t,
                  static_cast<unsigned long long>(x), moduli[i], out[i],
                  static_cast<unsigned long long>(y % moduli[i]));
    }
}

static void check_schedules() {
    static const uint32_t primes[15] = {2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37, 41, 43, 47};
    long before = checked;
    // the workloads' bases
    {
        const uint32_t S1[] = {4};
        check_schedule(primes, 5, S1, 1, 1);
        const uint32_t S2[] = {7};
        check_schedule(primes, 8, S2, 1, 2);
        const uint32_t S3[] = {8, 9};
        check_schedule(primes, 10, S3, 2, 3);
        const uint32_t S4[] = {11};
        check_schedule(primes, 12, S4, 1, 4);
        const uint32_t S5[] = {10, 11};
        check_schedule(primes, 12, S5, 2, 5);
        const uint32_t S6[] = {9};
        check_schedule(primes, 12, S6, 1, 6);
        const uint32_t f[] = {32, 167, 173}, F[] = {32, 97, 107}, S0[] = {0};
        check_schedule(f, 3, S0, 1, 7);
        check_schedule(F, 3, S0, 1, 8);
        const uint32_t c8[] = {3, 5, 7, 8, 11, 13, 17, 19}, S8[] = {3};
        check_schedule(c8, 8, S8, 1, 9);
    }
    // every scale set of small bases, and random ones of up to 15 primes
    for (uint32_t k = 2; k <= 6; ++k)
        for (uint32_t mask = 1; mask + 1 < (1u << k); ++mask) {
            uint32_t S[16], t = 0;
            for (uint32_t i = 0; i < k; ++i)
                if (mask & (1u << i)) S[t++] = i;
            check_schedule(primes, k, S, t, mask * 31 + k);
        }
    uint64_t r = 12345;
    for (int trial = 0; trial < 400; ++trial) {
        r = r * 6364136223846793005ull + 1442695040888963407ull;
        uint32_t k = 2 + static_cast<uint32_t>((r >> 33) % 14);  // 2..15
        uint64_t P = 1;
        for (uint32_t i = 0; i < k; ++i) P *= primes[i];
        if (P >= (1ull << 63)) k = 14;
        uint32_t S[16], t = 0;
        for (uint32_t i = 0; i < k; ++i)
            if ((r >> (i + 3)) & 1u) S[t++] = i;
        if (t == 0) S[t++] = k - 1;
        if (t == k) --t;
        check_schedule(primes, k, S, t, r);
    }
    printf("schedules: %ld checks\n", checked - before);
}

int main() {
    check_schedules();
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
