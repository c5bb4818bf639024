// Host-side plan: validation, label sizes, gate list, per-modulus constants.
#include "plan.hpp"

#include <string.h>

namespace redash {

namespace {

bool is_prime(uint32_t v) {
    if (v < 2) return false;
    for (uint32_t d = 2; d * d <= v; ++d)
        if (v % d == 0) return false;
    return true;
}

uint32_t bit_length(uint32_t v) {
    uint32_t b = 0;
    while (v) {
        ++b;
        v >>= 1;
    }
    return b;
}

uint32_t ipow(uint32_t m, uint32_t e) {
    uint64_t r = 1;
    for (uint32_t i = 0; i < e; ++i) r *= m;
    return static_cast<uint32_t>(r);
}

uint64_t ipow64(uint32_t m, uint32_t e) {
    uint64_t r = 1;
    for (uint32_t i = 0; i < e; ++i) r *= m;
    return r;
}

bool is_pow2(uint32_t v) { return v >= 2 && (v & (v - 1)) == 0; }

uint32_t gcd(uint32_t a, uint32_t b) {
    while (b) {
        const uint32_t r = a % b;
        a = b;
        b = r;
    }
    return a;
}

}  // namespace

bool modulus_ok(uint32_t m) { return m >= 2 && m <= 255 && (is_prime(m) || is_pow2(m)); }

void division_constants(uint32_t m, uint64_t x_bound, uint32_t *outM, uint32_t *outS, uint32_t *outFix) {
    if ((m & (m - 1)) == 0) {  // a power of two (m >= 2): umulhi(x, 2^(32-e)) = x >> e
        const uint32_t e = bit_length(m) - 1;
        *outM = 1u << (32 - e);
        *outS = 0;
        *outFix = 0;
        return;
    }
    // Round-up magic: s = floor(log2 m), M = ceil(2^(32+s) / m) < 2^32 for m
    // not a power of two.  The error of x M / 2^(32+s) over x / m is
    // x (m M - 2^(32+s)) / (m 2^(32+s)); it keeps the floor exact whenever it
    // stays below 1/m, i.e. x (m M - 2^(32+s)) < 2^(32+s).
    uint32_t s = bit_length(m) - 1;
    unsigned __int128 two = static_cast<unsigned __int128>(1) << (32 + s);
    unsigned __int128 M = (two + m - 1) / m;
    unsigned __int128 err = M * m - two;
    if (M < (static_cast<unsigned __int128>(1) << 32) &&
        static_cast<unsigned __int128>(x_bound - 1) * err < two) {
        *outM = static_cast<uint32_t>(M);
        *outS = s;
        *outFix = 0;
        return;
    }
    // General 32-bit case: l = ceil(log2 m), M' = floor(2^32 (2^l - m) / m) + 1,
    // q = (t + ((x - t) >> 1)) >> (l - 1) with t = umulhi(x, M').
    uint32_t l = bit_length(m - 1);
    unsigned __int128 Mp = ((static_cast<unsigned __int128>(1) << 32) *
                            ((static_cast<unsigned __int128>(1) << l) - m)) / m + 1;
    *outM = static_cast<uint32_t>(Mp);
    *outS = l - 1;
    *outFix = 1;
}

bool mul24_constants(uint32_t m, uint64_t x_bound, uint32_t *outM, uint32_t *outS) {
    if (x_bound > (1u << 24)) return false;
    for (uint32_t s = 31; s >= 1; --s) {
        const uint64_t two = 1ull << s;
        const uint64_t M = (two + m - 1) / m;
        if (M >= (1u << 24)) continue;
        if ((x_bound - 1) * M >= (1ull << 32)) continue;
        const uint64_t err = M * m - two;  // < m
        if ((x_bound - 1) * err < two) {
            *outM = static_cast<uint32_t>(M);
            *outS = s;
            return true;
        }
    }
    return false;
}

uint32_t inverse_mod(uint32_t a, uint32_t m) {
    a %= m;
    for (uint32_t x = 1; x < m; ++x)
        if ((a * x) % m == 1) return x;
    return 0;
}

uint32_t label_lambda(uint32_t m) {
    // least lambda with m^lambda >= 2^128, by exact integer comparison
    const unsigned __int128 limit = ~static_cast<unsigned __int128>(0);  // 2^128 - 1
    unsigned __int128 p = 1;
    uint32_t lam = 0;
    while (p <= limit / m) {  // p * m <= 2^128 - 1, i.e. still below 2^128
        p *= m;
        ++lam;
    }
    return lam + 1;  // the next power reaches at least 2^128
}

uint32_t label_words(uint32_t m) {
    uint32_t g = 32u / bit_length(m - 1);
    return (label_lambda(m) + g - 1) / g;
}

void fill_mod_const(uint32_t m, ModConst *mc) {
    memset(mc, 0, sizeof *mc);
    mc->m = m;
    mc->lam = label_lambda(m);
    mc->b = bit_length(m - 1);
    mc->g = 32u / mc->b;
    mc->W = (mc->lam + mc->g - 1) / mc->g;
    mc->glast = mc->lam - (mc->W - 1) * mc->g;
    mc->mask = (mc->b == 32) ? 0xffffffffu : ((1u << mc->b) - 1u);
    // Units of Z_m: every nonzero residue for a prime, the odd ones for 2^l.
    const bool pow2 = is_pow2(m) && m > 2;
    mc->phi = pow2 ? m / 2 : m - 1;
    mc->r0 = pow2 ? m / 2 : m - 1;
    // m^g reaches 2^32 only for m = 4 and m = 16 (b g = 32); it is stored
    // as 0, and those moduli take the generic paths (fast stays 0).
    const uint64_t pw_g64 = ipow64(m, mc->g), pw_last64 = ipow64(m, mc->glast);
    const bool full_word = pw_g64 >= (1ull << 32) || pw_last64 >= (1ull << 32);
    if (m > 2) {
        mc->pw_g = static_cast<uint32_t>(pw_g64);
        mc->pw_last = static_cast<uint32_t>(pw_last64);
    }
    uint64_t bound = (m > 2 && !full_word) ? pw_g64 : (1ull << 32);
    // Products c * d of two residues (< m^2) are reduced with the same
    // constants, so the bound covers them as well.
    uint64_t sq = static_cast<uint64_t>(m) * m;
    if (sq > bound) bound = sq;
    division_constants(m, bound, &mc->divM, &mc->divS, &mc->div_fix);

    if (m == 2) return;  // labels over Z_2 are bit vectors; no fast path needed
    for (uint32_t f = 0; f < mc->g; f += 2) {
        mc->sw_even |= mc->mask << (mc->b * f);
        mc->sw_ones |= 1u << (mc->b * f);
        mc->sw_k |= ((1u << mc->b) - m) << (mc->b * f);
    }
    mc->two_m = 2 * m;
    if (full_word) return;  // no fast constants: the packed-add fields above are all it uses
    mc->red_M = static_cast<uint32_t>(((1ull << 32) + m - 1) / m);
    bool ok = 3 * sq * m < (1ull << 32);  // x m < 2^32 for x < 3 m^2 (every m <= 255)
    uint64_t part = 1;
    for (int k = 0; k < 2; ++k) {
        const uint32_t nres = k ? mc->glast : mc->g;
        const uint32_t nlo = nres / 2, nhi = nres - nlo;
        uint32_t M = 0, sh = 0, fix = 0;
        if (nlo) division_constants(ipow(m, nlo), static_cast<uint64_t>(ipow(m, nres)), &M, &sh, &fix);
        ok = ok && fix == 0;  // the fast path has no fix-up step
        if (k) {
            mc->nlo_l = nlo;
            mc->pw_lo_l = ipow(m, nlo);
            mc->lo_M_l = M;
            mc->lo_s_l = sh;
        } else {
            mc->nlo_f = nlo;
            mc->pw_lo_f = ipow(m, nlo);
            mc->lo_M_f = M;
            mc->lo_s_f = sh;
        }
        const uint64_t hi = ipow(m, nhi), lo = ipow(m, nlo);
        if (hi > part) part = hi;
        if (lo > part) part = lo;
    }
    // (the split's parts also feed signed 24-bit multiply-adds: below 2^23)
    ok = ok && mul24_constants(m, part, &mc->sd_M, &mc->sd_s) && part < (1u << 23);
    mc->fast = ok ? 1u : 0u;
    // fraction-multiplication digits: exact while (m^n)^2 < 2^32
    mc->fd = (static_cast<uint64_t>(part) * part < (1ull << 32)) ? 1u : 0u;
    auto frac_mult = [](uint64_t M) { return M > 1 ? static_cast<uint32_t>((1ull << 32) / M + 1) : 0u; };
    for (int k = 0; k < 2; ++k) {
        const uint32_t nres = k ? mc->glast : mc->g;
        const uint32_t nlo = nres / 2, nhi = nres - nlo;
        const uint32_t chi = frac_mult(ipow(m, nhi)), clo = frac_mult(ipow(m, nlo));
        if (k) {
            mc->fc_hi_l = chi;
            mc->fc_lo_l = clo;
        } else {
            mc->fc_hi_f = chi;
            mc->fc_lo_f = clo;
        }
    }
}

int build_plan(const redash_params *p, Plan *pl) {
    if (!p || !pl) return REDASH_E_NULL;
    memset(pl, 0, sizeof *pl);
    if (p->k < 2 || p->k > static_cast<uint32_t>(kMaxK)) return REDASH_E_PARAM;
    if (p->t < 1 || p->t > p->k - 1) return REDASH_E_PARAM;
    unsigned __int128 P = 1;
    for (uint32_t i = 0; i < p->k; ++i) {
        uint32_t m = p->moduli[i];
        // primes or powers of two (Sec. 4 uses one 2^l modulus), ascending,
        // pairwise coprime (so at most one of them is even)
        if (!modulus_ok(m)) return REDASH_E_PARAM;
        if (i > 0 && m <= p->moduli[i - 1]) return REDASH_E_PARAM;
        for (uint32_t j = 0; j < i; ++j)
            if (gcd(m, p->moduli[j]) != 1) return REDASH_E_PARAM;
        P *= m;
    }
    if (P >= (static_cast<unsigned __int128>(1) << 63)) return REDASH_E_PARAM;
    uint64_t s = 1;
    uint32_t is_scale = 0;
    for (uint32_t a = 0; a < p->t; ++a) {
        uint32_t si = p->scale_idx[a];
        if (si >= p->k) return REDASH_E_PARAM;
        if (a > 0 && si <= p->scale_idx[a - 1]) return REDASH_E_PARAM;
        is_scale |= 1u << si;
        s *= p->moduli[si];
        pl->S[a] = si;
    }
    const uint64_t P64 = static_cast<uint64_t>(P);
    // Shift constants (Sec. 3.4): up by U = floor(P/2), down by floor(U/s).
    // Where P/(2s) is an integer these are P/2 and P/(2s) and the gadget
    // returns floor(x/s); otherwise (odd P, or a scaled power of two) it
    // returns floor((x + (U mod s)) / s).
    const uint64_t U = P64 / 2, down = U / s;

    pl->k = p->k;
    pl->t = p->t;
    pl->u = p->k - p->t;
    pl->n = p->n;
    pl->a0 = p->a0;
    pl->seed = p->seed;
    pl->gid = static_cast<uint32_t>(p->seed);
    pl->P = P64;
    pl->s = s;
    pl->is_scale_mask = is_scale;
    uint32_t u = 0, woff = 0;
    for (uint32_t i = 0; i < p->k; ++i) {
        if (!(is_scale & (1u << i))) pl->R[u++] = i;
        ModConst &mc = pl->mod[i];
        fill_mod_const(p->moduli[i], &mc);
        mc.woff = woff;
        woff += mc.W;
        mc.up = static_cast<uint32_t>(U % mc.m);
        mc.down = static_cast<uint32_t>(down % mc.m);
    }
    pl->total_words = woff;

    auto pack = [](uint32_t src, uint32_t dst, uint32_t kind, uint32_t phase, uint32_t coeff) {
        return src | (dst << 4) | (kind << 8) | (phase << 9) | (coeff << 16);
    };
    uint32_t G = 0;
    // Phase A (Sec. 3.2, once per scaling modulus): digit S[a] onto the later
    // scaling moduli, then onto every remaining modulus; L <- q^{-1}(L - E).
    for (uint32_t a = 0; a < pl->t; ++a) {
        uint32_t src = pl->S[a], q = p->moduli[src];
        for (uint32_t b = a + 1; b < pl->t; ++b) {
            uint32_t dst = pl->S[b];
            pl->gate[G++] = pack(src, dst, 0, 0, inverse_mod(q, p->moduli[dst]));
        }
        for (uint32_t b = 0; b < pl->u; ++b) {
            uint32_t dst = pl->R[b];
            pl->gate[G++] = pack(src, dst, 0, 0, inverse_mod(q, p->moduli[dst]));
        }
    }
    // Phase B (Sec. 3.3): mixed-radix conversion over R.  Digit R[b] onto the
    // later remaining moduli (the recursion of Eq. rns_to_mrs), then onto
    // every scaling modulus with its mixed-radix weight prod_{b'<b} R[b'].
    for (uint32_t b = 0; b < pl->u; ++b) {
        uint32_t src = pl->R[b], q = p->moduli[src];
        for (uint32_t c = b + 1; c < pl->u; ++c) {
            uint32_t dst = pl->R[c];
            pl->gate[G++] = pack(src, dst, 0, 1, inverse_mod(q, p->moduli[dst]));
        }
        for (uint32_t a = 0; a < pl->t; ++a) {
            uint32_t dst = pl->S[a], md = p->moduli[dst];
            uint32_t w = 1 % md;
            for (uint32_t c = 0; c < b; ++c) w = (w * (p->moduli[pl->R[c]] % md)) % md;
            pl->gate[G++] = pack(src, dst, 1, 1, w);
        }
    }
    pl->G = G;
    // Where every label lives while the evaluator walks the gates.  Phase A
    // reads the inputs and leaves its results in the output tensor (final
    // for R).  Phase B works on copies of the R labels: R[0] is only ever a
    // digit and is read in place, R[1..u-1] move to the working storage on
    // their first update; the S slots restart as zero accumulators.
    uint32_t wk = 0;
    for (uint32_t b = 1; b < pl->u; ++b) {
        pl->mod[pl->R[b]].wkoff = wk;
        wk += pl->mod[pl->R[b]].W;
    }
    pl->work_words = wk;
    uint32_t loc[kMaxK];
    for (uint32_t i = 0; i < pl->k; ++i) loc[i] = kLocIn;
    bool phase_b = false;
    for (uint32_t g = 0; g < G; ++g) {
        uint32_t &d = pl->gate[g];
        if (gate_phase(d) && !phase_b) {
            phase_b = true;
            for (uint32_t a = 0; a < pl->t; ++a) loc[pl->S[a]] = kLocZero;
        }
        const uint32_t src = gate_src(d), dst = gate_dst(d);
        const bool to_work = phase_b && !(is_scale & (1u << dst));
        d |= (loc[dst] << 10) | ((to_work ? 1u : 0u) << 12) | (loc[src] << 13);
        loc[dst] = to_work ? kLocWork : kLocOut;
        const ModConst &md = pl->mod[dst];
        if (g < kMaxTables && md.m > 2 && md.m <= kTableMaxModulus && md.fast) d |= 1u << 15;
    }
    pl->ntab = G < kMaxTables ? G : kMaxTables;
    return REDASH_OK;
}

namespace {

// One gate of a target's list: the digit it hashes and the gate index.
// Digits are numbered: Phase-A digit of S[a] is a, Phase-B digit of R[b] is
// kMaxK + b.
struct TGate {
    uint32_t digit, g;
};

struct Target {
    uint32_t mod;       // modulus index
    uint32_t from_in;   // starts from the input label (else from zero)
    uint32_t kind;      // 0: S[a] of Phase A, 1: R[j], 2: accumulator of S[a]
    uint32_t digit;     // the digit this target becomes (kind 0 and 1), else ~0u
    uint32_t nA;        // its first nA gates are Phase-A gates
    uint32_t n;
    TGate gate[kMaxK + kMaxK];
};

}  // namespace

void build_eval_plan(const Plan &P, EvalPlan *E) {
    memset(E, 0, sizeof *E);
    E->k = P.k;
    E->t = P.t;
    E->u = P.u;
    E->G = P.G;
    E->total_words = P.total_words;
    E->work_words = P.work_words;
    E->ntab = P.ntab;
    E->gid = P.gid;
    E->n = P.n;
    E->a0 = P.a0;
    for (uint32_t i = 0; i < P.k; ++i) E->mod[i] = P.mod[i];
    // gate lookup by (phase, digit modulus, destination modulus)
    uint32_t gidx[2][kMaxK][kMaxK];
    uint32_t toff = 0;
    for (uint32_t g = 0; g < P.G; ++g) {
        const uint32_t d = P.gate[g];
        gidx[gate_phase(d)][gate_src(d)][gate_dst(d)] = g;
        E->egate[g] = gate_dst(d) | (gate_kind(d) << 4) | (gate_tab(d) << 5) | (gate_coeff(d) << 6) | (toff << 14);
        toff += (P.mod[gate_src(d)].m - 1) * P.mod[gate_dst(d)].W;
    }
    // the targets in the order they are finished
    Target T[3 * kMaxK];
    uint32_t nt = 0;
    for (uint32_t a = 1; a < P.t; ++a) {
        Target &x = T[nt++];
        x = Target{P.S[a], 1, 0, a, 0, 0, {}};
        for (uint32_t b = 0; b < a; ++b) x.gate[x.n++] = TGate{b, gidx[0][P.S[b]][P.S[a]]};
        x.nA = x.n;
    }
    for (uint32_t j = 0; j < P.u; ++j) {
        Target &x = T[nt++];
        x = Target{P.R[j], 1, 1, kMaxK + j, 0, 0, {}};
        for (uint32_t a = 0; a < P.t; ++a) x.gate[x.n++] = TGate{a, gidx[0][P.S[a]][P.R[j]]};
        x.nA = x.n;
        for (uint32_t b = 0; b < j; ++b) x.gate[x.n++] = TGate{kMaxK + b, gidx[1][P.R[b]][P.R[j]]};
    }
    for (uint32_t a = 0; a < P.t; ++a) {
        Target &x = T[nt++];
        x = Target{P.S[a], 0, 2, ~0u, 0, 0, {}};
        for (uint32_t b = 0; b < P.u; ++b) x.gate[x.n++] = TGate{kMaxK + b, gidx[1][P.R[b]][P.S[a]]};
    }
    // blocks: pairs of consecutive targets; with an odd count the first
    // target (the one with the fewest gates) is alone
    uint32_t first[kMaxBlocks], second[kMaxBlocks], nb = 0;
    for (uint32_t next = 0; next < nt;) {
        const bool alone = (next == 0 && nt % 2);
        first[nb] = next;
        second[nb++] = alone ? ~0u : next + 1;
        next += alone ? 1 : 2;
    }
    uint32_t block_of[3 * kMaxK];
    for (uint32_t b = 0; b < nb; ++b) {
        block_of[first[b]] = b;
        if (second[b] != ~0u) block_of[second[b]] = b;
    }
    // where a digit is read from (outside its own block), and whether a
    // target must be stored for readers in later blocks
    auto digit_loc = [&](uint32_t digit) -> uint32_t {
        if (digit < kMaxK) return digit == 0 ? kDigIn : kDigOut;
        return digit == kMaxK ? kDigOut : kDigWork;
    };
    auto digit_mod = [&](uint32_t digit) -> uint32_t { return digit < kMaxK ? P.S[digit] : P.R[digit - kMaxK]; };
    auto read_elsewhere = [&](uint32_t ti) {
        const uint32_t digit = T[ti].digit;
        if (digit == ~0u) return false;
        for (uint32_t o = 0; o < nt; ++o)
            for (uint32_t i = 0; i < T[o].n; ++i)
                if (T[o].gate[i].digit == digit && block_of[o] != block_of[ti]) return true;
        return false;
    };
    // stores after gate i (0-based) of target ti: bit 0 output, bit 1 working
    auto stores_after = [&](uint32_t ti, uint32_t i) -> uint32_t {
        const Target &x = T[ti];
        uint32_t f = 0;
        if (x.kind == 1) {
            if (i + 1 == x.nA) f |= 1u;  // the Phase-A value is the output label of R[j]
            // R[0]'s digit is read from the output tensor; R[j], j >= 1, from the working storage
            if (i + 1 == x.n && x.digit != kMaxK && read_elsewhere(ti)) f |= 2u;
        } else if (i + 1 == x.n) {
            if (x.kind == 2 || read_elsewhere(ti)) f |= 1u;
        }
        return f;
    };
    uint32_t ns = 0;
    for (uint32_t b = 0; b < nb; ++b) {
        const Target &X = T[first[b]];
        const bool two = second[b] != ~0u;
        const Target &Y = two ? T[second[b]] : X;
        const uint32_t s0 = ns;
        uint32_t i = 0, j = 0;
        auto later_in_y = [&](uint32_t digit, uint32_t from) {
            if (!two) return false;
            for (uint32_t q = from; q < Y.n; ++q)
                if (Y.gate[q].digit == digit) return true;
            return false;
        };
        while (i < X.n || (two && j < Y.n)) {
            uint32_t st = 0;
            if (two && i < X.n && j < Y.n && X.gate[i].digit == Y.gate[j].digit) {
                // one digit for both slots: two consecutive gates of its run
                const uint32_t digit = X.gate[i].digit;
                st = X.gate[i].g | (1u << 8) | (digit_loc(digit) << 10) | (digit_mod(digit) << 12);
                st |= stores_after(first[b], i) << 16;
                st |= stores_after(second[b], j) << 18;
                ++i;
                ++j;
            } else if (i < X.n && !later_in_y(X.gate[i].digit, j)) {
                const uint32_t digit = X.gate[i].digit;
                st = X.gate[i].g | (digit_loc(digit) << 10) | (digit_mod(digit) << 12);
                st |= stores_after(first[b], i) << 16;
                ++i;
            } else {
                // slot 1 alone; its digit is read from slot 0 once slot 0 is final
                const uint32_t digit = Y.gate[j].digit;
                const uint32_t loc = (digit == X.digit && i == X.n) ? kDigSlot0 : digit_loc(digit);
                st = Y.gate[j].g | (1u << 9) | (loc << 10) | (digit_mod(digit) << 12);
                st |= stores_after(second[b], j) << 18;
                ++j;
            }
            E->step[ns++] = st;
        }
        uint32_t bd = X.mod | (X.from_in << 4) | ((ns - s0) << 24) | (s0 << 16);
        if (two) bd |= (1u << 5) | (Y.mod << 6) | (Y.from_in << 10);
        E->block[b] = bd;
    }
    E->nblocks = nb;
    E->nsteps = ns;
}

}  // namespace redash
