// Host-side plan of one scaling-gadget call: parameter validation, label
// sizes, the gate list and every per-modulus constant the kernels need.
// The plan is passed to the kernels by value as their argument block, so it
// holds no pointers and stays well under the kernel-argument limit.
#pragma once

#include <stdint.h>

#include "../../include/redash.h"

namespace redash {

constexpr int kMaxK = REDASH_MAX_K;
// gates = k(k-1)/2 + t(k-t) <= 105 + 56 for k = 15.
constexpr int kMaxGates = 168;

// Per base modulus.
struct ModConst {
    uint32_t m;        // the modulus
    uint32_t lam;      // residues per label: least lambda with m^lambda >= 2^128
    uint32_t b;        // bits per packed residue: bit length of m - 1
    uint32_t g;        // residues per 32-bit word: floor(32 / b)
    uint32_t W;        // words per label: ceil(lam / g)
    uint32_t glast;    // residues in the last word: lam - (W - 1) g
    uint32_t woff;     // word offset of this modulus in a gadget's k labels
    uint32_t mask;     // (1 << b) - 1
    uint32_t pw_g;     // m^g      (digits of one full word per 32-bit multiply);
                       // 0 stands for 2^32 (m = 4 and m = 16, whose fields fill the word)
    uint32_t pw_last;  // m^glast  (0 likewise)
    // floor(x / m) for 32-bit x: if div_fix == 0, umulhi(x, divM) >> divS is
    // exact for every x < m^g (checked when the plan is built); otherwise
    // the round-up method with a fix-up step:
    //   t = umulhi(x, divM); floor(x/m) = (t + ((x - t) >> 1)) >> divS.
    uint32_t divM, divS, div_fix;
    uint32_t up;       // floor(P/2) mod m             (ShiftUp)
    uint32_t down;     // floor(floor(P/2) / s) mod m  (ShiftDown)
    uint32_t phi;      // order of the unit group of Z_m: m - 1 (prime), m / 2 (power of two)
    uint32_t r0;       // radix of the offset's first digit: m - 1 (prime), m / 2 (2^l, l >= 2)
    // Evaluator fast path (fast == 1 when every bound below holds):
    //  * red: floor(x/m) = umulhi(x, red_M), red_M = ceil(2^32 / m), for
    //    every x < 3 m^2: with e = red_M m - 2^32 < m, x red_M / 2^32 =
    //    x/m + x e / (m 2^32), and the floor is exact while x e < 2^32, which
    //    x m < 2^32 guarantees (3 m^3 < 2^32 for every m <= 255) -- one
    //    multiply per residue;
    //  * sd: the same for every x below the larger part of a split word
    //    (parts below 2^23);
    //  * a word's nres digits D (nres = g, or glast for the last word) are
    //    split once as D = hi * m^nlo + lo, nlo = floor(nres/2), using
    //    floor(D / m^nlo) = umulhi(D, lo_M) >> lo_s (exact for every D below
    //    m^nres; the fast path requires it without a fix-up step).  Suffix
    //    _f: full words, _l: the last word.  (Separate fields, not arrays:
    //    a selected array element would be indexed at run time.)
    uint32_t fast;
    uint32_t two_m;  // 2m
    uint32_t red_M, sd_M, sd_s;
    uint32_t nlo_f, pw_lo_f, lo_M_f, lo_s_f;
    uint32_t nlo_l, pw_lo_l, lo_M_l, lo_s_l;
    // Digits by fraction multiplication (fd == 1 when m^(2 nhi) < 2^32 for
    // both word kinds, nhi = nres - nlo the larger part): for x < m^n,
    // F = x * (floor(2^32 / m^n) + 1) mod 2^32, then each digit, most
    // significant first, is umulhi(F, m) and F <- F m mod 2^32.  fc_hi_* and
    // fc_lo_* are those multipliers for the high and low parts of a word.
    uint32_t fd;
    uint32_t fc_hi_f, fc_lo_f, fc_hi_l, fc_lo_l;
    // Word offset of this modulus in the evaluator's working storage (only
    // the remaining moduli R[1..u-1] have one: their Phase-B copies).
    uint32_t wkoff;
    // Packed addition mod m in one word (m > 2): the even fields (0, 2, 4,
    // ...) of x, in place, and the odd fields shifted down by b, each have
    // b free bits above them.  sw_even masks the even fields, sw_ones has
    // bit 0 of each even field, sw_k holds 2^b - m in each even field.
    uint32_t sw_even, sw_ones, sw_k;
};

// Gate descriptor packed in one word:
//   bits 0-3 src modulus index, 4-7 dst modulus index, 8 kind (0 sub, 1 acc),
//   9 phase (0 A, 1 B), 10-11 where the destination label's current value
//   is, 12 where its new value goes, 13-14 where the digit label is, 15 the
//   gate's free operation uses a byte table (see below), 16-23 coefficient.
// The locations are those of the gate-by-gate order (the garbler and the
// split evaluator); the one-gadget-per-lane evaluator uses EvalPlan.
constexpr uint32_t gate_src(uint32_t d) { return d & 15u; }
constexpr uint32_t gate_dst(uint32_t d) { return (d >> 4) & 15u; }
constexpr uint32_t gate_kind(uint32_t d) { return (d >> 8) & 1u; }
constexpr uint32_t gate_phase(uint32_t d) { return (d >> 9) & 1u; }
constexpr uint32_t gate_tsrc(uint32_t d) { return (d >> 10) & 3u; }
constexpr uint32_t gate_tdst(uint32_t d) { return (d >> 12) & 1u; }
constexpr uint32_t gate_dsrc(uint32_t d) { return (d >> 13) & 3u; }
constexpr uint32_t gate_tab(uint32_t d) { return (d >> 15) & 1u; }
constexpr uint32_t gate_coeff(uint32_t d) { return (d >> 16) & 255u; }

// Free-operation tables: gate g < ntab whose output modulus m satisfies
// 2 < m <= kTableMaxModulus (and has the fast constants) gets 128 bytes of
// LDS holding c (v mod m) mod m for v < 3m, c the gate's coefficient.  The
// evaluator then needs no multiply and no reduction per residue.  A table of
// at most 128 bytes spans the 32 LDS banks once: lookups never conflict.
constexpr uint32_t kTableBytes = 128;
constexpr uint32_t kTableMaxModulus = 42;  // 3m <= 128
constexpr uint32_t kMaxTables = 125;       // keeps two evaluator workgroups per CU

// Label locations in the evaluator: the input LabelTensor, the output
// LabelTensor (which also holds intermediate labels until they are final),
// the working storage (Phase-B copies of the remaining moduli, whose Phase-A
// values are outputs), or a fresh accumulator (the all-zero label).
constexpr uint32_t kLocIn = 0, kLocOut = 1, kLocWork = 2, kLocZero = 3;

struct Plan {
    uint32_t k, t, u, G;
    uint32_t total_words;      // sum of W over the base (words per gadget per LabelTensor)
    uint32_t work_words;       // evaluator working words per gadget: sum of W over R[1..u-1]
    uint32_t ntab;             // gates 0..ntab-1 have a free-operation table slot
    uint32_t S[kMaxK];         // scaling modulus indices, ascending
    uint32_t R[kMaxK];         // remaining modulus indices, ascending
    uint32_t is_scale_mask;    // bit i set when modulus i is a scaling modulus
    uint32_t gid;              // gadget_id = seed mod 2^32
    uint64_t n, a0, seed;
    uint64_t P, s;
    ModConst mod[kMaxK];
    uint32_t gate[kMaxGates];
};

// Builds and validates the plan.  Returns REDASH_OK, REDASH_E_NULL or
// REDASH_E_PARAM.
int build_plan(const redash_params *p, Plan *out);

// ---------------------------------------------------------------------------
// Target-major schedule of the one-gadget-per-lane evaluator.
//
// Every label that projection gates update (a "target") is kept in
// registers from its first update to its last, so it is read once and
// written once.  The targets, in the order the evaluator finishes them:
// S[1..t-1] (Phase A: each becomes the digit of its division step),
// R[0..u-1] (Phase A, then the recursion of Phase B: R[j] becomes digit j of
// the mixed-radix conversion), then the accumulators of S[0..t-1] (Phase B).
// A target's gates come in the order the paper applies them (its Phase-A
// digits, then its Phase-B digits), since the division steps do not commute.
// Consecutive targets are paired into blocks of two register slots; a step
// hashes one digit label for the gates of both slots that take it (two
// consecutive gates of the canonical gate list, so the tweaks and tables do
// not change), or for one slot.  The digit label is read from the input
// tensor (S[0]), the output tensor (S[a], a >= 1, and R[0], which are final
// there), the working storage (R[j], j >= 1, stored once when final) or,
// when it is the block's own first target, its registers.
// ---------------------------------------------------------------------------

// Per gate: bits 0-3 dst modulus index, 4 kind (0 sub, 1 acc), 5 the gate's
// free operation uses its byte table, 6-13 coefficient, 14-31 word offset of
// the gate's table block in units of n words (sum of (q-1) W_dst over the
// earlier gates; below 2^18 for every base).
constexpr uint32_t eg_dst(uint32_t e) { return e & 15u; }
constexpr uint32_t eg_kind(uint32_t e) { return (e >> 4) & 1u; }
constexpr uint32_t eg_tab(uint32_t e) { return (e >> 5) & 1u; }
constexpr uint32_t eg_coeff(uint32_t e) { return (e >> 6) & 255u; }
constexpr uint32_t eg_toff(uint32_t e) { return e >> 14; }

// Per step: bits 0-7 the first gate g (the second, if any, is g + 1),
// 8 two gates (slot 0 takes g, slot 1 takes g + 1), 9 the single gate goes
// to slot 1, 10-11 where the digit label is (kDigIn, kDigOut, kDigWork,
// kDigSlot0), 12-15 the digit's modulus index, then what is stored after the
// step: 16 slot 0 to the output tensor, 17 slot 0 to the working storage,
// 18 slot 1 to the output tensor, 19 slot 1 to the working storage.
constexpr uint32_t kDigIn = 0, kDigOut = 1, kDigWork = 2, kDigSlot0 = 3;
constexpr uint32_t st_gate(uint32_t s) { return s & 255u; }
constexpr uint32_t st_two(uint32_t s) { return (s >> 8) & 1u; }
constexpr uint32_t st_slot1(uint32_t s) { return (s >> 9) & 1u; }
constexpr uint32_t st_dloc(uint32_t s) { return (s >> 10) & 3u; }
constexpr uint32_t st_dmod(uint32_t s) { return (s >> 12) & 15u; }
constexpr uint32_t st_store(uint32_t s) { return (s >> 16) & 15u; }  // bit 0 s0 out, 1 s0 work, 2 s1 out, 3 s1 work

// Per block: bits 0-3 slot 0's modulus index, 4 slot 0 starts from the
// input tensor (else from the all-zero label), 5 slot 1 is used, 6-9 slot
// 1's modulus index, 10 slot 1 starts from the input tensor, 16-23 first
// step, 24-31 number of steps.
constexpr uint32_t bk_mod0(uint32_t b) { return b & 15u; }
constexpr uint32_t bk_in0(uint32_t b) { return (b >> 4) & 1u; }
constexpr uint32_t bk_two(uint32_t b) { return (b >> 5) & 1u; }
constexpr uint32_t bk_mod1(uint32_t b) { return (b >> 6) & 15u; }
constexpr uint32_t bk_in1(uint32_t b) { return (b >> 10) & 1u; }
constexpr uint32_t bk_first(uint32_t b) { return (b >> 16) & 255u; }
constexpr uint32_t bk_steps(uint32_t b) { return b >> 24; }
constexpr int kMaxBlocks = 16;  // ceil((k + t - 1) / 2) <= 14

struct EvalPlan {
    uint32_t k, t, u, G;
    uint32_t total_words, work_words;
    uint32_t ntab;             // gates 0..ntab-1 have a free-operation table slot
    uint32_t nblocks, nsteps;
    uint32_t gid;
    uint64_t n, a0;
    ModConst mod[kMaxK];
    uint32_t egate[kMaxGates];
    uint32_t step[kMaxGates];
    uint32_t block[kMaxBlocks];
};

// The evaluator's target-major schedule for a plan built by build_plan.
void build_eval_plan(const Plan &P, EvalPlan *out);

// A modulus the library accepts: a prime or a power of two in 2..255.
bool modulus_ok(uint32_t m);

// Residues per label and words per label for a modulus (2..255).
uint32_t label_lambda(uint32_t m);
uint32_t label_words(uint32_t m);

// Fills one ModConst for modulus m (everything except woff, wkoff, up, down).
void fill_mod_const(uint32_t m, ModConst *mc);

// Constants for floor(x / d), every x < x_bound (x_bound <= 2^32): if fix is
// 0, umulhi(x, M) >> s; otherwise the round-up method with a fix-up step.
void division_constants(uint32_t d, uint64_t x_bound, uint32_t *M, uint32_t *s, uint32_t *fix);

// 24-bit multiply-shift constants: floor(x / m) = (x * M) >> s for every
// x < x_bound with x * M < 2^32 and M < 2^24.  Returns false if none exist.
bool mul24_constants(uint32_t m, uint64_t x_bound, uint32_t *M, uint32_t *s);

uint32_t inverse_mod(uint32_t a, uint32_t m);

}  // namespace redash
