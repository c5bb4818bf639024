// Kernels and C ABI of the ReDASH scaling-gadget library for gfx950.
//
// One thread evaluates (or garbles) one gadget instance.  Labels are packed
// words laid out [word][gadget], so a wavefront's label accesses are 64
// consecutive words; the gate list and all per-modulus constants are uniform
// and come from the kernel argument block (scalar registers).  The AES round
// tables are staged into LDS once per workgroup.  Nothing here uses MFMA: the work is table lookups, XORs, 32-bit
// multiplies for digit extraction and small modular arithmetic.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "../../include/redash.h"
#include "device.hpp"
#include "plan.hpp"

namespace redash {

struct SeedKey {
    uint32_t w[44];
};

// ---------------------------------------------------------------------------
// Evaluator: the hot path (Sec. 3.4 gadget, Sec. 2.3 projection gates).
//
// LDS of a workgroup (addresses from 0: the kernel declares no static LDS):
// the 64 KiB two-table image, the 88 round-key words, then one 128-byte
// free-operation table per gate (up to kMaxTables).  The working labels stay in global memory, mostly in L2: the
// output tensor (and the working storage for Phase-B copies) holds every
// intermediate label, each gate reads its destination label and its table
// row before the AES runs and writes the destination back after it.
// ---------------------------------------------------------------------------
constexpr uint32_t kEvalTableBase = kTableRegionBytes + 384;  // after the 352 key bytes
// LDS bytes of an evaluator workgroup with ntab free-operation tables.
constexpr uint32_t eval_lds_bytes(uint32_t ntab) { return kEvalTableBase + ntab * kTableBytes; }
static_assert(kLdsKeyWords * 4 <= 384, "round keys overlap the free-operation tables");
static_assert(2 * (kEvalTableBase + kMaxTables * kTableBytes) <= 160 * 1024, "two workgroups per CU");
static_assert(sizeof(EvalPlan) <= 4096, "the evaluator's plan is passed as its kernel argument block");
// Two workgroups of 768 threads share a CU (2 x 64.3 KiB of LDS): six waves
// per SIMD, which caps the kernel at 80 VGPRs.
constexpr int kEvalBlock = 768;
constexpr int kEvalWaves = 6;
// The one-gadget-per-lane evaluator k_eval: workgroup size and waves per SIMD.
constexpr int kLaneBlock = 768;
constexpr int kLaneWaves = 6;
// The garbler: the same LDS image without the free-operation tables; two
// workgroups of 512 per CU, four waves per SIMD (up to 128 VGPRs).
constexpr int kGarbleBlock = 512;
constexpr int kGarbleWaves = 4;

// The four places a label can be (kLocIn, kLocOut, kLocWork, kLocZero) for
// one thread: word w of a label starts at base + (offset + w) n, and the
// thread's gadget adds its byte offset 4 a (below 2^32).
struct LabelBufs {
    const uint32_t *in;
    uint32_t *out, *work;
    uint64_t n;
    uint32_t aoff;
    // word 0 of modulus mc's label in place `loc` (not kLocZero); uniform
    __device__ __forceinline__ const uint32_t *base(uint32_t loc, const ModConst &mc) const {
        if (loc == kLocIn) return in + static_cast<uint64_t>(mc.woff) * n;
        if (loc == kLocOut) return out + static_cast<uint64_t>(mc.woff) * n;
        return work + static_cast<uint64_t>(mc.wkoff) * n;
    }
    __device__ __forceinline__ uint32_t *dest(uint32_t to_work, const ModConst &mc) const {
        return to_work ? work + static_cast<uint64_t>(mc.wkoff) * n : out + static_cast<uint64_t>(mc.woff) * n;
    }
    // (opaque: the zero extension of the offset must sit next to the access,
    // or the scalar-base addressing form is not selected)
    __device__ __forceinline__ uint32_t get(const uint32_t *b, uint32_t w) const {
        return *reinterpret_cast<const uint32_t *>(reinterpret_cast<const char *>(b + w * n) + opaque(aoff));
    }
    __device__ __forceinline__ void put(uint32_t *b, uint32_t w, uint32_t v) const {
        *reinterpret_cast<uint32_t *>(reinterpret_cast<char *>(b + w * n) + opaque(aoff)) = v;
    }
};

// Fills the free-operation tables (gates 0..ntab-1 that have one): byte v of
// gate g's table is c (v mod m) mod m.  Wave w fills gates w, w + waves, ...
__device__ __forceinline__ void stage_free_op_tables(const Plan &P, uint32_t *lds, int tid, uint32_t nwaves) {
    const uint32_t wave = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(tid) / 64u);
    const uint32_t lane = static_cast<uint32_t>(tid) % 64u;
    for (uint32_t g = wave; g < P.ntab; g += nwaves) {
        const uint32_t d = P.gate[g];
        if (!gate_tab(d) || lane >= kTableBytes / 4) continue;
        const uint32_t m = P.mod[gate_dst(d)].m, c = gate_coeff(d);
        uint32_t w = 0;
        for (uint32_t k = 0; k < 4; ++k) {
            const uint32_t v = 4 * lane + k;
            w |= ((c * (v % m)) % m) << (8 * k);
        }
        lds[(kEvalTableBase + g * kTableBytes) / 4 + lane] = w;
    }
}

// ---------------------------------------------------------------------------
// The one-gadget-per-lane evaluator, target-major (EvalPlan): a block's two
// target labels stay in registers from their first gate to their last, so
// each is read and written once; a step hashes one digit label for one gate
// of each slot (four AES blocks interleaved) or for one slot.  Updates always
// act on slot 0: slot 1 is brought there by swapping the two slots.
// ---------------------------------------------------------------------------

__device__ __forceinline__ void swap_slots(uint32_t (&T)[2][kMaxW]) {
    static_for<kMaxW>([&](auto w) {
        const uint32_t v = T[0][w];
        T[0][w] = T[1][w];
        T[1][w] = v;
    });
}

// Register labels are right-aligned: a label of W words sits in positions
// kMaxW - W .. kMaxW - 1 of its array (W is 4, 5 or 6), so its last word --
// the one with its own digit count -- is always at position kMaxW - 1 and
// every word is at a constant position: the word loops below are unrolled
// with a uniform test per position, and no register moves.
__device__ __forceinline__ uint32_t label_off(const ModConst &mc) { return kMaxW - mc.W; }

__device__ __forceinline__ void load_label(uint32_t (&T)[kMaxW], const LabelBufs &LB, uint32_t loc, const ModConst &mc,
                                           bool from_input) {
    static_for<kMaxW>([&](auto p) { T[p] = 0; });
    if (from_input) {
        const uint32_t off = label_off(mc);
        const uint32_t *b = LB.base(loc, mc);
        static_for<kMaxW>([&](auto p) {
            if (p >= static_cast<int>(off)) T[p] = LB.get(b, p - off);
        });
    }
}

__device__ __forceinline__ void store_label(const uint32_t (&T)[kMaxW], const LabelBufs &LB, uint32_t to_work,
                                            const ModConst &mc) {
    const uint32_t off = label_off(mc);
    uint32_t *b = LB.dest(to_work, mc);
    static_for<kMaxW>([&](auto p) {
        if (p >= static_cast<int>(off)) LB.put(b, p - off, T[p]);
    });
}

// XOR-fold of a right-aligned register label with OFF = kMaxW - W: word w
// goes into lane w mod 4.
template <int OFF>
__device__ __forceinline__ void fold_regs(const uint32_t (&T)[kMaxW], uint32_t (&x)[4]) {
    static_for<kMaxW - OFF>([&](auto w) { x[w & 3] ^= T[w + OFF]; });
}

// Moduli without the fast constants (4 and 16, whose fields fill a word, and
// the primes 41, 47, 53, 59 and 61, whose split parts are too large for the
// 24-bit digit steps): one residue at a time with 32-bit divisions, over all
// kMaxW positions in a rolled loop that rotates the label and the row by one
// word per position (kMaxW rotations put both back in place).  The gadget
// configurations in use all take the fast path.
__device__ __forceinline__ void reg_update_generic(uint32_t e, const ModConst &mm, uint32_t (&V)[8],
                                                   uint32_t (&row)[kMaxW], uint32_t (&T)[kMaxW]) {
    const uint32_t coeff = eg_coeff(e), off = label_off(mm);
#pragma unroll 1
    for (uint32_t p = 0; p < static_cast<uint32_t>(kMaxW); ++p) {
        const uint32_t l = next_word(T);
        const uint32_t rw = next_word(row);
        uint32_t res = l;
        if (p >= off) {
            const bool last = (p + 1 == static_cast<uint32_t>(kMaxW));
            const uint32_t nres = last ? mm.glast : mm.g;
            uint32_t D = frac_carry_any(V, last ? mm.pw_last : mm.pw_g);
            res = 0;
            for (uint32_t j = nres; j-- > 0;) {
                uint32_t pd;
                if (j) {
                    const uint32_t qd = div_m(D, mm);
                    pd = D - qd * mm.m;
                    D = qd;
                } else {
                    pd = D;
                }
                const uint32_t ev = add_mod(pd, field(rw, j, mm), mm.m);
                const uint32_t lj = field(l, j, mm);
                const uint32_t r = eg_kind(e) == 0 ? mul_mod(coeff, sub_mod(lj, ev, mm.m), mm)
                                                   : add_mod(lj, mul_mod(coeff, ev, mm), mm.m);
                res |= r << (mm.b * j);
            }
        }
        T[kMaxW - 1] = res;
        row[kMaxW - 1] = rw;
    }
}

// The full words (positions kMaxW - W .. kMaxW - 2) with the word shape
// (residues per word, bits per residue) known at compile time: the shape is
// dispatched once per gate, not once per word.
template <bool ACC, bool TAB, int NR, int BB>
__device__ __forceinline__ void reg_full_words(const ModConst &mm, uint32_t coeff, uint32_t (&V)[8],
                                               const uint32_t (&row)[kMaxW], uint32_t (&T)[kMaxW], uint32_t tk) {
    const uint32_t off = label_off(mm);
    static_for<kMaxW - 1>([&](auto p) {
        if (p >= static_cast<int>(off)) {
            const uint32_t D = frac_mul_carry(V, mm.pw_g);
            T[p] = fast_word_c<ACC, NR, BB, TAB>(D, mm.lo_M_f, mm.lo_s_f, mm.pw_lo_f, mm.fc_hi_f, mm.fc_lo_f, row[p],
                                                 T[p], coeff, mm, tk);
        }
    });
}

template <bool ACC, bool TAB>
__device__ __forceinline__ void reg_update_fast(uint32_t e, const ModConst &mm, uint32_t (&V)[8],
                                                const uint32_t (&row)[kMaxW], uint32_t (&T)[kMaxW], uint32_t tk) {
    const uint32_t coeff = eg_coeff(e);
    // full words: g = floor(32 / b) residues of b bits
    switch (mm.fd ? mm.g | (mm.b << 8) : 0u) {
#define REDASH_FULL(NR, BB) \
    case (NR) | ((BB) << 8): reg_full_words<ACC, TAB, NR, BB>(mm, coeff, V, row, T, tk); break;
        REDASH_FULL(16, 2) REDASH_FULL(10, 3) REDASH_FULL(8, 4) REDASH_FULL(6, 5) REDASH_FULL(5, 6)
        REDASH_FULL(4, 7) REDASH_FULL(4, 8)
#undef REDASH_FULL
        default: {
            const uint32_t off = label_off(mm);
            static_for<kMaxW - 1>([&](auto p) {
                if (p >= static_cast<int>(off)) {
                    const uint32_t D = frac_mul_carry(V, mm.pw_g);
                    T[p] = fast_word<ACC>(D, mm.g, mm.nlo_f, mm.lo_M_f, mm.lo_s_f, mm.pw_lo_f, row[p], T[p], coeff,
                                          mm);
                }
            });
        }
    }
    const uint32_t D = frac_mul_carry(V, mm.pw_last);
    T[kMaxW - 1] = fast_word_any<ACC, TAB>(D, mm.glast, mm.nlo_l, mm.lo_M_l, mm.lo_s_l, mm.pw_lo_l, mm.fc_hi_l,
                                           mm.fc_lo_l, row[kMaxW - 1], T[kMaxW - 1], coeff, mm, tk);
}

// Applies gate g's free operation to the register label T: E = row + pad,
// then L <- c (L - E) (sub: division step and the recursion of Eq.
// rns_to_mrs) or L <- L + c E (acc: the mixed-radix recombination onto a
// scaling modulus).  For an output modulus m <= 42 the product c (v mod m)
// mod m comes from the gate's byte table in LDS: a sub gate's new residue is
// T[l + 2m - p - r], an acc gate's is l + T[p + r] reduced once.
__device__ __forceinline__ void reg_update(uint32_t g, uint32_t e, const ModConst &mm, uint32_t (&V)[8],
                                           uint32_t (&row)[kMaxW], uint32_t (&T)[kMaxW]) {
    if (mm.m == 2) {  // W = 4: positions 2..5
        const bool flip = eg_kind(e) == 0 || (eg_coeff(e) & 1u);  // sub: q^{-1} = 1 mod 2
        if (flip) {
            static_for<4>([&](auto w) { T[w + 2] ^= bits_word(V, w) ^ row[w + 2]; });
        }
    } else if (eg_tab(e)) {
        const uint32_t tk = kEvalTableBase + g * kTableBytes + (eg_kind(e) ? 0u : mm.two_m);
        if (eg_kind(e)) {
            reg_update_fast<true, true>(e, mm, V, row, T, tk);
        } else {
            reg_update_fast<false, true>(e, mm, V, row, T, tk);
        }
    } else if (mm.fast) {
        if (eg_kind(e)) {
            reg_update_fast<true, false>(e, mm, V, row, T, 0);
        } else {
            reg_update_fast<false, false>(e, mm, V, row, T, 0);
        }
    } else {
        reg_update_generic(e, mm, V, row, T);
    }
}

// The free-operation tables of an EvalPlan (as stage_free_op_tables).
__device__ __forceinline__ void stage_free_op_tables_e(const EvalPlan &P, uint32_t *lds, int tid, uint32_t nwaves) {
    const uint32_t wave = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(tid) / 64u);
    const uint32_t lane = static_cast<uint32_t>(tid) % 64u;
    for (uint32_t g = wave; g < P.ntab; g += nwaves) {
        const uint32_t e = P.egate[g];
        if (!eg_tab(e) || lane >= kTableBytes / 4) continue;
        const uint32_t m = P.mod[eg_dst(e)].m, c = eg_coeff(e);
        uint32_t w = 0;
        for (uint32_t k = 0; k < 4; ++k) {
            const uint32_t v = 4 * lane + k;
            w |= ((c * (v % m)) % m) << (8 * k);
        }
        lds[(kEvalTableBase + g * kTableBytes) / 4 + lane] = w;
    }
}

// One step's NG gates g, g+1 (NG = 2) or g: requests their rows (the colour
// is known before hashing), then runs the 2 NG AES blocks interleaved.
//
// The gadget index a (below 2^30) is a 32-bit register: the row offset
// a (q-1) W + (c-1) W and the tweak (a0 + a) G + g are each one
// 32 x 32 + 64-bit multiply-add from it, instead of 64-bit values kept live
// across the whole gadget.
__device__ __forceinline__ uint64_t mad64(uint32_t x, uint32_t y, uint64_t z) {
    return static_cast<uint64_t>(x) * y + z;
}

template <int NG>
__device__ __forceinline__ void step_hash(const EvalPlan &P, uint32_t g, uint32_t q, const uint32_t (&x)[4],
                                          uint32_t colour, const PermTE02 &TT, const uint32_t *K, uint32_t a,
                                          const uint32_t *__restrict__ tab, uint32_t (&V)[2][8],
                                          uint32_t (&row)[2][kMaxW]) {
    static_for<NG>([&](auto j) {
        const uint32_t e = P.egate[g + j];
        const uint32_t Wd = P.mod[eg_dst(e)].W;
        static_for<kMaxW>([&](auto w) { row[j][w] = 0; });
        if (colour != 0) {  // right-aligned like the labels
            const uint32_t *rp = tab + static_cast<uint64_t>(eg_toff(e)) * P.n +
                                 mad64(opaque(a), (q - 1) * Wd, static_cast<uint64_t>(colour - 1) * Wd);
            const int off = kMaxW - static_cast<int>(Wd);
            static_for<kMaxW>([&](auto p) {
                if (p >= off) row[j][p] = rp[p - off];
            });
        }
    });
    uint32_t Vn[NG][8];
    const uint64_t tau = mad64(opaque(a), P.G, P.a0 * P.G + g);
    hash_fraction_n<NG>(TT, LdsKey{K}, x[0], x[1], x[2], x[3], tau, P.gid, Vn);
    static_for<NG>([&](auto j) { static_for<8>([&](auto l) { V[j][l] = Vn[j][l]; }); });
}

template <int BLOCK>
__global__ void __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(kLaneWaves, kLaneWaves)))
k_eval(const EvalPlan P, const uint32_t *__restrict__ in, const uint32_t *__restrict__ tab, uint32_t *out,
       uint32_t *work) {
    extern __shared__ uint32_t lds[];
    uint32_t *K = lds + kTableRegionBytes / 4;
    const int tid = threadIdx.x;
    const int nthr = blockDim.x;  // BLOCK or fewer (a multiple of 64)
    stage_perm_te02(lds, tid, nthr);
    stage_hash_key(K, tid, nthr);
    stage_free_op_tables_e(P, lds, tid, static_cast<uint32_t>(nthr) / 64u);
    __syncthreads();
    const PermTE02 TT = perm_te02();
    const uint32_t a = blockIdx.x * static_cast<uint32_t>(nthr) + static_cast<uint32_t>(tid);  // n < 2^30
    if (a >= P.n) return;  // no barrier follows
    const LabelBufs LB{in, out, work, P.n, a * 4u};

    for (uint32_t b = 0; b < P.nblocks; ++b) {
        const uint32_t bd = P.block[b];
        uint32_t T[2][kMaxW];
        load_label(T[0], LB, kLocIn, P.mod[bk_mod0(bd)], bk_in0(bd) != 0);
        load_label(T[1], LB, kLocIn, P.mod[bk_mod1(bd)], bk_two(bd) && bk_in1(bd));
        const uint32_t s_end = bk_first(bd) + bk_steps(bd);
        for (uint32_t s = bk_first(bd); s < s_end; ++s) {
            const uint32_t sd = P.step[s];
            const bool two = st_two(sd) != 0;
            const bool alone1 = !two && st_slot1(sd);
            if (alone1) swap_slots(T);  // slot 1's gate acts on slot 0's registers
            // The digit label: folded into 128 bits for the hash, colour =
            // residue 0.  A residue >= q only occurs in a malformed input
            // label; it selects the implicit zero row, the output is garbage
            // and decode flags it.
            const ModConst mq = P.mod[st_dmod(sd)];
            const uint32_t q = mq.m;
            uint32_t x[4] = {0, 0, 0, 0}, w0;
            if (st_dloc(sd) == kDigSlot0) {  // the block's first target, now in T[1]
                switch (label_off(mq)) {
                    case 0: fold_regs<0>(T[1], x); w0 = T[1][0]; break;
                    case 1: fold_regs<1>(T[1], x); w0 = T[1][1]; break;
                    default: fold_regs<2>(T[1], x); w0 = T[1][2]; break;
                }
            } else {
                const uint32_t *dig = LB.base(st_dloc(sd), mq);
                w0 = LB.get(dig, 0);
                x[0] = w0;
                static_for<kMaxW - 1>([&](auto w1) {
                    constexpr int w = decltype(w1)::value + 1;
                    if (w < static_cast<int>(mq.W)) x[w & 3] ^= LB.get(dig, w);
                });
            }
            uint32_t colour = w0 & mq.mask;
            if (colour >= q) colour = 0;
            const uint32_t g = st_gate(sd);
            uint32_t V[2][8], row[2][kMaxW];
            if (two) {
                step_hash<2>(P, g, q, x, colour, TT, K, a, tab, V, row);
            } else {
                step_hash<1>(P, g, q, x, colour, TT, K, a, tab, V, row);
            }
            // one copy of the update code: gate j acts on slot 0, then the
            // slots (and the gate's pad and row) move along
            const uint32_t ng = two ? 2u : 1u;
#pragma unroll 1
            for (uint32_t j = 0; j < ng; ++j) {
                const uint32_t e = P.egate[g + j];
                const ModConst mm = P.mod[eg_dst(e)];
                reg_update(g + j, e, mm, V[0], row[0], T[0]);
                if (two) {
                    swap_slots(T);
                    static_for<8>([&](auto l) { V[0][l] = V[1][l]; });
                    static_for<kMaxW>([&](auto w) { row[0][w] = row[1][w]; });
                }
            }
            if (alone1) swap_slots(T);
            const uint32_t f = st_store(sd);
            if (f & 3u) store_label(T[0], LB, (f >> 1) & 1u, P.mod[bk_mod0(bd)]);
            if ((f & 3u) == 3u) store_label(T[0], LB, 0, P.mod[bk_mod0(bd)]);
            if (f & 12u) store_label(T[1], LB, (f >> 3) & 1u, P.mod[bk_mod1(bd)]);
            if ((f & 12u) == 12u) store_label(T[1], LB, 0, P.mod[bk_mod1(bd)]);
        }
    }
}

// ---------------------------------------------------------------------------
// The evaluator for calls too small to fill the GPU one gadget per lane.
// A group of `split` waves shares 64 gadgets (one per lane); within a run of
// gates that share a digit label (distinct destinations, no dependence among
// them) wave j of the group takes gates j, j + split, ...; a workgroup
// barrier after each run makes the updated labels (in global memory; the
// waves of a workgroup share one write-through L1) visible to every wave
// before the next run reads them.  The gate a wave works on stays uniform.
// Same LDS image as k_eval.
//
// One launch may hold two kinds of workgroup: 0 .. nb0-1 give each group
// split0 waves, the others split1; the gadgets are first, first + 1, ... in
// workgroup order (blockDim / split0 per workgroup of the first kind, then
// blockDim / split1 per workgroup of the second).  The workgroups are
// dispatched in order, so the second kind takes the CUs the first frees.
// ---------------------------------------------------------------------------
struct SplitLaunch {
    uint32_t first;   // the launch's first gadget
    uint32_t nb0;     // workgroups of the first kind
    uint32_t split0;  // waves per 64 gadgets in them (2, 4 or 12)
    uint32_t split1;  // waves per 64 gadgets in the others
};
static_assert(sizeof(Plan) + 4 * sizeof(void *) + sizeof(SplitLaunch) <= 4096,
              "the split evaluator's arguments fit the kernel argument block");

template <int BLOCK>
__global__ void __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(kEvalWaves, kEvalWaves)))
k_eval_split(const Plan P, const uint32_t *__restrict__ in, const uint32_t *__restrict__ tab, uint32_t *out,
             uint32_t *work, const SplitLaunch L) {
    extern __shared__ uint32_t lds[];
    uint32_t *K = lds + kTableRegionBytes / 4;
    const int tid = threadIdx.x;
    const int nthr = blockDim.x;  // a multiple of 64 split0 and of 64 split1, at most BLOCK
    stage_perm_te02(lds, tid, nthr);
    stage_hash_key(K, tid, nthr);
    stage_free_op_tables(P, lds, tid, static_cast<uint32_t>(nthr) / 64u);
    __syncthreads();
    const PermTE02 TT = perm_te02();
    const uint32_t wave = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(tid) / 64u);
    const uint32_t wg = blockIdx.x;
    const bool kind1 = wg >= L.nb0;
    const uint32_t split = kind1 ? L.split1 : L.split0;
    const uint32_t part = wave % split, grp = wave / split;
    const uint32_t per0 = static_cast<uint32_t>(nthr) / L.split0;
    const uint32_t start = kind1 ? L.nb0 * per0 + (wg - L.nb0) * (static_cast<uint32_t>(nthr) / L.split1) : wg * per0;
    const uint64_t a = static_cast<uint64_t>(L.first) + start + grp * 64u + static_cast<uint32_t>(tid) % 64u;
    const bool live = a < P.n;  // dead lanes still take every barrier
    const LabelBufs LB{in, out, work, P.n, static_cast<uint32_t>(live ? a : 0) * 4u};
    const uint64_t tau0 = (P.a0 + a) * P.G;
    uint64_t toff = 0;  // table offset of gate g
    for (uint32_t g = 0; g < P.G;) {
        const uint32_t src = gate_src(P.gate[g]);
        uint32_t r = 1;
        while (g + r < P.G && gate_src(P.gate[g + r]) == src) ++r;
        const ModConst mq = P.mod[src];
        const uint32_t q = mq.m;
        // Every gate of the run hashes the same digit label: the wave reads,
        // folds and colours it once per run.
        uint32_t x[4] = {0, 0, 0, 0}, colour = 0;
        if (live && part < r) {
            const uint32_t *dig = LB.base(gate_dsrc(P.gate[g + part]), mq);
            const uint32_t w0 = LB.get(dig, 0);
            x[0] = w0;
            static_for<kMaxW - 1>([&](auto w1) {
                constexpr int w = decltype(w1)::value + 1;
                if (w < static_cast<int>(mq.W)) x[w & 3] ^= LB.get(dig, w);
            });
            colour = w0 & mq.mask;
            if (colour >= q) colour = 0;
        }
        for (uint32_t i = 0; i < r; ++i) {
            const uint32_t d = P.gate[g + i];
            if (i % split == part && live) {
                const ModConst mm = P.mod[gate_dst(d)];
                const uint32_t Wd = mm.W;
                // the row (right-aligned, as the register labels)
                uint32_t row[kMaxW];
                static_for<kMaxW>([&](auto p) { row[p] = 0; });
                if (colour != 0) {
                    const uint32_t *rp = tab + toff + (a * (q - 1) + (colour - 1)) * Wd;
                    const int off = kMaxW - static_cast<int>(Wd);
                    static_for<kMaxW>([&](auto p) {
                        if (p >= off) row[p] = rp[p - off];
                    });
                }
                uint32_t T[kMaxW];
                load_label(T, LB, gate_tsrc(d), mm, gate_tsrc(d) != kLocZero);
                uint32_t Vn[1][8];
                hash_fraction_n<1, true>(TT, LdsKey{K}, x[0], x[1], x[2], x[3], tau0 + g + i, P.gid, Vn);
                const uint32_t e = gate_dst(d) | (gate_kind(d) << 4) | (gate_tab(d) << 5) | (gate_coeff(d) << 6);
                reg_update(g + i, e, mm, Vn[0], row, T);
                store_label(T, LB, gate_tdst(d), mm);
            }
            toff += P.n * (q - 1) * P.mod[gate_dst(d)].W;
        }
        __syncthreads();
        g += r;
    }
}

// ---------------------------------------------------------------------------
// Garbler: offsets, zero-labels, garbled rows.
// ---------------------------------------------------------------------------

// Offsets R_m: digits of rho(1, i) in the radices (r0, m, m, ...), then
// residue 0 mapped to a unit of Z_m (d + 1 for a prime m, r0 = m - 1;
// 2d + 1 for m = 2^l, r0 = m/2), so that the m colours of a wire are
// distinct.  One thread per modulus.
__global__ void __launch_bounds__(64) k_offsets(const Plan P, const SeedKey key, uint32_t *__restrict__ offsets) {
    __shared__ uint32_t TT[kTableWords];
    stage_round_tables(TT, threadIdx.x, 64);
    __syncthreads();
    const uint32_t i = threadIdx.x;
    if (i >= P.k) return;
    const ModConst &mc = P.mod[i];
    uint32_t V[8];
    prg_fraction(TT, key.w, 1u, i, V);
    uint32_t words[kMaxW] = {0, 0, 0, 0, 0, 0};
    for (uint32_t r = 0; r < mc.lam; ++r) {
        const uint32_t radix = r ? mc.m : mc.r0;
        uint32_t dgt = frac_mul_carry(V, radix);
        if (r == 0) dgt = (mc.r0 == mc.m - 1) ? dgt + 1 : 2 * dgt + 1;
        const uint32_t w = r / mc.g, pos = r % mc.g;
#pragma unroll
        for (int ww = 0; ww < kMaxW; ++ww)
            if (ww == static_cast<int>(w)) words[ww] |= dgt << (mc.b * pos);
    }
    for (uint32_t w = 0; w < mc.W; ++w) {
#pragma unroll
        for (int ww = 0; ww < kMaxW; ++ww)
            if (ww == static_cast<int>(w)) offsets[mc.woff + w] = words[ww];
    }
}

__device__ __forceinline__ uint32_t inverse_unit(uint32_t r, const ModConst &mc) {
    // r^(phi - 1) mod m for a unit r, phi the order of the unit group
    // (m - 1 for a prime, m/2 for a power of two)
    uint32_t e = mc.phi - 1, base = r, acc = 1 % mc.m;
    while (e) {
        if (e & 1u) acc = mul_mod(acc, base, mc);
        base = mul_mod(base, base, mc);
        e >>= 1;
    }
    return acc;
}

// The garbler's label access: like the evaluator's, except that a label read
// from the input tensor (the input zero-labels Z) is taken as Z - (P/2 mod m) R,
// the ShiftUp of Sec. 3.4 applied as a free constant addition.
__device__ __forceinline__ void load_zero_label(const LabelBufs &LB, uint32_t loc, const ModConst &mc,
                                                const uint32_t *__restrict__ offsets, uint32_t (&L)[kMaxW]) {
    static_for<kMaxW>([&](auto w) { L[w] = 0; });
    if (loc == kLocZero) return;
    const uint32_t *p = LB.base(loc, mc);
    const uint32_t neg_up = (mc.m - mc.up) % mc.m;
    static_for<kMaxW>([&](auto w) {
        if (w < static_cast<int>(mc.W)) {
            L[w] = LB.get(p, w);
            if (loc == kLocIn) L[w] = label_axpy(L[w], offsets[mc.woff + w], neg_up, w, mc);
        }
    });
}

// One garbled row over Z_m: (B - pad) word by word, pad the first lambda_m
// base-m digits of the hash fraction V (consumed), stored at rp.
__device__ __forceinline__ void store_row(uint32_t (&V)[8], const uint32_t (&B)[kMaxW], const ModConst &mm,
                                          uint32_t *rp) {
    if (mm.m == 2) {
#pragma unroll
        for (int w = 0; w < 4; ++w) rp[w] = B[w] ^ bits_word(V, w);
        return;
    }
    uint32_t b[kMaxW];
    static_for<kMaxW>([&](auto w) { b[w] = B[w]; });
    if (mm.fast) {
#pragma unroll 1
        for (uint32_t w = 0; w + 1 < mm.W; ++w) {
            const uint32_t D = frac_mul_carry(V, mm.pw_g);
            rp[w] = row_word_any(D, mm.g, mm.lo_M_f, mm.lo_s_f, mm.pw_lo_f, mm.fc_hi_f, mm.fc_lo_f, next_word(b), mm);
        }
        const uint32_t D = frac_mul_carry(V, mm.pw_last);
        rp[mm.W - 1] = row_word_any(D, mm.glast, mm.lo_M_l, mm.lo_s_l, mm.pw_lo_l, mm.fc_hi_l, mm.fc_lo_l, b[0], mm);
    } else {
#pragma unroll 1
        for (uint32_t w = 0; w < mm.W; ++w) rp[w] = label_sub(next_word(b), pad_word(V, w, mm), w, mm);
    }
}

// Hash fractions of two labels (folded into xa, xb) under the same tweak tau:
// the four AES blocks run interleaved.
__device__ __forceinline__ void hash_fraction_two(const PermTE02 &T, const LdsKey &rk, const uint32_t (&xa)[4],
                                                  const uint32_t (&xb)[4], uint64_t tau, uint32_t gid,
                                                  uint32_t (&Va)[8], uint32_t (&Vb)[8]) {
    uint32_t u[2][4], s[4][4], k0[2], k1[2];
    static_for<2>([&](auto j) {
        const uint32_t(&x)[4] = j ? xb : xa;
        u[j][0] = x[2];
        u[j][1] = x[3];
        u[j][2] = x[2] ^ x[0];
        u[j][3] = x[3] ^ x[1];
    });
    static_for<2>([&](auto h) {
        const uint64_t tw = tau * 4u + static_cast<uint64_t>(h);
        k0[h] = static_cast<uint32_t>(tw);
        k1[h] = static_cast<uint32_t>(tw >> 32);
    });
    static_for<2>([&](auto j) {
        static_for<2>([&](auto h) {
            s[2 * j + h][0] = u[j][0] ^ k0[h];
            s[2 * j + h][1] = u[j][1] ^ k1[h];
            s[2 * j + h][2] = u[j][2];
            s[2 * j + h][3] = u[j][3] ^ gid;
        });
    });
    aes128_encrypt_n<4>(T, s, rk);
    static_for<2>([&](auto h) {
        Va[4 * h + 0] = s[h][0] ^ u[0][0] ^ k0[h];
        Va[4 * h + 1] = s[h][1] ^ u[0][1] ^ k1[h];
        Va[4 * h + 2] = s[h][2] ^ u[0][2];
        Va[4 * h + 3] = s[h][3] ^ u[0][3] ^ gid;
        Vb[4 * h + 0] = s[2 + h][0] ^ u[1][0] ^ k0[h];
        Vb[4 * h + 1] = s[2 + h][1] ^ u[1][1] ^ k1[h];
        Vb[4 * h + 2] = s[2 + h][2] ^ u[1][2];
        Vb[4 * h + 3] = s[2 + h][3] ^ u[1][3] ^ gid;
    });
}

__device__ __forceinline__ void fold_label(const uint32_t (&A)[kMaxW], const ModConst &mq, uint32_t (&x)[4]) {
    x[0] = A[0];
    x[1] = x[2] = x[3] = 0;
    static_for<kMaxW - 1>([&](auto w1) {
        constexpr int w = decltype(w1)::value + 1;
        if (w < static_cast<int>(mq.W)) x[w & 3] ^= A[w];
    });
}

// Garbler (Sec. 2.3 projection gates with row reduction, the gadget of
// Sec. 3.4 applied to zero-labels).  One thread per gadget; labels live
// where the evaluator keeps them (zin read with the ShiftUp, zout, work).
// Per gate q -> m the q labels of the digit wire are walked by colour:
// colour c holds the value v_c = (c - c_0) R_q[0]^{-1} mod q, so the label
// steps by the uniform label R_q[0]^{-1} R_q.  Colour 0 gives
// B0 = H(A_{v_0}) - (v_0 mod m) R_m; colour c >= 1 gives the row
// B0 + (v_c mod m) R_m - H(A_{v_c}), two colours per AES batch.  The walk
// keeps B_c = B0 + (v_c mod m) R_m, starting from B_0 = H(A_{v_0}).
// GIVEN: the input zero-labels are the caller's (zin, read only; zin_w
// unused), e.g. the output zero-labels of a garbled linear layer; otherwise
// they are drawn from the PRG into zin_w (== zin).
template <int BLOCK, bool GIVEN>
__global__ void __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(kGarbleWaves, kGarbleWaves)))
k_garble(const Plan P, const SeedKey key, const uint32_t *__restrict__ offsets, const uint32_t *zin,
         uint32_t *zin_w, uint32_t *zout, uint32_t *__restrict__ tab, uint32_t *work) {
    extern __shared__ uint32_t lds[];
    uint32_t *K = lds + kTableRegionBytes / 4;
    const int tid = threadIdx.x;
    const int nthr = blockDim.x;  // BLOCK or fewer (a multiple of 64)
    stage_perm_te02(lds, tid, nthr);
    stage_hash_key(K, tid, nthr);
    __syncthreads();
    const PermTE02 TT = perm_te02();
    const LdsKey HK{K};
    const uint64_t a = static_cast<uint64_t>(blockIdx.x) * nthr + tid;
    if (a >= P.n) return;  // no barrier follows
    const uint64_t n = P.n;
    const uint64_t ga = P.a0 + a;
    const LabelBufs LB{zin, zout, work, n, static_cast<uint32_t>(a) * 4u};

    // Input zero-labels Z: digits of rho(2, ga k + i) (Sec. 2.3 label sampling).
    for (uint32_t i = 0; i < (GIVEN ? 0u : P.k); ++i) {
        const ModConst mc = P.mod[i];
        uint32_t s[1][4];
        uint32_t V[8];
        static_for<2>([&](auto h) {
            const uint64_t c = (ga * P.k + i) * 2u + static_cast<uint64_t>(h);
            s[0][0] = static_cast<uint32_t>(c);
            s[0][1] = static_cast<uint32_t>(c >> 32);
            s[0][2] = 0;
            s[0][3] = 2u << 24;
            aes128_encrypt_n<1>(TT, s, ArgKey{key.w});
            static_for<4>([&](auto l) { V[4 * h + l] = s[0][l]; });
        });
        uint32_t *dst = zin_w + static_cast<uint64_t>(mc.woff) * n;
        for (uint32_t w = 0; w < mc.W; ++w) LB.put(dst, w, prg_word(V, w, mc));
    }

    const uint64_t tau0 = ga * P.G;
    uint64_t toff = 0;
    for (uint32_t g = 0; g < P.G; ++g) {
        const uint32_t d = P.gate[g];
        const ModConst mq = P.mod[gate_src(d)];
        const ModConst mm = P.mod[gate_dst(d)];
        const uint32_t q = mq.m, m = mm.m;
        uint32_t Rq[kMaxW], Rm[kMaxW];
        static_for<kMaxW>([&](auto w) {
            Rq[w] = w < static_cast<int>(mq.W) ? offsets[mq.woff + w] : 0u;
            Rm[w] = w < static_cast<int>(mm.W) ? offsets[mm.woff + w] : 0u;
        });
        uint32_t A[kMaxW], T[kMaxW];
        load_zero_label(LB, gate_dsrc(d), mq, offsets, A);
        load_zero_label(LB, gate_tsrc(d), mm, offsets, T);
        const uint32_t rinv = inverse_unit(Rq[0] & mq.mask, mq);
        // v: the value of colour 0; A <- A0 + v R_q
        uint32_t v = mul_mod((q - (A[0] & mq.mask)) % q, rinv, mq);
        static_for<kMaxW>([&](auto w) {
            if (w < static_cast<int>(mq.W)) A[w] = label_axpy(A[w], Rq[w], v, w, mq);
        });
        // uniform steps: the input label by rinv R_q, the output label by
        // (rinv mod m) R_m, or ((rinv - q) mod m) R_m when v wraps past q
        // (split into even and odd fields for swar_add; m = 2 steps by XOR)
        const uint32_t s1 = rinv % m, s2 = (rinv % m + m - q % m) % m;
        uint32_t Rse[kMaxW], Rso[kMaxW], U1e[kMaxW], U1o[kMaxW], U2e[kMaxW], U2o[kMaxW];
        static_for<kMaxW>([&](auto w) {
            const uint32_t rs = w < static_cast<int>(mq.W) ? label_axpy(0u, Rq[w], rinv, w, mq) : 0u;
            const uint32_t u1 = w < static_cast<int>(mm.W) ? label_axpy(0u, Rm[w], s1, w, mm) : 0u;
            const uint32_t u2 = w < static_cast<int>(mm.W) ? label_axpy(0u, Rm[w], s2, w, mm) : 0u;
            Rse[w] = q == 2 ? rs : rs & mq.sw_even;
            Rso[w] = (rs >> mq.b) & mq.sw_even;
            U1e[w] = m == 2 ? u1 : u1 & mm.sw_even;
            U1o[w] = (u1 >> mm.b) & mm.sw_even;
            U2e[w] = m == 2 ? u2 : u2 & mm.sw_even;
            U2o[w] = (u2 >> mm.b) & mm.sw_even;
        });
        const uint64_t tau = tau0 + g;

        // colour 0: the pad H(A_v0) starts the walk B_c = B0 + (v_c mod m) R_m,
        // with B0 = H(A_v0) - (v0 mod m) R_m (row reduction: no row stored)
        uint32_t B[kMaxW];
        {
            uint32_t x[4], V0[1][8];
            fold_label(A, mq, x);
            hash_fraction_n<1>(TT, HK, x[0], x[1], x[2], x[3], tau, P.gid, V0);
            static_for<kMaxW>([&](auto w) { B[w] = 0; });
#pragma unroll 1
            for (uint32_t w = 0; w < mm.W; ++w) {
                const uint32_t pw = pad_word(V0[0], w, mm);
                static_for<kMaxW>([&](auto ww) {
                    if (ww == static_cast<int>(w)) B[ww] = pw;
                });
            }
        }
        // The free operation on the destination zero-label, as the evaluator
        // applies it to labels (E replaced by B0).
        {
            const uint32_t coeff = gate_coeff(d);
            const uint32_t negv = (m - v % m) % m;
            uint32_t *dst = LB.dest(gate_tdst(d), mm);
            static_for<kMaxW>([&](auto w) {
                if (w < static_cast<int>(mm.W)) {
                    const uint32_t b0 = label_axpy(B[w], Rm[w], negv, w, mm);
                    LB.put(dst, w,
                           gate_kind(d) == 0 ? label_scaled_sub(T[w], b0, coeff, w, mm)
                                             : label_axpy(T[w], b0, coeff, w, mm));
                }
            });
        }
        // colours 1..q-1, two per AES batch
        uint32_t *gate_rows = tab + toff + a * (q - 1) * mm.W;
        auto step = [&](uint32_t(&Ax)[kMaxW], uint32_t(&Bx)[kMaxW], uint32_t &vx) {
            static_for<kMaxW>([&](auto w) {
                if (w < static_cast<int>(mq.W)) Ax[w] = q == 2 ? Ax[w] ^ Rse[w] : swar_add(Ax[w], Rse[w], Rso[w], mq);
            });
            const uint32_t vn = vx + rinv;
            const bool wrap = vn >= q;
            vx = wrap ? vn - q : vn;
            static_for<kMaxW>([&](auto w) {
                if (w < static_cast<int>(mm.W))
                    Bx[w] = m == 2 ? Bx[w] ^ (wrap ? U2e[w] : U1e[w])
                                   : swar_add(Bx[w], wrap ? U2e[w] : U1e[w], wrap ? U2o[w] : U1o[w], mm);
            });
        };
#pragma unroll 1
        for (uint32_t c = 1; c < q; c += 2) {
            step(A, B, v);
            if (c + 1 < q) {
                uint32_t A2[kMaxW], B2[kMaxW];
                uint32_t v2 = v;
                static_for<kMaxW>([&](auto w) {
                    A2[w] = A[w];
                    B2[w] = B[w];
                });
                step(A2, B2, v2);
                uint32_t xa[4], xb[4], Va[8], Vb[8];
                fold_label(A, mq, xa);
                fold_label(A2, mq, xb);
                hash_fraction_two(TT, HK, xa, xb, tau, P.gid, Va, Vb);
                store_row(Va, B, mm, gate_rows + (c - 1) * mm.W);
                store_row(Vb, B2, mm, gate_rows + c * mm.W);
                static_for<kMaxW>([&](auto w) {
                    A[w] = A2[w];
                    B[w] = B2[w];
                });
                v = v2;
            } else {
                uint32_t x[4], V1[1][8];
                fold_label(A, mq, x);
                hash_fraction_n<1>(TT, HK, x[0], x[1], x[2], x[3], tau, P.gid, V1);
                store_row(V1[0], B, mm, gate_rows + (c - 1) * mm.W);
            }
        }
        toff += n * (q - 1) * mm.W;
    }
    // Output zero-labels: the working labels plus (P/(2s) mod m) R, the
    // ShiftDown of Sec. 3.4.
    for (uint32_t i = 0; i < P.k; ++i) {
        const ModConst mc = P.mod[i];
        uint32_t *p = zout + static_cast<uint64_t>(mc.woff) * n;
        for (uint32_t w = 0; w < mc.W; ++w)
            LB.put(p, w, label_axpy(LB.get(p, w), offsets[mc.woff + w], mc.down, w, mc));
    }
}

// ---------------------------------------------------------------------------
// Encode (stand-in for oblivious transfer) and decode.
// ---------------------------------------------------------------------------
template <int BLOCK>
__global__ void __launch_bounds__(BLOCK) k_encode(const Plan P, const int64_t *__restrict__ x,
                                                  const uint32_t *__restrict__ zero,
                                                  const uint32_t *__restrict__ offsets, uint32_t *__restrict__ lab) {
    __shared__ uint32_t Rl[kMaxK * kMaxW];
    for (uint32_t i = threadIdx.x; i < P.total_words; i += BLOCK) Rl[i] = offsets[i];
    __syncthreads();
    const uint64_t a = static_cast<uint64_t>(blockIdx.x) * BLOCK + threadIdx.x;
    if (a >= P.n) return;
    const uint64_t n = P.n;
    int64_t r = x[a] % static_cast<int64_t>(P.P);
    if (r < 0) r += static_cast<int64_t>(P.P);
    for (uint32_t i = 0; i < P.k; ++i) {
        const ModConst &mc = P.mod[i];
        const uint32_t v = static_cast<uint32_t>(static_cast<uint64_t>(r) % mc.m);
        const uint64_t base = static_cast<uint64_t>(mc.woff) * n + a;
        for (uint32_t w = 0; w < mc.W; ++w)
            lab[base + static_cast<uint64_t>(w) * n] = label_axpy(zero[base + static_cast<uint64_t>(w) * n],
                                                                  Rl[mc.woff + w], v, w, mc);
    }
}

__global__ void k_zero_u64(uint64_t *p) { *p = 0; }

template <int BLOCK>
__global__ void __launch_bounds__(BLOCK) k_decode(const Plan P, const uint32_t *__restrict__ Y,
                                                  const uint32_t *__restrict__ O, const uint32_t *__restrict__ offsets,
                                                  int64_t *__restrict__ y, unsigned long long *__restrict__ bad) {
    __shared__ uint32_t Rl[kMaxK * kMaxW];
    for (uint32_t i = threadIdx.x; i < P.total_words; i += BLOCK) Rl[i] = offsets[i];
    __syncthreads();
    const uint64_t a = static_cast<uint64_t>(blockIdx.x) * BLOCK + threadIdx.x;
    if (a >= P.n) return;
    const uint64_t n = P.n;
    bool ok = true;
    uint32_t v[kMaxK];
    for (uint32_t i = 0; i < P.k; ++i) {
        const ModConst &mc = P.mod[i];
        const uint64_t base = static_cast<uint64_t>(mc.woff) * n + a;
        const uint32_t y0 = Y[base] & mc.mask, o0 = O[base] & mc.mask;
        const uint32_t vi = mul_mod(sub_mod(y0, o0, mc.m), inverse_unit(Rl[mc.woff] & mc.mask, mc), mc);
        for (uint32_t w = 0; w < mc.W; ++w) {
            const uint64_t at = base + static_cast<uint64_t>(w) * n;
            if (label_axpy(O[at], Rl[mc.woff + w], vi, w, mc) != Y[at]) ok = false;
        }
#pragma unroll
        for (int j = 0; j < kMaxK; ++j)
            if (j == static_cast<int>(i)) v[j] = vi;
    }
    // Garner: mixed-radix digits d_i of the CRT value, then y = sum d_i prod_{l<i} m_l.
    uint64_t val = 0, weight = 1;
    uint32_t dig[kMaxK];
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
        if (i < static_cast<int>(P.k)) {
            const ModConst &mc = P.mod[i];
            uint32_t cur = 0, wmod = 1 % mc.m;  // sum_{j<i} d_j prod_{l<j} m_l  (mod m_i)
#pragma unroll
            for (int j = 0; j < kMaxK; ++j) {
                if (j < i) {
                    cur = add_mod(cur, mul_mod(dig[j] % mc.m, wmod, mc), mc.m);
                    wmod = mul_mod(wmod, P.mod[j].m % mc.m, mc);
                }
            }
            // wmod = prod_{l<i} m_l mod m_i, a unit since the base is coprime
            dig[i] = mul_mod(sub_mod(v[i], cur, mc.m), inverse_unit(wmod, mc), mc);
            val += static_cast<uint64_t>(dig[i]) * weight;
            weight *= mc.m;
        }
    }
    // signed range [-floor(P/2), ceil(P/2) - 1] (Sec. 2.4)
    int64_t out = static_cast<int64_t>(val);
    if (val >= (P.P + 1) / 2) out -= static_cast<int64_t>(P.P);
    y[a] = out;
    if (!ok) atomicAdd(bad, 1ull);
}

// ---------------------------------------------------------------------------
// The hash alone.
// ---------------------------------------------------------------------------
template <int BLOCK>
__global__ void __launch_bounds__(BLOCK) k_hash(const ModConst mq, const ModConst mm, uint64_t count,
                                                const uint32_t *__restrict__ lab, uint32_t gid,
                                                const uint64_t *__restrict__ tau, uint32_t *__restrict__ out) {
    __shared__ uint32_t TT[kTableWords];
    stage_round_tables(TT, threadIdx.x, BLOCK);
    __syncthreads();
    const uint64_t a = static_cast<uint64_t>(blockIdx.x) * BLOCK + threadIdx.x;
    if (a >= count) return;
    uint32_t x[4] = {0, 0, 0, 0};
#pragma unroll
    for (int w = 0; w < kMaxW; ++w)
        if (w < static_cast<int>(mq.W)) x[w & 3] ^= lab[static_cast<uint64_t>(w) * count + a];
    uint32_t V[8];
    hash_fraction(TT, x[0], x[1], x[2], x[3], tau[a], gid, mm.m != 2, V);
#pragma unroll
    for (int w = 0; w < kMaxW; ++w)
        if (w < static_cast<int>(mm.W)) out[static_cast<uint64_t>(w) * count + a] = pad_word(V, w, mm);
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
namespace {

constexpr int kMaxDevices = 64;

// Per device: its compute units and the largest LDS allocation a block may
// request, read on the first call that runs on it (they do not change while
// the process runs).
struct DeviceInfo {
    int cus, max_lds;
};
std::mutex g_dev_mu;
DeviceInfo g_dev[kMaxDevices] = {};

int device_info(DeviceInfo *out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return REDASH_E_HIP;
    std::lock_guard<std::mutex> lock(g_dev_mu);
    DeviceInfo &d = g_dev[dev];
    if (d.cus <= 0) {
        int cus = 0, lds = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            return REDASH_E_HIP;
        if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
            return REDASH_E_HIP;
        d = DeviceInfo{cus, lds};
    }
    *out = d;
    return REDASH_OK;
}

// The plan of the parameters this host thread passed last, and its
// evaluator schedule once a call needed it: a layer evaluated call after call
// with the same parameters builds them once.  (redash_params has no padding:
// equal bytes are equal parameters; unused entries that differ only cost a
// rebuild.)
struct PlanCache {
    bool valid, has_eval;
    redash_params p;
    Plan P;
    EvalPlan E;
};
thread_local PlanCache t_plan;

int cached_plan(const redash_params *p, const Plan **out) {
    if (!p) return REDASH_E_NULL;
    PlanCache &c = t_plan;
    if (!c.valid || memcmp(&c.p, p, sizeof *p) != 0) {
        c.valid = false;
        const int rc = build_plan(p, &c.P);
        if (rc) return rc;
        c.p = *p;
        c.valid = true;
        c.has_eval = false;
    }
    *out = &c.P;
    return REDASH_OK;
}

// The evaluator schedule of P (the cached plan's, kept with it).
const EvalPlan &eval_plan(const Plan &P) {
    PlanCache &c = t_plan;
    if (&P != &c.P) {  // not reached: every entry point takes its plan from the cache
        static thread_local EvalPlan E;
        build_eval_plan(P, &E);
        return E;
    }
    if (!c.has_eval) {
        build_eval_plan(c.P, &c.E);
        c.has_eval = true;
    }
    return c.E;
}

// Threads per workgroup for n gadgets: the smallest multiple of 64 that keeps
// the grid within one round of two workgroups per CU (the LDS image allows two),
// at most `most`.  Small launches thus spread over every CU instead of filling
// a few with long-running waves; large ones use `most`.
int block_for(uint64_t n, int most, int *out) {
    DeviceInfo d;
    const int rc = device_info(&d);
    if (rc) return rc;
    const uint64_t slots = 2ull * static_cast<uint64_t>(d.cus);
    const uint64_t b = 64 * ((n + 64 * slots - 1) / (64 * slots));
    *out = b < 64 ? 64 : (b > static_cast<uint64_t>(most) ? most : static_cast<int>(b));
    return REDASH_OK;
}

// Largest LDS allocation a block may request on the current device.
int max_lds_bytes(size_t *out) {
    DeviceInfo d;
    const int rc = device_info(&d);
    if (rc) return rc;
    *out = static_cast<size_t>(d.max_lds);
    return REDASH_OK;
}

// Allows a kernel to use more than the default 64 KiB of dynamic LDS.
int allow_lds(const void *kernel, size_t bytes) {
    if (bytes <= 64 * 1024) return REDASH_OK;
    return hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes)) ==
                   hipSuccess
               ? REDASH_OK
               : REDASH_E_HIP;
}

unsigned grid_for(uint64_t n, int block) { return static_cast<unsigned>((n + block - 1) / block); }

int launched() {
    return hipGetLastError() == hipSuccess ? REDASH_OK : REDASH_E_HIP;
}

// Launches k_eval_split (it may use more than 64 KiB of LDS).
int launch_split_kernel(const Plan &P, uint32_t lds, const uint32_t *in, const uint32_t *tab, uint32_t *out,
                        uint32_t *work, const SplitLaunch &L, unsigned grid, int threads, hipStream_t stream) {
    const int rc = allow_lds(reinterpret_cast<const void *>(&k_eval_split<kEvalBlock>), lds);
    if (rc) return rc;
    hipLaunchKernelGGL(k_eval_split<kEvalBlock>, dim3(grid), dim3(threads), lds, stream, P, in, tab, out, work, L);
    return launched();
}

// Gadgets per workgroup of the split evaluator at full size: a multiple of 64
// with per * split <= kEvalBlock (768, 384, 192 and 64 for 1, 2, 4 and 12 waves).
constexpr uint32_t split_most(uint32_t split) { return kEvalBlock / split / 64 * 64; }

// k_eval_split over gadgets first .. first + count - 1 (of the plan's n), each
// group of 64 gadgets on `split` waves (12, 4 or 2).
int launch_split(uint32_t split, const Plan &P, uint32_t lds, const uint32_t *in, const uint32_t *tab, uint32_t *out,
                 uint32_t *work, uint64_t first, uint64_t count, hipStream_t stream) {
    int per = 0;
    const int rc = block_for(count, static_cast<int>(split_most(split)), &per);
    if (rc) return rc;
    const SplitLaunch L{static_cast<uint32_t>(first), grid_for(count, per), split, split};
    return launch_split_kernel(P, lds, in, tab, out, work, L, grid_for(count, per), per * static_cast<int>(split),
                               stream);
}

// The split evaluator for `count` gadgets that one round of two workgroups
// per CU holds with 64, 192 or 384 gadgets per workgroup (12, 4 or 2 waves
// per 64 gadgets); 0 when the count needs more than one such round.
uint32_t split_for(uint64_t count, uint64_t cus) {
    if (count <= 2 * cus * 64) return 12;
    if (count <= 2 * cus * kEvalBlock / 4) return 4;
    if (count <= 2 * cus * kEvalBlock / 2) return 2;
    return 0;
}

// Launches the evaluators for n gadgets.  A call that one round of two
// workgroups per CU holds when a gadget takes 12, 4 or 2 waves runs on
// k_eval_split with that split (runs of gates sharing a digit have at most
// k - 1 gates, 11 on the 12-prime base: with 12 waves one gate per wave and
// run).  A call a little above one full round of the 4- or 2-wave split
// (98,304 or 196,608 gadgets on 256 CUs, plus at most 64 gadgets per CU) runs
// that round and its rest as one launch, the rest's workgroups on 12 waves per
// 64 gadgets after the round's: they take the CUs the round frees first,
// instead of adding a wave to some SIMDs for the whole call.  A larger call
// runs on k_eval, one gadget per lane: whole rounds of two full workgroups per
// CU, and a rest that the 12-wave split holds in one round goes to it after
// them instead of running as a last round with few waves per SIMD, whose
// gadgets would take the latency of their gate chain (a larger rest costs
// k_eval no more than it would cost the split).
int launch_eval(const Plan &P, uint32_t lds, const uint32_t *in, const uint32_t *tab, uint32_t *out, uint32_t *work,
                hipStream_t stream) {
    DeviceInfo d;
    int rc = device_info(&d);
    if (rc) return rc;
    const uint64_t ncu = static_cast<uint64_t>(d.cus);
    for (const uint32_t split : {4u, 2u}) {
        const uint32_t per0 = split_most(split);
        const uint64_t full = 2 * ncu * per0;
        if (P.n > full && P.n - full <= ncu * 64) {
            const uint32_t nb0 = static_cast<uint32_t>(2 * ncu);
            const unsigned grid = nb0 + grid_for(P.n - full, 64);
            return launch_split_kernel(P, lds, in, tab, out, work, SplitLaunch{0, nb0, split, 12}, grid, kEvalBlock,
                                       stream);
        }
    }
    if (const uint32_t split = split_for(P.n, ncu))
        return launch_split(split, P, lds, in, tab, out, work, 0, P.n, stream);
    const uint64_t round = 2 * ncu * kLaneBlock;  // gadgets of one round, one per lane
    uint64_t bulk = P.n;
    const uint64_t rest = P.n % round;
    if (P.n > round && rest > 0 && rest <= 2 * ncu * 64) bulk = P.n - rest;
    if ((rc = allow_lds(reinterpret_cast<const void *>(&k_eval<kLaneBlock>), lds))) return rc;
    int block = 0;
    if ((rc = block_for(bulk, kLaneBlock, &block))) return rc;
    const EvalPlan &E = eval_plan(P);
    hipLaunchKernelGGL(k_eval<kLaneBlock>, dim3(grid_for(bulk, block)), dim3(block), lds, stream, E, in, tab, out,
                       work);
    if ((rc = launched())) return rc;
    if (bulk == P.n) return REDASH_OK;
    return launch_split(split_for(P.n - bulk, ncu), P, lds, in, tab, out, work, bulk, P.n - bulk, stream);
}


SeedKey seed_key(uint64_t seed) {
    RoundKeys rk = make_seed_round_keys(seed);
    SeedKey k;
    memcpy(k.w, rk.w, sizeof k.w);
    return k;
}

}  // namespace

}  // namespace redash

using namespace redash;

extern "C" {

int redash_plan(const redash_params *p, redash_sizes *out) {
    if (!p || !out) return REDASH_E_NULL;
    const Plan *PP = nullptr;
    int rc = cached_plan(p, &PP);
    if (rc) return rc;
    const Plan &P = *PP;
    out->label_words = P.n * P.total_words;
    uint64_t tw = 0;
    for (uint32_t g = 0; g < P.G; ++g) {
        const uint32_t d = P.gate[g];
        tw += P.n * (P.mod[gate_src(d)].m - 1) * P.mod[gate_dst(d)].W;
    }
    out->table_words = tw;
    out->offset_words = P.total_words;
    out->gates = P.G;
    out->work_words = P.n * P.work_words;
    return REDASH_OK;
}

}  // extern "C"

namespace {

template <bool GIVEN>
int garble_scale(const redash_params *p, uint32_t *d_offsets, const uint32_t *d_in_zero, uint32_t *d_in_zero_w,
                 uint32_t *d_out_zero, uint32_t *d_tables, uint32_t *d_work, hipStream_t stream) {
    const Plan *PP = nullptr;
    int rc = cached_plan(p, &PP);
    if (rc) return rc;
    const Plan &P = *PP;
    if (P.n >= (1ull << 30)) return REDASH_E_PARAM;  // 4 a must fit in 32 bits
    if (!d_offsets) return REDASH_E_NULL;
    if (P.n > 0 && (!d_in_zero || !d_out_zero || !d_tables || (P.work_words && !d_work))) return REDASH_E_NULL;
    const SeedKey key = seed_key(P.seed);
    hipLaunchKernelGGL(k_offsets, dim3(1), dim3(64), 0, stream, P, key, d_offsets);
    if ((rc = launched())) return rc;
    if (P.n == 0) return REDASH_OK;
    size_t max_lds = 0;
    if ((rc = max_lds_bytes(&max_lds))) return rc;
    const uint32_t lds = kEvalTableBase;  // the AES image and the round keys
    if (lds > max_lds) return REDASH_E_HIP;
    if ((rc = allow_lds(reinterpret_cast<const void *>(&k_garble<kGarbleBlock, GIVEN>), lds))) return rc;
    int block = 0;
    if ((rc = block_for(P.n, kGarbleBlock, &block))) return rc;
    hipLaunchKernelGGL((k_garble<kGarbleBlock, GIVEN>), dim3(grid_for(P.n, block)), dim3(block), lds, stream, P, key,
                       d_offsets, d_in_zero, d_in_zero_w, d_out_zero, d_tables, d_work);
    return launched();
}

}  // namespace

extern "C" {

int redash_garble_scale(const redash_params *p, uint32_t *d_offsets, uint32_t *d_in_zero, uint32_t *d_out_zero,
                        uint32_t *d_tables, uint32_t *d_work, hipStream_t stream) {
    return garble_scale<false>(p, d_offsets, d_in_zero, d_in_zero, d_out_zero, d_tables, d_work, stream);
}

int redash_garble_scale_given(const redash_params *p, uint32_t *d_offsets, const uint32_t *d_in_zero,
                              uint32_t *d_out_zero, uint32_t *d_tables, uint32_t *d_work, hipStream_t stream) {
    return garble_scale<true>(p, d_offsets, d_in_zero, nullptr, d_out_zero, d_tables, d_work, stream);
}

int redash_encode(const redash_params *p, const int64_t *d_x, const uint32_t *d_in_zero, const uint32_t *d_offsets,
                  uint32_t *d_in_labels, hipStream_t stream) {
    const Plan *PP = nullptr;
    int rc = cached_plan(p, &PP);
    if (rc) return rc;
    const Plan &P = *PP;
    if (!d_offsets) return REDASH_E_NULL;
    if (P.n == 0) return REDASH_OK;
    if (!d_x || !d_in_zero || !d_in_labels) return REDASH_E_NULL;
    hipLaunchKernelGGL(k_encode<256>, dim3(grid_for(P.n, 256)), dim3(256), 0, stream, P, d_x, d_in_zero, d_offsets,
                       d_in_labels);
    return launched();
}

int redash_eval_scale(const redash_params *p, const uint32_t *d_in_labels, const uint32_t *d_tables,
                      uint32_t *d_out_labels, uint32_t *d_work, hipStream_t stream) {
    const Plan *PP = nullptr;
    int rc = cached_plan(p, &PP);
    if (rc) return rc;
    const Plan &P = *PP;
    if (P.n >= (1ull << 30)) return REDASH_E_PARAM;  // 4 a must fit in 32 bits
    if (P.n == 0) return REDASH_OK;
    if (!d_in_labels || !d_tables || !d_out_labels || (P.work_words && !d_work)) return REDASH_E_NULL;
    size_t max_lds = 0;
    if ((rc = max_lds_bytes(&max_lds))) return rc;
    const uint32_t lds = eval_lds_bytes(P.ntab);
    if (lds > max_lds) return REDASH_E_HIP;
    return launch_eval(P, lds, d_in_labels, d_tables, d_out_labels, d_work, stream);
}

}  // extern "C"

namespace {

// Working storage of redash_eval_scale_noalloc.  In host code the name
// `scratch` only stands in for the device array: kernels get the device
// address that hipGetSymbolAddress returns on each GPU (every GPU holds its
// own copy at its own address).
__device__ __align__(256) uint32_t scratch[REDASH_NOALLOC_WORK_WORDS];

std::mutex g_scratch_mu;
uint32_t *g_scratch_ptr[kMaxDevices] = {};

// Device address of the current GPU's scratch array, looked up once per GPU
// (with that GPU current) on its first use.
int scratch_address(uint32_t **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return REDASH_E_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return REDASH_E_HIP;
        g_scratch_ptr[dev] = static_cast<uint32_t *>(ptr);
    }
    *out = g_scratch_ptr[dev];
    return REDASH_OK;
}

}  // namespace

extern "C" {

int redash_eval_scale_noalloc(const redash_params *p, const uint32_t *d_in_labels, const uint32_t *d_tables,
                              uint32_t *d_out_labels, hipStream_t stream) {
    const Plan *PP = nullptr;
    int rc = cached_plan(p, &PP);
    if (rc) return rc;
    const Plan &P = *PP;
    if (P.n >= (1ull << 30)) return REDASH_E_PARAM;  // 4 a must fit in 32 bits
    if (P.n * P.work_words > REDASH_NOALLOC_WORK_WORDS) return REDASH_E_SIZE;
    if (P.n == 0) return REDASH_OK;
    if (!d_in_labels || !d_tables || !d_out_labels) return REDASH_E_NULL;
    uint32_t *work = nullptr;
    if ((rc = scratch_address(&work))) return rc;
    size_t max_lds = 0;
    if ((rc = max_lds_bytes(&max_lds))) return rc;
    const uint32_t lds = eval_lds_bytes(P.ntab);
    if (lds > max_lds) return REDASH_E_HIP;
    return launch_eval(P, lds, d_in_labels, d_tables, d_out_labels, work, stream);
}

int redash_decode(const redash_params *p, const uint32_t *d_out_labels, const uint32_t *d_out_zero,
                  const uint32_t *d_offsets, int64_t *d_y, uint64_t *d_bad_count, hipStream_t stream) {
    const Plan *PP = nullptr;
    int rc = cached_plan(p, &PP);
    if (rc) return rc;
    const Plan &P = *PP;
    if (!d_offsets || !d_bad_count) return REDASH_E_NULL;
    if (P.n > 0 && (!d_out_labels || !d_out_zero || !d_y)) return REDASH_E_NULL;
    unsigned long long *bad = reinterpret_cast<unsigned long long *>(d_bad_count);
    hipLaunchKernelGGL(k_zero_u64, dim3(1), dim3(1), 0, stream, reinterpret_cast<uint64_t *>(bad));
    if ((rc = launched())) return rc;
    if (P.n == 0) return REDASH_OK;
    hipLaunchKernelGGL(k_decode<256>, dim3(grid_for(P.n, 256)), dim3(256), 0, stream, P, d_out_labels, d_out_zero,
                       d_offsets, d_y, bad);
    return launched();
}

int redash_hash_labels(uint32_t q, uint32_t m, uint64_t count, const uint32_t *d_labels, uint32_t gadget_id,
                       const uint64_t *d_tau, uint32_t *d_out, hipStream_t stream) {
    if (!modulus_ok(q) || !modulus_ok(m)) return REDASH_E_PARAM;
    if (count == 0) return REDASH_OK;
    if (!d_labels || !d_tau || !d_out) return REDASH_E_NULL;
    ModConst mq, mm;
    fill_mod_const(q, &mq);
    fill_mod_const(m, &mm);
    hipLaunchKernelGGL(k_hash<256>, dim3(grid_for(count, 256)), dim3(256), 0, stream, mq, mm, count, d_labels,
                       gadget_id, d_tau, d_out);
    return launched();
}

const char *redash_strerror(int code) {
    switch (code) {
        case REDASH_OK: return "ok";
        case REDASH_E_PARAM: return "invalid parameters";
        case REDASH_E_NULL: return "null pointer";
        case REDASH_E_HIP: return "HIP launch or runtime error";
        case REDASH_E_LABEL: return "output label failed the decode check";
        case REDASH_E_SIZE: return "the call needs more working storage than the fixed buffer holds";
        default: return "unknown error";
    }
}

}  // extern "C"
