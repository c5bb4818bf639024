// Garbled linear layers (dense, 2-D convolution) on LabelTensors for gfx950.
//
// With public integer weights, a linear layer is free label arithmetic
// (Sec. 2.3): Y_o = sum_j w_oj X_j mod m, residue by residue, and the garbler
// sets Z_o = sum_j w_oj Z_j - b_o R.  Every residue of every label is an
// independent convolution with the same weights, so the layer is one dense
// integer contraction per (modulus, packed word): int8 matrix cores do it.
//
//   * A weight acts through its residue mod m; reduced into the signed range
//     of Z_m it fits a signed byte for every m <= 255 (|w| <= 127).
//   * A residue v in [0, m) enters as the byte v - 128 (v XOR 0x80), so the
//     inputs need no per-modulus centring; the contraction then yields
//     sum w (v - 128) and adding 128 * sum_k w (the row sums, prepared with
//     the weights) restores sum w v exactly.
//   * The int32 accumulators are reduced mod m in the epilogue and the
//     residues are packed straight into PK32 words.
//
// One workgroup (4 waves) computes, for one modulus i, a tile of 64 output
// channels x XT output positions of one output row, packed word by packed
// word of the labels.  Wave q takes residue j0 + q of the word; its 64 x XT
// tile is 4 x (XT/16) MFMA 16x16x64 tiles.  Per channel chunk the weights (64
// channels x the chunk's K bytes; staged once per modulus when there is one
// chunk) and the four residues' input halos are staged in LDS; the output
// words are merged across the waves in LDS and stored coalesced.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "../../include/redash.h"
#include "plan.hpp"

namespace redash {

namespace {

constexpr int kLinBlock = 256;      // 4 waves
constexpr int kLinOTile = 64;       // output channels per workgroup
constexpr uint32_t kLinMaxLds = 160 * 1024;
constexpr uint32_t kLinMaxK = 16384;  // c_in kh kw: |sum w v| < 127 * 250 * 2^14 < 2^29
constexpr uint32_t kLinMaxTaps = 64;
constexpr uint32_t kLinTwoPerCu = 80 * 1024;  // LDS bytes that let two workgroups share a CU

struct LinMod {
    uint32_t m, b, g, W, glast;
    uint32_t woff;                // word offset of this modulus's block (in units of n)
    uint32_t divM, divS, div_fix; // floor(u / m) for every 32-bit u
    uint32_t off;                 // m ceil(2^29 / m): makes every sum non-negative
};

struct LinPlan {
    uint32_t k;
    uint32_t c_in, c_out, kh, kw, stride, pad;
    uint32_t in_rows, in_cols;    // input rows and columns of one image (dense: 1, batch)
    uint32_t rows, cols, nimg;    // output rows, columns, images (dense: 1, batch, 1)
    uint32_t sN, sC, sY, sX;      // input activation index = img sN + c sC + y sY + x sX
    uint32_t oN, oO, oY, oX;      // output activation index, likewise
    uint32_t xt, xtiles;          // output positions per tile, tiles per row
    uint32_t ck, kc, taps, ncc;   // channel chunk, K bytes per chunk (64-padded), kh kw, chunks
    uint32_t o_pad, ogroups;      // c_out rounded up to 64, its groups of 64
    uint32_t xw;                  // staged input columns per row
    uint32_t xw_magic;            // floor(e / xw) = umulhi(e, xw_magic) for every staged item index e
    uint32_t kw_magic;            // floor(t / kw) = umulhi(t, kw_magic) for every tap t < 64
    uint32_t lg_ck, lg_c16n;      // log2 ck, log2 (ck / 16)
    uint32_t swz_shift, swz_mask; // 16-byte chunk swizzle of a staged column (see k_linear)
    uint32_t ostride;             // words per output-channel row of the merged output words
    uint32_t astride;             // LDS bytes per staged weight row
    uint32_t lds_a, lds_b, lds_bytes;
    uint64_t n_in, n_out;         // activations
    uint64_t rowsum_off;          // byte offset of the row sums in the prepared buffer
    LinMod mod[kMaxK];
};

uint32_t gcd32(uint32_t a, uint32_t b) {
    while (b) {
        const uint32_t r = a % b;
        a = b;
        b = r;
    }
    return a;
}

uint32_t round_up(uint32_t v, uint32_t q) { return (v + q - 1) / q * q; }

// LDS bytes of one residue's input halo for a tile of xt positions.
uint32_t halo_bytes(const LinPlan &L, uint32_t xt, uint32_t *xw_out) {
    const uint32_t xw = (xt - 1) * L.stride + L.kw;
    if (xw_out) *xw_out = xw;
    return L.kh * xw * L.ck;
}

// LDS bytes of a workgroup with tiles of xt positions: the weights, then the
// four residues' halos (reused for the output words at the end).
uint32_t lds_for(const LinPlan &L, uint32_t xt) {
    const uint32_t hb = 4 * halo_bytes(L, xt, nullptr), ob = kLinOTile * (xt + 4) * 4;
    return L.lds_a + (hb > ob ? hb : ob);
}

int build_lin_plan(const redash_linear_params *p, LinPlan *L) {
    if (!p || !L) return REDASH_E_NULL;
    memset(L, 0, sizeof *L);
    if (p->k < 1 || p->k > static_cast<uint32_t>(kMaxK)) return REDASH_E_PARAM;
    unsigned __int128 P = 1;
    for (uint32_t i = 0; i < p->k; ++i) {
        const uint32_t m = p->moduli[i];
        if (!modulus_ok(m)) return REDASH_E_PARAM;
        if (i > 0 && m <= p->moduli[i - 1]) return REDASH_E_PARAM;
        for (uint32_t j = 0; j < i; ++j)
            if (gcd32(m, p->moduli[j]) != 1) return REDASH_E_PARAM;
        P *= m;
    }
    if (P >= (static_cast<unsigned __int128>(1) << 63)) return REDASH_E_PARAM;
    if (!p->batch || !p->c_in || !p->h_in || !p->w_in || !p->c_out || !p->kh || !p->kw || !p->stride)
        return REDASH_E_PARAM;
    if (p->pad >= p->kh || p->pad >= p->kw) return REDASH_E_PARAM;
    if (p->h_in + 2 * p->pad < p->kh || p->w_in + 2 * p->pad < p->kw) return REDASH_E_PARAM;
    const uint64_t taps = static_cast<uint64_t>(p->kh) * p->kw;
    if (taps > kLinMaxTaps || taps * p->c_in > kLinMaxK) return REDASH_E_PARAM;
    const uint32_t ho = (p->h_in + 2 * p->pad - p->kh) / p->stride + 1;
    const uint32_t wo = (p->w_in + 2 * p->pad - p->kw) / p->stride + 1;
    const uint64_t n_in = static_cast<uint64_t>(p->batch) * p->c_in * p->h_in * p->w_in;
    const uint64_t n_out = static_cast<uint64_t>(p->batch) * p->c_out * ho * wo;
    if (n_in >= (1ull << 30) || n_out >= (1ull << 30)) return REDASH_E_PARAM;

    L->k = p->k;
    L->c_in = p->c_in;
    L->c_out = p->c_out;
    L->kh = p->kh;
    L->kw = p->kw;
    L->stride = p->stride;
    L->pad = p->pad;
    L->n_in = n_in;
    L->n_out = n_out;
    const bool dense = p->h_in == 1 && p->w_in == 1 && p->kh == 1 && p->kw == 1;
    if (dense) {
        // (batch, c_in) row-major: the batch is the position axis of one image
        L->in_rows = 1;
        L->in_cols = p->batch;
        L->rows = 1;
        L->cols = p->batch;
        L->nimg = 1;
        L->sN = 0;
        L->sC = 1;
        L->sY = 0;
        L->sX = p->c_in;
        L->oN = 0;
        L->oO = 1;
        L->oY = 0;
        L->oX = p->c_out;
    } else {
        L->in_rows = p->h_in;
        L->in_cols = p->w_in;
        L->rows = ho;
        L->cols = wo;
        L->nimg = p->batch;
        L->sN = p->c_in * p->h_in * p->w_in;
        L->sC = p->h_in * p->w_in;
        L->sY = p->w_in;
        L->sX = 1;
        L->oN = p->c_out * ho * wo;
        L->oO = ho * wo;
        L->oY = wo;
        L->oX = 1;
    }
    L->taps = static_cast<uint32_t>(taps);
    // channel chunk: 64, or fewer when the channels are few or the taps many
    const uint32_t cin16 = round_up(p->c_in, 16);
    uint32_t ck = 64;
    while (ck > 16 && (ck / 2 >= cin16 || round_up(L->taps * ck, 64) > 1024)) ck /= 2;
    L->ck = ck;
    L->kc = round_up(L->taps * ck, 64);
    L->ncc = (p->c_in + ck - 1) / ck;
    L->o_pad = round_up(p->c_out, kLinOTile);
    L->ogroups = L->o_pad / kLinOTile;
    // A staged column holds ck channel bytes in ck/16 chunks of 16; chunk q of
    // column x sits at q ^ ((x >> swz_shift) & swz_mask), so that the 16-byte
    // reads of 8 consecutive columns fall in 8 distinct 4-bank groups.
    L->swz_mask = ck / 16 - 1;
    L->swz_shift = ck == 64 ? 1 : ck == 32 ? 2 : 3;
    // weight rows padded by 16 bytes: 8 consecutive rows in distinct bank groups
    L->astride = L->kc + 16;
    L->lds_a = kLinOTile * L->astride;
    // Tile width: 64, 32 or 16 positions, no wider than the row needs; the
    // widest that lets two workgroups share a CU, else the widest that fits.
    uint32_t need = 16;
    while (need < 64 && need < L->cols) need *= 2;
    L->xt = 0;
    for (uint32_t xt = need; xt >= 16 && !L->xt; xt /= 2)
        if (lds_for(*L, xt) <= kLinTwoPerCu) L->xt = xt;
    for (uint32_t xt = need; xt >= 16 && !L->xt; xt /= 2)
        if (lds_for(*L, xt) <= kLinMaxLds) L->xt = xt;
    if (!L->xt) return REDASH_E_PARAM;
    halo_bytes(*L, L->xt, &L->xw);
    // with M = ceil(2^32 / d), umulhi(e, M) = floor(e / d) whenever e d < 2^32
    // (the error e (M d - 2^32) / (d 2^32) < e / 2^32 stays below 1/d):
    // e < kh (ck/16) xw <= 64 * 4 * 133 for the items, t < 64 for the taps
    if (static_cast<uint64_t>(L->kh) * (ck / 16) * L->xw * L->xw >= (1ull << 32)) return REDASH_E_PARAM;
    L->xw_magic = static_cast<uint32_t>(((1ull << 32) + L->xw - 1) / L->xw);
    L->kw_magic = static_cast<uint32_t>(((1ull << 32) + p->kw - 1) / p->kw);
    L->lg_ck = ck == 64 ? 6 : ck == 32 ? 5 : 4;
    L->lg_c16n = L->lg_ck - 4;
    L->ostride = L->xt + 4;  // the four lane groups of an atomic OR fall 16 banks apart
    L->lds_bytes = lds_for(*L, L->xt);
    L->lds_b = L->lds_bytes - L->lds_a;
    L->xtiles = (L->cols + L->xt - 1) / L->xt;

    uint32_t woff = 0;
    for (uint32_t i = 0; i < p->k; ++i) {
        ModConst mc;
        fill_mod_const(p->moduli[i], &mc);
        LinMod &lm = L->mod[i];
        lm.m = mc.m;
        lm.b = mc.b;
        lm.g = mc.g;
        lm.W = mc.W;
        lm.glast = mc.glast;
        lm.woff = woff;
        woff += mc.W;
        // every u below 2^31 (see the epilogue): the multiply-shift needs no fix-up
        division_constants(mc.m, 1ull << 31, &lm.divM, &lm.divS, &lm.div_fix);
        lm.off = static_cast<uint32_t>(((1ull << 29) + mc.m - 1) / mc.m * mc.m);
    }
    L->rowsum_off = static_cast<uint64_t>(L->k) * L->ncc * L->o_pad * L->kc;
    return REDASH_OK;
}

uint64_t prepared_bytes(const LinPlan &L) { return L.rowsum_off + 4ull * L.k * L.o_pad; }

uint32_t total_words(const LinPlan &L) {
    uint32_t t = 0;
    for (uint32_t i = 0; i < L.k; ++i) t += L.mod[i].W;
    return t;
}

}  // namespace

// ---------------------------------------------------------------------------
// Weight preparation.
// Prepared layout: for modulus i, channel chunk cc, output channel o < o_pad:
// kc bytes, byte tap * ck + c_local = the weight w[o][cc ck + c_local][tap]
// reduced into the signed range of Z_m (0 beyond c_out, c_in or the taps).
// Then int32 row sums sum_{c, tap} of those values, [i][o].
// ---------------------------------------------------------------------------
__device__ __forceinline__ int32_t signed_residue(int32_t w, uint32_t m) {
    int32_t r = w % static_cast<int32_t>(m);
    if (r < 0) r += static_cast<int32_t>(m);
    return r >= static_cast<int32_t>((m + 1) / 2) ? r - static_cast<int32_t>(m) : r;
}

__global__ void __launch_bounds__(256) k_linear_prepare(const LinPlan L, const int32_t *__restrict__ wts,
                                                        uint8_t *__restrict__ prep) {
    const uint64_t total = L.rowsum_off;
    for (uint64_t e = static_cast<uint64_t>(blockIdx.x) * 256 + threadIdx.x; e < total;
         e += static_cast<uint64_t>(gridDim.x) * 256) {
        const uint32_t kb = static_cast<uint32_t>(e % L.kc);
        uint64_t r = e / L.kc;
        const uint32_t o = static_cast<uint32_t>(r % L.o_pad);
        r /= L.o_pad;
        const uint32_t cc = static_cast<uint32_t>(r % L.ncc);
        const uint32_t i = static_cast<uint32_t>(r / L.ncc);
        const uint32_t tap = kb / L.ck, c = cc * L.ck + kb % L.ck;
        int32_t v = 0;
        if (o < L.c_out && c < L.c_in && tap < L.taps)
            v = signed_residue(wts[(static_cast<uint64_t>(o) * L.c_in + c) * L.taps + tap], L.mod[i].m);
        prep[e] = static_cast<uint8_t>(static_cast<int8_t>(v));
    }
}

__global__ void __launch_bounds__(256) k_linear_rowsums(const LinPlan L, const int32_t *__restrict__ wts,
                                                        uint8_t *__restrict__ prep) {
    const uint32_t e = blockIdx.x * 256 + threadIdx.x;
    if (e >= L.k * L.o_pad) return;
    const uint32_t i = e / L.o_pad, o = e % L.o_pad;
    int32_t s = 0;
    if (o < L.c_out)
        for (uint32_t c = 0; c < L.c_in; ++c)
            for (uint32_t t = 0; t < L.taps; ++t)
                s += signed_residue(wts[(static_cast<uint64_t>(o) * L.c_in + c) * L.taps + t], L.mod[i].m);
    reinterpret_cast<int32_t *>(prep + L.rowsum_off)[e] = s;
}

// ---------------------------------------------------------------------------
// The layer kernel.
// ---------------------------------------------------------------------------
typedef int32_t v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t lin_div(uint32_t u, const LinMod &M) {
    const uint32_t t = __umulhi(u, M.divM);
    return M.div_fix ? (t + ((u - t) >> 1)) >> M.divS : t >> M.divS;
}

template <int NCB, bool GARBLE>
__global__ void __launch_bounds__(kLinBlock) k_linear(const LinPlan L, const uint32_t *__restrict__ in,
                                                      const uint8_t *__restrict__ prep,
                                                      const int64_t *__restrict__ bias,
                                                      const uint32_t *__restrict__ offsets,
                                                      uint32_t *__restrict__ out) {
    extern __shared__ __align__(16) uint8_t lds[];
    uint8_t *Al = lds;
    uint8_t *Bl = lds + L.lds_a;
    uint32_t *Ol = reinterpret_cast<uint32_t *>(lds + L.lds_a);  // after a word's last compute

    const uint32_t tid = threadIdx.x, lane = tid % 64;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid / 64);
    const uint32_t tile = blockIdx.x, i = blockIdx.y, og = blockIdx.z;
    const uint32_t xtile = tile % L.xtiles;
    const uint32_t row = (tile / L.xtiles) % L.rows;
    const uint32_t img = tile / (L.xtiles * L.rows);
    const LinMod M = L.mod[i];
    constexpr uint32_t XT = 16 * NCB;
    const uint32_t x0 = xtile * XT;
    const int32_t *rowsum = reinterpret_cast<const int32_t *>(prep + L.rowsum_off) + i * L.o_pad + og * kLinOTile;
    const uint32_t rowb = L.xw * L.ck;  // bytes per staged row of one residue
    const uint32_t halo = L.kh * rowb;  // bytes per residue
    const uint32_t mask = (1u << M.b) - 1u;
    const uint32_t ksteps = L.kc / 64;
    const uint32_t kg = 16 * (lane / 16);

    // output channel of element r of row block ob for this lane
    auto o_local = [&](int ob, int r) -> uint32_t { return ob * 16 + 4 * (lane / 16) + r; };
    // byte offset of channel byte c (a multiple of 4) of staged column x
    auto col_off = [&](uint32_t x, uint32_t c) -> uint32_t {
        return x * L.ck + ((((c >> 4) ^ (x >> L.swz_shift)) & L.swz_mask) << 4) + (c & 15u);
    };

    // 128 * row sum per lane row (restores sum w v from sum w (v - 128)), and
    // for the garbler -b_o mod m
    int32_t rs[4][4];
    uint32_t negb[4][4];
#pragma unroll
    for (int ob = 0; ob < 4; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            rs[ob][r] = M.m > 128 ? 128 * rowsum[o_local(ob, r)] : 0;
            negb[ob][r] = 0;
            if constexpr (GARBLE) {
                const uint32_t o = og * kLinOTile + o_local(ob, r);
                if (bias && o < L.c_out) {
                    int64_t bm = bias[o] % static_cast<int64_t>(M.m);
                    if (bm < 0) bm += M.m;
                    negb[ob][r] = (M.m - static_cast<uint32_t>(bm)) % M.m;
                }
            }
        }

    const int32_t ybase = static_cast<int32_t>(row * L.stride) - static_cast<int32_t>(L.pad);
    const int32_t xbase = static_cast<int32_t>(x0 * L.stride) - static_cast<int32_t>(L.pad);
    const uint32_t c16n = L.ck / 16;
    const uint32_t items = L.kh * c16n * L.xw;
    const bool full16 = L.c_in % 16 == 0;
    // residues of moduli up to 128 are valid signed bytes as they are; above
    // that they enter as v - 128 (v XOR 0x80), and 128 * rowsum restores sum w v
    const bool shifted = M.m > 128;
    const uint32_t flip = shifted ? 0x80808080u : 0u;
    bool a_staged = false;

    for (uint32_t w = 0; w < M.W; ++w) {
        const uint32_t g = (w + 1 == M.W) ? M.glast : M.g;
        const uint32_t *src = in + (static_cast<uint64_t>(M.woff) + w) * L.n_in;
        uint32_t part[4][NCB][4];
#pragma unroll
        for (int ob = 0; ob < 4; ++ob)
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                for (int r = 0; r < 4; ++r) part[ob][cb][r] = 0;

        for (uint32_t j0 = 0; j0 < g; j0 += 4) {
            v4i acc[4][NCB];
#pragma unroll
            for (int ob = 0; ob < 4; ++ob)
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) acc[ob][cb] = v4i{0, 0, 0, 0};
            for (uint32_t cc = 0; cc < L.ncc; ++cc) {
                __syncthreads();  // the previous fragments (and output words) have been read
                if (L.ncc > 1 || !a_staged) {
                    // weights of this chunk: 64 rows of kc bytes, 16 bytes per load
                    const uint8_t *ap = prep + ((static_cast<uint64_t>(i) * L.ncc + cc) * L.o_pad +
                                                og * kLinOTile) * L.kc;
                    const uint32_t per_row = L.kc / 16;
                    for (uint32_t e = tid; e < kLinOTile * per_row; e += kLinBlock) {
                        const uint32_t rr = e / per_row, q = e % per_row;
                        *reinterpret_cast<uint4 *>(Al + rr * L.astride + 16 * q) =
                            *reinterpret_cast<const uint4 *>(ap + static_cast<uint64_t>(rr) * L.kc + 16 * q);
                    }
                    a_staged = true;
                }
                // input halos of residues j0 .. j0+3; an item is (row r, 16 channels,
                // column xin): 16 loads in flight, then one 16-byte store per residue
                for (uint32_t e = tid; e < items; e += kLinBlock) {
                    const uint32_t q1 = __umulhi(e, L.xw_magic);  // e / xw
                    const uint32_t xin = e - q1 * L.xw;
                    const uint32_t c16 = q1 & (c16n - 1u);
                    const uint32_t r = q1 >> L.lg_c16n;
                    const int32_t y = ybase + static_cast<int32_t>(r), x = xbase + static_cast<int32_t>(xin);
                    const uint32_t c0 = cc * L.ck + 16 * c16;
                    const bool valid = y >= 0 && y < static_cast<int32_t>(L.in_rows) && x >= 0 &&
                                       x < static_cast<int32_t>(L.in_cols) && c0 < L.c_in;
                    uint32_t wd[16];
                    if (valid) {
                        const uint32_t *sp = src + (img * L.sN + static_cast<uint32_t>(y) * L.sY +
                                                    static_cast<uint32_t>(x) * L.sX + c0 * L.sC);
                        if (full16) {
#pragma unroll
                            for (int q = 0; q < 16; ++q) wd[q] = sp[q * L.sC];
                        } else {
                            // channels past c_in meet zero weights: read any valid one
                            const uint32_t last = L.c_in - 1 - c0;
#pragma unroll
                            for (int q = 0; q < 16; ++q) wd[q] = sp[(static_cast<uint32_t>(q) < last ? static_cast<uint32_t>(q) : last) * L.sC];
                        }
                    } else {
#pragma unroll
                        for (int q = 0; q < 16; ++q) wd[q] = 0;
                    }
                    const uint32_t dsto = r * rowb + xin * L.ck + (((c16 ^ (xin >> L.swz_shift)) & L.swz_mask) << 4);
#pragma unroll
                    for (int jq = 0; jq < 4; ++jq) {
                        if (j0 + jq < g) {
                            const uint32_t sh = M.b * (j0 + jq);
                            uint4 v;
                            uint32_t *vv = reinterpret_cast<uint32_t *>(&v);
#pragma unroll
                            for (int d = 0; d < 4; ++d) {
                                const uint32_t f0 = __builtin_amdgcn_ubfe(wd[4 * d], sh, M.b);
                                const uint32_t f1 = __builtin_amdgcn_ubfe(wd[4 * d + 1], sh, M.b);
                                const uint32_t f2 = __builtin_amdgcn_ubfe(wd[4 * d + 2], sh, M.b);
                                const uint32_t f3 = __builtin_amdgcn_ubfe(wd[4 * d + 3], sh, M.b);
                                vv[d] = (f0 | (f1 << 8) | (f2 << 16) | (f3 << 24)) ^ flip;
                            }
                            *reinterpret_cast<uint4 *>(Bl + jq * halo + dsto) = v;
                        }
                    }
                }
                __syncthreads();
                if (j0 + wave < g) {
                    const uint8_t *Bw = Bl + wave * halo;
                    for (uint32_t kk = 0; kk < ksteps; ++kk) {
                        v4i a[4];
#pragma unroll
                        for (int ob = 0; ob < 4; ++ob)
                            a[ob] = *reinterpret_cast<const v4i *>(Al + (ob * 16 + lane % 16) * L.astride + kk * 64 +
                                                                   kg);
                        const uint32_t kidx = kk * 64 + kg;
                        uint32_t tap = kidx >> L.lg_ck;
                        const uint32_t coff = kidx & (L.ck - 1u);
                        if (tap >= L.taps) tap = 0;  // K padding: the weights there are 0
                        const uint32_t dy = __umulhi(tap, L.kw_magic), dx = tap - dy * L.kw;
#pragma unroll
                        for (int cb = 0; cb < NCB; ++cb) {
                            const uint32_t xcol = (cb * 16 + lane % 16) * L.stride + dx;
                            const v4i bf = *reinterpret_cast<const v4i *>(Bw + dy * rowb + col_off(xcol, coff));
#pragma unroll
                            for (int ob = 0; ob < 4; ++ob)
                                acc[ob][cb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[ob], bf, acc[ob][cb], 0, 0, 0);
                        }
                    }
                }
            }
            // epilogue of residue j0 + wave: u = sum w v + m ceil(2^29/m) (+ (-b mod m) R_j)
            // lies in [0, 2^31); its residue mod m goes into the field
            if (j0 + wave < g) {
                const uint32_t j = j0 + wave, sh = M.b * j;
                uint32_t Rj = 0;
                if constexpr (GARBLE) Rj = (offsets[M.woff + w] >> sh) & mask;
#pragma unroll
                for (int ob = 0; ob < 4; ++ob)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        uint32_t extra = static_cast<uint32_t>(rs[ob][r]) + M.off;
                        if constexpr (GARBLE) extra += negb[ob][r] * Rj;
#pragma unroll
                        for (int cb = 0; cb < NCB; ++cb) {
                            const uint32_t u = static_cast<uint32_t>(acc[ob][cb][r]) + extra;
                            part[ob][cb][r] |= (u - lin_div(u, M) * M.m) << sh;
                        }
                    }
            }
        }
        // merge the waves' fields (disjoint bits) and store whole words
        __syncthreads();
        for (uint32_t e = tid; e < kLinOTile * L.ostride; e += kLinBlock) Ol[e] = 0;
        __syncthreads();
#pragma unroll
        for (int ob = 0; ob < 4; ++ob)
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (part[ob][cb][r])
                        atomicOr(&Ol[o_local(ob, r) * L.ostride + cb * 16 + lane % 16], part[ob][cb][r]);
        __syncthreads();
        uint32_t *dstp = out + (static_cast<uint64_t>(M.woff) + w) * L.n_out;
        for (uint32_t e = tid; e < kLinOTile * XT; e += kLinBlock) {
            const uint32_t ol = e / XT, xl = e % XT;
            const uint32_t o = og * kLinOTile + ol, x = x0 + xl;
            if (o < L.c_out && x < L.cols) dstp[img * L.oN + o * L.oO + row * L.oY + x * L.oX] = Ol[ol * L.ostride + xl];
        }
    }
}

namespace {

int lin_launched() { return hipGetLastError() == hipSuccess ? REDASH_OK : REDASH_E_HIP; }

int lin_allow_lds(const void *kernel, uint32_t bytes) {
    if (bytes <= 64 * 1024) return REDASH_OK;
    return hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes)) ==
                   hipSuccess
               ? REDASH_OK
               : REDASH_E_HIP;
}

template <int NCB, bool GARBLE>
int launch_linear_ncb(const LinPlan &L, const uint32_t *in, const uint8_t *prep, const int64_t *bias,
                      const uint32_t *offsets, uint32_t *out, hipStream_t stream) {
    int rc = lin_allow_lds(reinterpret_cast<const void *>(&k_linear<NCB, GARBLE>), L.lds_bytes);
    if (rc) return rc;
    const uint64_t tiles = static_cast<uint64_t>(L.nimg) * L.rows * L.xtiles;
    if (tiles >= (1ull << 31)) return REDASH_E_PARAM;
    hipLaunchKernelGGL((k_linear<NCB, GARBLE>), dim3(static_cast<uint32_t>(tiles), L.k, L.ogroups),
                       dim3(kLinBlock), L.lds_bytes, stream, L, in, prep, bias, offsets, out);
    return lin_launched();
}

template <bool GARBLE>
int launch_linear(const LinPlan &L, const uint32_t *in, const uint8_t *prep, const int64_t *bias,
                  const uint32_t *offsets, uint32_t *out, hipStream_t stream) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess) return REDASH_E_HIP;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) return REDASH_E_HIP;
    if (L.lds_bytes > static_cast<uint32_t>(v)) return REDASH_E_HIP;
    switch (L.xt) {
        case 64: return launch_linear_ncb<4, GARBLE>(L, in, prep, bias, offsets, out, stream);
        case 32: return launch_linear_ncb<2, GARBLE>(L, in, prep, bias, offsets, out, stream);
        default: return launch_linear_ncb<1, GARBLE>(L, in, prep, bias, offsets, out, stream);
    }
}

}  // namespace

}  // namespace redash

using namespace redash;

extern "C" {

int redash_linear_plan(const redash_linear_params *p, redash_linear_sizes *out) {
    if (!p || !out) return REDASH_E_NULL;
    LinPlan L;
    const int rc = build_lin_plan(p, &L);
    if (rc) return rc;
    const uint32_t tw = total_words(L);
    out->in_label_words = L.n_in * tw;
    out->out_label_words = L.n_out * tw;
    out->prepared_bytes = prepared_bytes(L);
    out->h_out = (p->h_in + 2 * p->pad - p->kh) / p->stride + 1;
    out->w_out = (p->w_in + 2 * p->pad - p->kw) / p->stride + 1;
    out->offset_words = tw;
    return REDASH_OK;
}

int redash_linear_prepare(const redash_linear_params *p, const int32_t *d_weights, uint8_t *d_prepared,
                          hipStream_t stream) {
    LinPlan L;
    const int rc = build_lin_plan(p, &L);
    if (rc) return rc;
    if (!d_weights || !d_prepared) return REDASH_E_NULL;
    const uint64_t blocks = (L.rowsum_off + 255) / 256;
    hipLaunchKernelGGL(k_linear_prepare, dim3(static_cast<uint32_t>(blocks < 65536 ? blocks : 65536)), dim3(256),
                       0, stream, L, d_weights, d_prepared);
    if (lin_launched()) return REDASH_E_HIP;
    hipLaunchKernelGGL(k_linear_rowsums, dim3((L.k * L.o_pad + 255) / 256), dim3(256), 0, stream, L, d_weights,
                       d_prepared);
    return lin_launched();
}

int redash_linear_eval(const redash_linear_params *p, const uint32_t *d_in_labels, const uint8_t *d_prepared,
                       uint32_t *d_out_labels, hipStream_t stream) {
    LinPlan L;
    const int rc = build_lin_plan(p, &L);
    if (rc) return rc;
    if (!d_in_labels || !d_prepared || !d_out_labels) return REDASH_E_NULL;
    return launch_linear<false>(L, d_in_labels, d_prepared, nullptr, nullptr, d_out_labels, stream);
}

int redash_linear_garble(const redash_linear_params *p, const uint32_t *d_in_zero, const uint8_t *d_prepared,
                         const int64_t *d_bias, const uint32_t *d_offsets, uint32_t *d_out_zero,
                         hipStream_t stream) {
    LinPlan L;
    const int rc = build_lin_plan(p, &L);
    if (rc) return rc;
    if (!d_in_zero || !d_prepared || !d_offsets || !d_out_zero) return REDASH_E_NULL;
    return launch_linear<true>(L, d_in_zero, d_prepared, d_bias, d_offsets, d_out_zero, stream);
}

}  // extern "C"
