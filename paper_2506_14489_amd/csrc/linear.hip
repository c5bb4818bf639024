// Garbled linear layers (dense, 2-D convolution) on LabelTensors for gfx950.
//
// With public integer weights, a linear layer is free label arithmetic
// (Sec. 2.3): Y_o = sum_j w_oj X_j mod m, residue by residue, and the garbler
// sets Z_o = sum_j w_oj Z_j - b_o R.  Every residue of every label is an
// independent convolution with the same weights, so the layer is one dense
// integer contraction per (modulus, residue): int8 matrix cores do it.
//
//   * A weight acts through its residue mod m; reduced into the signed range
//     of Z_m it fits a signed byte for every m <= 255 (|w| <= 127).
//   * A residue v < m <= 128 is a valid signed byte as it is; for m > 128 it
//     enters as v - 128 (v XOR 0x80), and adding 128 * sum_k w (the row sums,
//     prepared with the weights) restores sum w v exactly.
//
// Two kernels per call:
//   k_linear_unpack  reads the packed input labels once and writes every
//                    residue as a byte into residue planes in the caller's
//                    working buffer: plane (i, r) holds residue r of modulus
//                    i for every input position, channel-last with the zero
//                    padding already in place, so that a 16-byte load gives a
//                    matrix-core fragment of 16 channels (HBM-bound);
//   k_linear_gemm_w  (one channel chunk) per workgroup: one modulus and 64
//                    output channels, the weights staged in LDS once; each
//                    wave then takes its own row segment of XT (32 or 16)
//                    output positions, 4 x (XT/16) MFMA 16x16x64 tiles, and
//                    runs through every residue of the modulus with its own
//                    staged input halo, reducing the int32 sums mod m into
//                    PK32 fields and storing each packed word whole;
//   k_linear_gemm    (several channel chunks) per workgroup: one modulus, 64
//                    output channels and a row segment; wave q takes residue
//                    j0 + q of each packed word, the halos and the weights of
//                    each chunk staged by the workgroup, the residues of a
//                    word merged across the waves in LDS.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <type_traits>

#include "../../include/redash.h"
#include "plan.hpp"

namespace redash {

namespace {

constexpr int kLinBlock = 256;      // 4 waves
constexpr int kLinOTile = 64;       // output channels per workgroup
constexpr uint32_t kLinMaxLds = 160 * 1024;
constexpr uint32_t kLinMaxK = 16384;  // c_in kh kw (the epilogue bounds below)
constexpr uint32_t kLinMaxTaps = 64;
constexpr uint32_t kLinMaxPairs = 96;  // (modulus, packed word) pairs: sum of W <= 15 * 6
constexpr int kXcds = 8;               // MI355X: workgroups go round-robin to 8 XCDs

struct LinMod {
    uint32_t m, b, g, W, glast;
    uint32_t woff;     // word offset of this modulus's block (in units of n)
    // Residue planes: a plane byte holds f = 8 / bp residues of bp bits
    // (m <= 16: m = 2 eight of one bit, 3 and 4 four of two bits, 5..16 two
    // of four bits) or one residue byte (m > 16).  Plane pn(w, j) = w ppw +
    // j / f of this modulus holds field j mod f of residues j of packed word w.
    uint32_t pl_off;   // planes of the earlier moduli
    uint32_t bp, lgf;  // bits per field in a plane byte, log2 f
    uint32_t ppw;      // planes per full packed word: ceil(g / f)
    uint32_t rep;      // a bp-bit mask in every byte (f > 1)
    // floor(u / m) = umulhi(u, divM) >> divS for every u the epilogue sees
    uint32_t divM, divS;
    uint32_t off;      // a multiple of m above |sum w v|: keeps u >= 0
};

struct LinPlan {
    uint32_t k;
    uint32_t c_in, c_out, kh, kw, stride, pad;
    uint32_t in_rows, in_cols;    // input rows and columns of one image (dense: 1, batch)
    uint32_t rows, cols, nimg;    // output rows, columns, images (dense: 1, batch, 1)
    uint32_t sN, sC, sY, sX;      // input activation index = img sN + c sC + y sY + x sX
    uint32_t oN, oO, oY, oX;      // output activation index, likewise
    uint32_t hp, wp, cp;          // plane rows and columns (padded) and channels (ncc ck)
    uint32_t xt, xtiles;          // output positions per tile, tiles per row
    uint32_t ck, kc, taps, ncc;   // channel chunk, K bytes per chunk (64-padded), kh kw, chunks
    uint32_t lg_ck;
    uint32_t kw_magic;            // floor(t / kw) = (t kw_magic) >> 16 for every tap t < 64
    uint32_t o_pad, ogroups;      // c_out rounded up to 64, its groups of 64
    uint32_t astride;             // LDS bytes per staged weight row
    uint32_t ostride;             // words per output-channel row of the merged output words
    uint32_t xw, xstride;         // staged input columns of a tile; LDS bytes per staged column
    uint32_t wpair;               // staging: the two columns of an 8-lane write group lie wpair apart
    uint32_t halo;                // LDS bytes of one residue's staged input (kh xw xstride)
    uint32_t lds_a, lds_b, lds_o, lds_bytes;
    uint32_t npairs;
    uint32_t word_split;          // k_linear_gemm: one workgroup per packed word (else per modulus)
    uint32_t fold_c;              // column fold (see the plan): the layer's own c_in, else 0
    uint32_t fold_magic;          // floor(c / fold_c) = (c fold_magic) >> 16 for every c < 64
    uint32_t flat, tile_rows;     // k_linear_gemm over the flattened plane (see the plan); rows of tiles
    uint64_t n_in, n_out;         // activations
    uint64_t plane_bytes;         // nimg hp wp cp
    uint64_t rowsum_off;          // byte offset of the row sums in the prepared buffer
    uint32_t total_planes;        // residue planes over the base
    uint8_t pair_mod[kLinMaxPairs], pair_word[kLinMaxPairs];
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
    // Column fold: with few input channels the kw columns of a kernel row
    // become kw c_in channels of a kh x 1 kernel (plane byte (y, x, dx c_in +
    // c) holds input (y, x + dx, c)), so that a K slice carries kw c_in
    // weights instead of c_in and up to 16 - c_in zeros (the 7x7 stride-2
    // stem over 3 channels: 4 K steps of 64 instead of 13), where the staged
    // halo of a 16-position tile still fits (kh (15 stride + 1) 16-byte
    // pieces per channel chunk of 16, 32 or 64).  From here on c_in, kw and
    // taps are those of the folded layer.
    L->fold_c = 0;
    L->fold_magic = 0;
    const uint32_t cf = p->kw * p->c_in, ckf = cf <= 16 ? 16u : cf <= 32 ? 32u : 64u;
    if (!dense && p->kw > 1 && p->c_in < 16 && cf <= 64 &&
        p->kh * (15 * p->stride + 1) * (ckf / 16) <= 2 * kLinBlock) {
        L->fold_c = p->c_in;
        // ceil(2^16 / c_in): as for the taps below, exact for every c < 64
        L->fold_magic = ((1u << 16) + p->c_in - 1) / p->c_in;
        L->c_in = p->kw * p->c_in;
        L->kw = 1;
        L->taps = p->kh;
    }
    // channel chunk: 64, or fewer when the channels are few or the taps many
    const uint32_t cin16 = round_up(L->c_in, 16);
    uint32_t ck = 64;
    while (ck > 16 && (ck / 2 >= cin16 || round_up(L->taps * ck, 64) > 1024)) ck /= 2;
    L->ck = ck;
    L->lg_ck = ck == 64 ? 6 : ck == 32 ? 5 : 4;
    L->kc = round_up(L->taps * ck, 64);
    L->ncc = (L->c_in + ck - 1) / ck;
    L->cp = L->ncc * ck;
    L->hp = L->in_rows + 2 * p->pad;
    // folded: plane column x serves output column x / stride
    L->wp = L->fold_c ? (L->cols - 1) * p->stride + 1 : L->in_cols + 2 * p->pad;
    // M = ceil(2^16 / kw) <= 2^16: with e = M kw - 2^16 < kw, (t M) >> 16 =
    // floor(t/kw + t e / (kw 2^16)), and t e / 2^16 < 64 kw / 2^16 < 1 keeps
    // the error below 1/kw for every tap t < 64 and kw <= 64 (t M < 2^22: a
    // 24-bit multiply).  (2^32 / kw would not fit 32 bits for kw = 1.)
    L->kw_magic = ((1u << 16) + L->kw - 1) / L->kw;
    L->o_pad = round_up(p->c_out, kLinOTile);
    L->ogroups = L->o_pad / kLinOTile;
    // 16-byte LDS reads of 16 rows (or columns) at a stride of S bytes, four
    // 16-byte chunks each, run without bank conflicts on this LDS when
    // S / 16 = 2 mod 4 (measured: 96, 160, 224, 608 are conflict-free; 80,
    // 112, 128, 592 are not).  Weight rows: kc is a multiple of 64, so kc + 32.
    L->astride = L->kc + 32;
    L->lds_a = kLinOTile * L->astride;
    // Staged input: per residue kh rows of xw columns of ck channel bytes,
    // columns padded to xstride.  A fragment reads 16 columns conv-stride
    // apart: with 64-channel chunks the padding makes stride * xstride / 16
    // = 2 mod 4 where it can (odd strides: 96 bytes; strides 2 mod 4: 80).
    // 16-byte LDS writes go 8 lanes per cycle over 32 banks: the 8 lanes of
    // a write group take two columns wpair apart so that their 4 chunks each
    // fall in distinct bank groups (xstride / 16 = 6: 2 apart; 5: 4 apart).
    if (ck == 64) {
        L->xstride = (p->stride % 2 == 1) ? 96 : 80;
        L->wpair = L->xstride == 96 ? 2 : 4;
    } else {
        L->xstride = ck == 16 ? 16 : ck + 16;
        L->wpair = 1;
    }
    // tile width: 32 or 16 positions, no wider than the row needs (64 would
    // not fit the registers of two waves per SIMD), and at most 512 staged
    // 16-byte pieces per residue (two per thread)
    L->xt = 32;
    while (L->xt > 16 && L->xt / 2 >= L->cols) L->xt /= 2;
    auto pieces = [&](uint32_t xt) { return L->kh * ((xt - 1) * p->stride + L->kw) * (ck / 16); };
    if (L->xt == 32 && pieces(32) > 2 * kLinBlock) L->xt = 16;
    // a 3x3 kernel over several 64-channel chunks keeps the next chunk's
    // weights in registers, which only the 16-position tile has room for
    if (L->ncc > 1 && ck == 64 && p->kh == 3 && p->kw == 3) L->xt = 16;
    if (pieces(L->xt) > 2 * kLinBlock) return REDASH_E_PARAM;
    L->xw = (L->xt - 1) * p->stride + L->kw;
    L->halo = L->kh * L->xw * L->xstride;
    L->tile_rows = L->rows;
    // Flattened tiles for narrow rows (3x3, stride 1, several chunks, at
    // most 8 output columns): output q = y wp + x of the padded plane reads
    // q + dy wp + dx, so a tile of 16 consecutive q stages one run of
    // 16 + 2 wp + 2 plane positions and reads tap (dy, dx) at offset
    // dy wp + dx; outputs with x >= cols are dropped at the store.  A
    // 16-position tile over a 7-position row otherwise leaves 9 of 16
    // matrix columns idle.
    L->flat = 0;
    if (p->stride == 1 && L->kh == 3 && L->kw == 3 && ck == 64 && L->ncc > 1 && L->cols <= 8 && L->xt == 16) {
        L->flat = 1;
        L->xw = 16 + 2 * L->wp + 2;
        L->halo = L->xw * L->xstride;
        L->tile_rows = 1;
        if (L->xw * (ck / 16) > 2 * kLinBlock) return REDASH_E_PARAM;  // not reached: wp <= 10
    }
    L->ostride = L->xt + 4;  // the four lane groups of an atomic OR fall 16 banks apart
    L->lds_b = 4 * L->halo;
    // the merged output words overlay the staged inputs (used at the end of
    // a packed word, after every wave has read its fragments)
    L->lds_o = kLinOTile * L->ostride * 4;
    // then the accumulator seeds of the 64 output channels (base, -b mod m)
    L->lds_bytes = L->lds_a + (L->lds_b > L->lds_o ? L->lds_b : L->lds_o) + 2 * kLinOTile * 4;
    if (L->lds_bytes > kLinMaxLds) return REDASH_E_PARAM;
    L->xtiles = L->flat ? (L->rows * L->wp + 15) / 16 : (L->cols + L->xt - 1) / L->xt;
    L->plane_bytes = static_cast<uint64_t>(L->nimg) * L->hp * L->wp * L->cp;
    if (L->plane_bytes >= (1ull << 32)) return REDASH_E_PARAM;  // 32-bit offsets within a plane

    uint32_t woff = 0, pl_off = 0, np = 0;
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
        lm.pl_off = pl_off;
        lm.bp = mc.b == 1 ? 1u : mc.b == 2 ? 2u : mc.b <= 4 ? 4u : 8u;
        const uint32_t f = 8 / lm.bp;
        lm.lgf = f == 8 ? 3u : f == 4 ? 2u : f == 2 ? 1u : 0u;
        lm.ppw = (mc.g + f - 1) / f;
        lm.rep = f > 1 ? ((1u << lm.bp) - 1u) * 0x01010101u : 0xffffffffu;
        woff += mc.W;
        pl_off += (mc.W - 1) * lm.ppw + (mc.glast + f - 1) / f;
        // |sum w v| <= K floor(m/2) (m - 1) =: B (signed weights, residues v < m);
        // u = sum w v + off (+ (-b mod m) R_j, below m^2) lies in [0, 2B + m^2),
        // below 2^31 for K <= 16384, and u / m < 2^23 (a signed 24-bit product)
        const uint64_t K = static_cast<uint64_t>(L->taps) * L->c_in;
        const uint64_t B = K * (mc.m / 2) * (mc.m - 1);
        lm.off = static_cast<uint32_t>((B + mc.m - 1) / mc.m * mc.m);
        const uint64_t u_max = lm.off + B + static_cast<uint64_t>(mc.m) * mc.m;
        if (u_max >= (1ull << 31) || u_max / mc.m >= (1ull << 23)) return REDASH_E_PARAM;
        if (u_max * mc.m < (1ull << 32)) {
            lm.divM = static_cast<uint32_t>(((1ull << 32) + mc.m - 1) / mc.m);  // exact: u m < 2^32
            lm.divS = 0;
        } else {
            uint32_t fix = 0;
            division_constants(mc.m, 1ull << 31, &lm.divM, &lm.divS, &fix);
            if (fix) return REDASH_E_PARAM;  // not reached: below 2^31 the round-up method is exact
        }
        for (uint32_t w = 0; w < mc.W; ++w) {
            if (np >= kLinMaxPairs) return REDASH_E_PARAM;
            L->pair_mod[np] = static_cast<uint8_t>(i);
            L->pair_word[np] = static_cast<uint8_t>(w);
            ++np;
        }
    }
    L->npairs = np;
    // A workgroup per packed word rather than per modulus (both contraction
    // kernels) when the per-modulus grid is small: the small moduli, with the
    // most residues (128 for m = 2, 25 for 37 at 128-bit labels), would
    // otherwise set the launch's length; measured slower on large grids,
    // where the chip is full either way.
    const uint64_t tiles = static_cast<uint64_t>(L->nimg) * L->tile_rows * L->xtiles;
    const uint64_t grid_mod = (L->ncc > 1 ? tiles : (tiles + 3) / 4) * L->k * L->ogroups;  // 4 tiles per workgroup
    L->word_split = grid_mod < 2048 ? 1u : 0u;
    L->total_planes = pl_off;
    L->rowsum_off = static_cast<uint64_t>(L->k) * L->ncc * L->o_pad * L->kc;
    return REDASH_OK;
}

uint64_t prepared_bytes(const LinPlan &L) { return L.rowsum_off + 4ull * L.k * L.o_pad; }

uint64_t work_bytes(const LinPlan &L) { return static_cast<uint64_t>(L.total_planes) * L.plane_bytes; }

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
        if (o < L.c_out && c < L.c_in && tap < L.taps) {
            // folded: channel c = dx c_in' + c' of kernel row tap is weight
            // (o, c', tap, dx) of the layer's kh x kw kernel (kw = c_in / c_in')
            const uint32_t kw0 = L.fold_c ? L.c_in / L.fold_c : 1u;
            const uint64_t at = L.fold_c ? (static_cast<uint64_t>(o) * L.fold_c + c % L.fold_c) * (L.taps * kw0) +
                                               static_cast<uint64_t>(tap) * kw0 + c / L.fold_c
                                         : (static_cast<uint64_t>(o) * L.c_in + c) * L.taps + tap;
            v = signed_residue(wts[at], L.mod[i].m);
        }
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
// Residue planes.  Plane pl_off_i + pn(w, j) (see LinMod) holds plane_bytes
// bytes: position (img, yp, xp) of the zero-padded input at
// ((img hp + yp) wp + xp) cp, its cp channel bytes after it.  A byte holds f
// residues of a modulus m <= 16 in bp-bit fields, or one residue v (16 < m <=
// 128) or v XOR 0x80 (m > 128); padding holds the byte of v = 0, channels
// past c_in meet zero weights.
// ---------------------------------------------------------------------------

// A word at byte offset `off` (below 2^32) of a uniform base: the offset stays
// a 32-bit VGPR next to a scalar base address.
__device__ __forceinline__ uint32_t load_word(const uint32_t *base, uint32_t off) {
    asm("" : "+v"(off));
    return *reinterpret_cast<const uint32_t *>(reinterpret_cast<const char *>(base) + off);
}

typedef int32_t v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4i load16(const uint8_t *base, uint32_t off) {
    asm("" : "+v"(off));
    return *reinterpret_cast<const v4i *>(base + off);
}

// A workgroup takes 64 padded positions and one 64-channel chunk of a packed
// word.  Loads: thread (p, c16) = (tid % 64, tid / 64) reads 16 channel words
// of position p, so each load instruction reads 64 consecutive positions of
// one channel plane; the words go through LDS ([position][channel], rows
// padded to 68 words).  Stores: thread (p, c16) = (tid / 4, tid % 4) writes
// the 16-byte piece of position p, channels 16 c16.., of every residue of the
// word: consecutive threads write consecutive pieces.
__global__ void __launch_bounds__(256) k_linear_unpack(const LinPlan L, const uint32_t *__restrict__ in,
                                                       uint8_t *__restrict__ planes) {
    __shared__ __align__(16) uint32_t T[64 * 68];
    // workgroups go round-robin to the XCDs by linear index: remap so that
    // each XCD takes runs of RUN neighbouring position blocks, the 8 XCDs
    // working on 8 neighbouring runs, so that most lines that neighbouring
    // blocks share (input rows are not line-aligned) are fetched into one L2
    // (one contiguous range per XCD fetches the fewest lines but streams
    // from HBM more slowly: 0.73 ms against 0.51)
    const uint32_t nx = gridDim.x, ny = gridDim.y, nt = nx * ny * gridDim.z;
    const uint32_t lin = blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z);
    constexpr uint32_t RUN = 16;
    const uint32_t full = nt / (kXcds * RUN) * (kXcds * RUN);
    const uint32_t lg = lin < full ? lin / (kXcds * RUN) * (kXcds * RUN) + (lin % kXcds) * RUN + (lin / kXcds) % RUN : lin;
    const uint32_t bx = lg % nx, by = (lg / nx) % ny, bz = lg / (nx * ny);
    const uint32_t pair = by;
    const uint32_t i = L.pair_mod[pair], w = L.pair_word[pair];
    const LinMod M = L.mod[i];
    const uint32_t g = (w + 1 == M.W) ? M.glast : M.g;
    const uint32_t tid = threadIdx.x;
    const uint32_t npos = L.nimg * L.hp * L.wp;
    const uint32_t pp0 = bx * 64, cbase = 64 * bz;
    const uint32_t ngrp = (L.cp - cbase) / 16 < 4 ? (L.cp - cbase) / 16 : 4u;  // 16-channel groups of this chunk
    const uint32_t flip = M.m > 128 ? 0x80808080u : 0u;
    // position of (padded) index pp: inside the input, and the word offset there
    auto at = [&](uint32_t pp, bool &inside) -> uint32_t {
        const uint32_t xp = pp % L.wp, t = pp / L.wp;
        const uint32_t yp = t % L.hp, img = t / L.hp;
        const int32_t y = static_cast<int32_t>(yp) - static_cast<int32_t>(L.pad);
        const int32_t x = static_cast<int32_t>(xp) - static_cast<int32_t>(L.pad);
        inside = y >= 0 && y < static_cast<int32_t>(L.in_rows) && x >= 0 && x < static_cast<int32_t>(L.in_cols);
        return inside ? (img * L.sN + static_cast<uint32_t>(y) * L.sY + static_cast<uint32_t>(x) * L.sX) * 4u : 0u;
    };
    if (L.fold_c) {
        // folded layer: channel c = dx c_in' + c' of plane column xp is input
        // channel c' at padded column xp + dx; outside the input the word is
        // 0, whose fields are the residues of the padding value 0
        const uint32_t p = tid % 64, c16 = tid / 64, pp = pp0 + p;
        if (pp < npos && c16 < ngrp) {
            const uint32_t xp = pp % L.wp, t = pp / L.wp;
            const int32_t y = static_cast<int32_t>(t % L.hp) - static_cast<int32_t>(L.pad);
            const uint32_t img = t / L.hp;
            const uint32_t *src = in + (static_cast<uint64_t>(M.woff) + w) * L.n_in;
            v4i q4[4];
#pragma unroll
            for (int d = 0; d < 4; ++d)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t ch = cbase + 16 * c16 + static_cast<uint32_t>(4 * d + k);
                    const uint32_t dx = __umul24(ch, L.fold_magic) >> 16, c = ch - dx * L.fold_c;
                    const int32_t x = static_cast<int32_t>(xp + dx) - static_cast<int32_t>(L.pad);
                    const bool ok = ch < L.c_in && y >= 0 && y < static_cast<int32_t>(L.in_rows) && x >= 0 &&
                                    x < static_cast<int32_t>(L.in_cols);
                    const uint32_t a =
                        ok ? (img * L.sN + static_cast<uint32_t>(y) * L.sY + static_cast<uint32_t>(x) * L.sX + c * L.sC) * 4u
                           : 0u;
                    const uint32_t v = load_word(src, a);
                    q4[d][k] = static_cast<int32_t>(ok ? v : 0u);
                }
#pragma unroll
            for (int d = 0; d < 4; ++d) *reinterpret_cast<v4i *>(&T[p * 68 + 16 * c16 + 4 * d]) = q4[d];
        }
    } else {
        const uint32_t p = tid % 64, c16 = tid / 64, pp = pp0 + p;
        if (pp < npos && c16 < ngrp) {
            bool inside = false;
            const uint32_t a0 = at(pp, inside);
            const uint32_t *src = in + (static_cast<uint64_t>(M.woff) + w) * L.n_in;
            const uint32_t step = L.sC * 4u;
            const uint32_t c0 = cbase + 16 * c16;
            // padding reads position (0, 0) channel 0, channels past c_in the
            // last channel: masked below
            const bool live = inside && c0 < L.c_in;
            const uint32_t cb = live ? c0 : 0u, last = live ? L.c_in - 1 - c0 : 0u;
            v4i q4[4];
#pragma unroll
            for (int d = 0; d < 4; ++d)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t q = static_cast<uint32_t>(4 * d + k);
                    q4[d][k] = static_cast<int32_t>(load_word(src, a0 + (cb + (q < last ? q : last)) * step));
                }
#pragma unroll
            for (int d = 0; d < 4; ++d) *reinterpret_cast<v4i *>(&T[p * 68 + 16 * c16 + 4 * d]) = q4[d];
        }
    }
    __syncthreads();
    const uint32_t p = tid / 4, c16 = tid % 4, pp = pp0 + p;
    if (pp >= npos || c16 >= ngrp) return;  // no barrier follows
    bool inside = false;
    (void)at(pp, inside);
    inside = inside || L.fold_c;  // folded: padding was read as 0 words
    const uint32_t c0 = cbase + 16 * c16;
    uint32_t wd[16];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const v4i v = *reinterpret_cast<const v4i *>(&T[p * 68 + 16 * c16 + 4 * d]);
#pragma unroll
        for (int k = 0; k < 4; ++k) wd[4 * d + k] = static_cast<uint32_t>(v[k]);
    }
    const uint32_t nlive = !inside || c0 >= L.c_in ? 0u : (L.c_in - c0 < 16 ? L.c_in - c0 : 16u);  // live channels
    uint8_t *dst = planes + static_cast<uint64_t>(M.pl_off + w * M.ppw) * L.plane_bytes + static_cast<uint64_t>(pp) * L.cp + c0;
    const uint32_t nplanes = (g + (1u << M.lgf) - 1) >> M.lgf;
    for (uint32_t h = 0; h < nplanes; ++h) {
        v4i v;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            uint32_t y = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t q = static_cast<uint32_t>(4 * d + k);
                uint32_t x;
                if (M.lgf == 0) {
                    x = __builtin_amdgcn_ubfe(wd[q], M.b * h, M.b);  // one residue
                } else if (M.bp == M.b) {
                    x = __builtin_amdgcn_ubfe(wd[q], 8 * h, 8);  // f adjacent fields, as in the word
                } else {
                    // b = 3: residues 2h and 2h + 1 into 4-bit fields
                    x = __builtin_amdgcn_ubfe(wd[q], 6 * h, 3) | (__builtin_amdgcn_ubfe(wd[q], 6 * h + 3, 3) << 4);
                }
                y |= (q < nlive ? x : 0u) << (8 * k);
            }
            v[d] = static_cast<int32_t>(y ^ flip);
        }
        *reinterpret_cast<v4i *>(dst + static_cast<uint64_t>(h) * L.plane_bytes) = v;
    }
}

// Residue j's values from a 16-byte piece of its plane: field j mod f of
// every byte (f > 1), or the bytes themselves.
__device__ __forceinline__ v4i plane_field(const v4i &v, const LinMod &M, uint32_t j) {
    if (M.lgf == 0) return v;
    const uint32_t sh = M.bp * (j & ((1u << M.lgf) - 1u));
    v4i r;
#pragma unroll
    for (int d = 0; d < 4; ++d) r[d] = static_cast<int32_t>((static_cast<uint32_t>(v[d]) >> sh) & M.rep);
    return r;
}

// ---------------------------------------------------------------------------
// The contraction.
// ---------------------------------------------------------------------------
// K33 (> 0): a 3x3 kernel with 64-channel chunks (taps = K steps, kc = 576)
// and K33 bytes per staged column, the K loop unrolled with every fragment
// offset known but the row stride; 0: any kernel.
template <int NCB, bool GARBLE, int K33>
__global__ void __launch_bounds__(kLinBlock) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_linear_gemm(const LinPlan L, const uint8_t *__restrict__ planes, const uint8_t *__restrict__ prep,
              const int64_t *__restrict__ bias, const uint32_t *__restrict__ offsets, uint32_t *__restrict__ out) {
    extern __shared__ __align__(16) uint8_t lds[];
    uint8_t *Al = lds;
    uint8_t *Bl = lds + L.lds_a;
    uint32_t *Ol = reinterpret_cast<uint32_t *>(lds + L.lds_a);  // overlays Bl

    const uint32_t tid = threadIdx.x, lane = tid % 64;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid / 64);
    // consecutive tiles (neighbouring output rows, which share input rows) on
    // one XCD, whose L2 then serves the shared plane rows
    const uint32_t nb = gridDim.x, full = nb / kXcds * kXcds;
    const uint32_t tile = blockIdx.x < full ? (blockIdx.x % kXcds) * (nb / kXcds) + blockIdx.x / kXcds : blockIdx.x;
    // one packed word (pair table entry blockIdx.z, the output channel group
    // blockIdx.y: the words of the small moduli, with the most residues, are
    // dispatched first for every group) or every word of modulus blockIdx.y
    const uint32_t i = L.word_split ? L.pair_mod[blockIdx.z] : blockIdx.y;
    const uint32_t og = L.word_split ? blockIdx.y : blockIdx.z;
    const uint32_t xtile = tile % L.xtiles;
    const uint32_t row = (tile / L.xtiles) % L.tile_rows;
    const uint32_t img = tile / (L.xtiles * L.tile_rows);
    const LinMod M = L.mod[i];
    const uint32_t w_lo = L.word_split ? L.pair_word[blockIdx.z] : 0u;
    const uint32_t w_hi = L.word_split ? w_lo + 1 : M.W;
    constexpr uint32_t XT = 16 * NCB;
    const uint32_t x0 = xtile * XT;
    const int32_t *rowsum = reinterpret_cast<const int32_t *>(prep + L.rowsum_off) + i * L.o_pad + og * kLinOTile;
    const uint32_t ksteps = L.kc / 64;
    const uint32_t kg = 16 * (lane / 16);
    // staged bytes between kernel rows: a row of the halo, or wp positions of the flattened run
    const uint32_t rowb = (L.flat ? L.wp : L.xw) * L.xstride;

    // output channel of element r of row block ob for this lane
    auto o_local = [&](int ob, int r) -> uint32_t { return ob * 16 + 4 * (lane / 16) + r; };

    // The accumulators start at base = 128 rowsum (m > 128) + off (+ (-b mod
    // m) R_j for the garbler) and end at u = sum w v + off (+ ...) in
    // [0, 2^31) with u / m < 2^23.  The 64 output channels' base and -b mod m
    // sit in LDS after the staging area (read at each residue's first chunk).
    uint32_t *sbase = reinterpret_cast<uint32_t *>(lds + L.lds_bytes - 2 * kLinOTile * 4);
    uint32_t *snegb = sbase + kLinOTile;
    if (tid < kLinOTile) {
        const bool shifted = M.m > 128;
        sbase[tid] = (shifted ? static_cast<uint32_t>(128 * rowsum[tid]) : 0u) + M.off;
        uint32_t nb = 0;
        if constexpr (GARBLE) {
            const uint32_t o = og * kLinOTile + tid;
            if (bias && o < L.c_out) {
                int64_t bm = bias[o] % static_cast<int64_t>(M.m);
                if (bm < 0) bm += M.m;
                nb = (M.m - static_cast<uint32_t>(bm)) % M.m;
            }
        }
        snegb[tid] = nb;
    }
    __syncthreads();

    // This thread's (at most two) staged pieces: piece e = tid + 256 t of a
    // residue's halo is (row dy, column xin, 16 channels c16); its plane
    // offset (the column clamped into the padded row: the columns past the
    // row feed outputs that are dropped) and its LDS offset.
    const uint32_t c16n = L.ck / 16;
    const uint32_t pieces = (L.flat ? 1u : L.kh) * L.xw * c16n;
    uint32_t poff[2], loff[2];
    bool pval[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const uint32_t e = tid + t * kLinBlock;
        pval[t] = e < pieces;
        const uint32_t ee = pval[t] ? e : 0u;
        const uint32_t c16 = ee % c16n, dy = ee / (c16n * L.xw);
        // column of this piece: within each full group of 2 wpair columns,
        // write slot j takes column j / 2 + (j % 2) wpair (a bijection)
        uint32_t xin = (ee / c16n) % L.xw;
        const uint32_t grp = 2 * L.wpair, gb = xin - xin % grp;
        if (gb + grp <= L.xw) xin = gb + (xin - gb) / 2 + ((xin - gb) % 2) * L.wpair;
        uint32_t xp = x0 * L.stride + xin;
        const uint32_t xlim = L.flat ? L.hp * L.wp : L.wp;  // flattened: the image's last position
        xp = xp < xlim ? xp : xlim - 1;
        poff[t] = ((img * L.hp + row * L.stride + dy) * L.wp + xp) * L.cp + 16 * c16;
        loff[t] = dy * rowb + xin * L.xstride + 16 * c16;
    }
    // fragment columns of this lane in the staged rows (tile column cb)
    uint32_t colb[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) colb[cb] = (cb * 16 + lane % 16) * L.stride * L.xstride;

    // Stages (w, j0, cc) in order: packed word, group of four residues,
    // channel chunk.  The pieces of the next stage are loaded into registers
    // while the current stage computes.
    struct Stage {
        uint32_t w, j0, cc;
    };
    auto g_of = [&](uint32_t w) { return (w + 1 == M.W) ? M.glast : M.g; };
    auto advance = [&](Stage &st) {
        if (++st.cc == L.ncc) {
            st.cc = 0;
            st.j0 += 4;
            if (st.j0 >= g_of(st.w)) {
                st.j0 = 0;
                ++st.w;
            }
        }
    };
    auto load_stage = [&](v4i (&pf)[2][4], const Stage &st) {
        const uint32_t g = g_of(st.w);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t j = st.j0 + q < g ? st.j0 + q : 0u;
            const uint8_t *plane =
                planes + static_cast<uint64_t>(M.pl_off + st.w * M.ppw + (j >> M.lgf)) * L.plane_bytes;
#pragma unroll
            for (int t = 0; t < 2; ++t) pf[t][q] = load16(plane, pval[t] ? poff[t] + st.cc * L.ck : 0u);
        }
    };

    uint32_t part[4][NCB][4];
    v4i acc[4][NCB];
    bool a_staged = false;
    Stage cur{w_lo, 0, 0}, ahead{w_lo, 0, 0};
    v4i pfA[2][4];
    load_stage(pfA, ahead);
    advance(ahead);
    // 3x3 kernels on 64-channel chunks (kc = 576: 64 rows of 36 16-byte
    // pieces, 9 per thread): the next chunk's weights are loaded into
    // registers while the current stage computes, as the input pieces are
    constexpr bool kWpf = K33 > 0 && NCB == 1;  // with 32-position tiles the registers do not suffice
    constexpr int kWq = kWpf ? 9 : 1;
    v4i wf[kWq];
    auto load_weights = [&](uint32_t cc) {
        const uint8_t *ap = prep + ((static_cast<uint64_t>(i) * L.ncc + cc) * L.o_pad + og * kLinOTile) * L.kc;
#pragma unroll
        for (int q = 0; q < kWq; ++q) {
            const uint32_t e = tid + kLinBlock * q, rr = e / 36, p = e % 36;
            wf[q] = *reinterpret_cast<const v4i *>(ap + static_cast<uint64_t>(rr) * L.kc + 16 * p);
        }
    };
    if constexpr (kWpf) load_weights(0);

    // One stage with the pieces in pf; returns false after the last stage.
    auto stage = [&](v4i (&pf)[2][4]) -> bool {
        const uint32_t w = cur.w, j0 = cur.j0, cc = cur.cc;
        const uint32_t g = g_of(w);
        const uint32_t j = j0 + wave;  // this wave's residue
        if (j0 == 0 && cc == 0) {
#pragma unroll
            for (int ob = 0; ob < 4; ++ob)
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                    for (int r = 0; r < 4; ++r) part[ob][cb][r] = 0;
        }
        if (cc == 0) {
            uint32_t Rj = 0;
            if constexpr (GARBLE) Rj = (offsets[M.woff + w] >> (M.b * j)) & ((1u << M.b) - 1u);
#pragma unroll
            for (int ob = 0; ob < 4; ++ob)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int32_t b0 = static_cast<int32_t>(sbase[o_local(ob, r)] + snegb[o_local(ob, r)] * Rj);
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb) acc[ob][cb][r] = b0;
                }
        }
        __syncthreads();  // the previous stage's fragments have been read
        if (L.ncc > 1 || !a_staged) {
            if constexpr (kWpf) {
                // weights of chunk cc from the registers, then the next chunk's
#pragma unroll
                for (int q = 0; q < kWq; ++q) {
                    const uint32_t e = tid + kLinBlock * q, rr = e / 36, p = e % 36;
                    *reinterpret_cast<v4i *>(Al + rr * L.astride + 16 * p) = wf[q];
                }
                if (L.ncc > 1) load_weights(cc + 1 < L.ncc ? cc + 1 : 0u);
            } else {
                // weights of chunk cc: 64 rows of kc bytes, 16 bytes per load
                const uint8_t *ap =
                    prep + ((static_cast<uint64_t>(i) * L.ncc + cc) * L.o_pad + og * kLinOTile) * L.kc;
                const uint32_t per_row = L.kc / 16;
                for (uint32_t e = tid; e < kLinOTile * per_row; e += kLinBlock) {
                    const uint32_t rr = e / per_row, q = e % per_row;
                    *reinterpret_cast<uint4 *>(Al + rr * L.astride + 16 * q) =
                        *reinterpret_cast<const uint4 *>(ap + static_cast<uint64_t>(rr) * L.kc + 16 * q);
                }
            }
            a_staged = true;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (j0 + q < g) {
#pragma unroll
                for (int t = 0; t < 2; ++t)
                    if (pval[t]) *reinterpret_cast<v4i *>(Bl + q * L.halo + loff[t]) = plane_field(pf[t][q], M, j0 + q);
            }
        // pf is free: the next stage
        if (ahead.w < w_hi) load_stage(pf, ahead);
        advance(ahead);
        __syncthreads();
        if (j < g) {
            const uint8_t *Bw = Bl + wave * L.halo;
            if constexpr (K33 > 0) {
                // K step t is tap t = 3 dy + dx, the lane's 16 channels at kg
                const uint8_t *Ar = Al + (lane % 16) * (576 + 32) + kg;
#pragma unroll
                for (int dy = 0; dy < 3; ++dy) {
                    const uint8_t *Br = Bw + dy * rowb + kg;
#pragma unroll
                    for (int dx = 0; dx < 3; ++dx) {
                        const int kk = 3 * dy + dx;
                        v4i a[4];
#pragma unroll
                        for (int ob = 0; ob < 4; ++ob)
                            a[ob] = *reinterpret_cast<const v4i *>(Ar + ob * 16 * (576 + 32) + kk * 64);
#pragma unroll
                        for (int cb = 0; cb < NCB; ++cb) {
                            const v4i bf = *reinterpret_cast<const v4i *>(Br + colb[cb] + dx * K33);
#pragma unroll
                            for (int ob = 0; ob < 4; ++ob)
                                acc[ob][cb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[ob], bf, acc[ob][cb], 0, 0, 0);
                        }
                    }
                }
            } else {
                for (uint32_t kk = 0; kk < ksteps; ++kk) {
                    v4i a[4];
#pragma unroll
                    for (int ob = 0; ob < 4; ++ob)
                        a[ob] = *reinterpret_cast<const v4i *>(Al + (ob * 16 + lane % 16) * L.astride + kk * 64 + kg);
                    const uint32_t kidx = kk * 64 + kg;
                    uint32_t tap = kidx >> L.lg_ck;
                    if (tap >= L.taps) tap = 0;  // K padding: the weights there are 0
                    const uint32_t dy = __umul24(tap, L.kw_magic) >> 16, dx = tap - dy * L.kw;
                    const uint32_t boff = dy * rowb + dx * L.xstride + (kidx & (L.ck - 1u));
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb) {
                        const v4i bf = *reinterpret_cast<const v4i *>(Bw + boff + colb[cb]);
#pragma unroll
                        for (int ob = 0; ob < 4; ++ob)
                            acc[ob][cb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[ob], bf, acc[ob][cb], 0, 0, 0);
                    }
                }
            }
        }
        if (cc + 1 == L.ncc && j < g) {
            // epilogue of residue j: the residue of u mod m goes into the field
            const uint32_t sh = M.b * j;
            auto epilogue = [&](auto shifts) {
#pragma unroll
                for (int ob = 0; ob < 4; ++ob)
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const uint32_t u = static_cast<uint32_t>(acc[ob][cb][r]);
                            uint32_t q = __umulhi(u, M.divM);  // < 2^23
                            if constexpr (decltype(shifts)::value) q >>= M.divS;
                            const uint32_t res =
                                static_cast<uint32_t>(__mul24(static_cast<int32_t>(q), -static_cast<int32_t>(M.m))) + u;
                            part[ob][cb][r] |= res << sh;
                        }
            };
            if (M.divS == 0)
                epilogue(std::integral_constant<bool, false>{});
            else
                epilogue(std::integral_constant<bool, true>{});
        }
        advance(cur);
        if (cur.w != w) {
            // word w complete: merge the waves' fields (disjoint bits), store
            // whole words.  Ol overlays the staged inputs: every wave must be
            // done with its fragments first.
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
                const uint32_t o = og * kLinOTile + ol;
                uint32_t y = row, x = x0 + xl;
                if (L.flat) {
                    y = x / L.wp;
                    x -= y * L.wp;
                }
                if (o < L.c_out && x < L.cols && y < L.rows)
                    dstp[img * L.oN + o * L.oO + y * L.oY + x * L.oX] = Ol[ol * L.ostride + xl];
            }
        }
        return cur.w < w_hi;
    };
    while (stage(pfA)) {
    }
}

// ---------------------------------------------------------------------------
// The contraction for one channel chunk (ncc = 1), with independent waves.
// A workgroup stages the weights of its modulus and 64 output channels once;
// then each wave takes its own tile (one output row segment of XT positions,
// the 64 channels), stages its own input halo and runs through every residue
// of every packed word of the modulus in turn: MFMA over the halo, the next
// residue's halo written over it (LDS operations of a wave complete in
// order), the one after loaded into registers, the epilogue, and each packed
// word stored whole when its last residue is done.  No barrier after the
// weights are staged.
// ---------------------------------------------------------------------------
constexpr int kWavePieces = 8;  // staged 16-byte pieces per lane (a halo has at most 512)

// PL: staged pieces per lane (a 3x3 halo of 64-channel columns has at most 7 x 64)
template <int NCB, bool GARBLE, int K33, int PL>
__global__ void __launch_bounds__(kLinBlock) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_linear_gemm_w(const LinPlan L, const uint8_t *__restrict__ planes, const uint8_t *__restrict__ prep,
                const int64_t *__restrict__ bias, const uint32_t *__restrict__ offsets, uint32_t *__restrict__ out) {
    extern __shared__ __align__(16) uint8_t lds[];
    uint8_t *Al = lds;
    const uint32_t tid = threadIdx.x, lane = tid % 64;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid / 64);
    uint8_t *Bw = lds + L.lds_a + wave * L.halo;
    // accumulator seeds per output channel: 128 rowsum (m > 128) + off, and
    // for the garbler (-b mod m), to be multiplied by R_j
    int32_t *seed = reinterpret_cast<int32_t *>(lds + L.lds_a + 4 * L.halo);
    int32_t *negb = seed + kLinOTile;
    // one packed word (pair table entry blockIdx.z, output channel group
    // blockIdx.y) or every word of modulus blockIdx.y, as in k_linear_gemm
    const uint32_t i = L.word_split ? L.pair_mod[blockIdx.z] : blockIdx.y;
    const uint32_t og = L.word_split ? blockIdx.y : blockIdx.z;
    const LinMod M = L.mod[i];
    const uint32_t w_lo = L.word_split ? L.pair_word[blockIdx.z] : 0u;
    const uint32_t w_hi = L.word_split ? w_lo + 1 : M.W;
    if (tid < kLinOTile) {
        const int32_t *rs = reinterpret_cast<const int32_t *>(prep + L.rowsum_off) + i * L.o_pad + og * kLinOTile;
        seed[tid] = static_cast<int32_t>((M.m > 128 ? static_cast<uint32_t>(128 * rs[tid]) : 0u) + M.off);
        uint32_t nb = 0;
        if constexpr (GARBLE) {
            const uint32_t o = og * kLinOTile + tid;
            if (bias && o < L.c_out) {
                int64_t bm = bias[o] % static_cast<int64_t>(M.m);
                if (bm < 0) bm += M.m;
                nb = (M.m - static_cast<uint32_t>(bm)) % M.m;
            }
        }
        negb[tid] = static_cast<int32_t>(nb);
    }

    // weights of the one chunk: 64 rows of kc bytes
    {
        const uint8_t *ap = prep + (static_cast<uint64_t>(i) * L.o_pad + og * kLinOTile) * L.kc;
        const uint32_t per_row = L.kc / 16;
        for (uint32_t e = tid; e < kLinOTile * per_row; e += kLinBlock) {
            const uint32_t rr = e / per_row, q = e % per_row;
            *reinterpret_cast<uint4 *>(Al + rr * L.astride + 16 * q) =
                *reinterpret_cast<const uint4 *>(ap + static_cast<uint64_t>(rr) * L.kc + 16 * q);
        }
    }
    __syncthreads();  // the only barrier

    // this wave's tile; consecutive workgroups (neighbouring rows) on one XCD
    const uint32_t nb = gridDim.x, full = nb / kXcds * kXcds;
    const uint32_t blk = blockIdx.x < full ? (blockIdx.x % kXcds) * (nb / kXcds) + blockIdx.x / kXcds : blockIdx.x;
    const uint32_t tile = blk * 4 + wave;
    if (tile >= L.nimg * L.rows * L.xtiles) return;  // no barrier follows
    const uint32_t xtile = tile % L.xtiles;
    const uint32_t row = (tile / L.xtiles) % L.rows;
    const uint32_t img = tile / (L.xtiles * L.rows);
    constexpr uint32_t XT = 16 * NCB;
    const uint32_t x0 = xtile * XT;
    const uint32_t kg = 16 * (lane / 16);
    const uint32_t rowb = L.xw * L.xstride;
    auto o_local = [&](int ob, int r) -> uint32_t { return ob * 16 + 4 * (lane / 16) + r; };
    const bool full_tile = x0 + XT <= L.cols && (og + 1) * kLinOTile <= L.c_out;

    // staged pieces of this lane: piece e = lane + 64 s is (row dy, column,
    // 16 channels); plane offset (column clamped into the padded row) and LDS
    // offset (16 bits, 0xffff: not staged; two per register); the 8 lanes of
    // a write group take columns wpair apart
    const uint32_t c16n = L.ck / 16;
    const uint32_t pieces = L.kh * L.xw * c16n;
    uint32_t poff[PL], loff2[(PL + 1) / 2];
#pragma unroll
    for (int s = 0; s < (PL + 1) / 2; ++s) loff2[s] = 0;
#pragma unroll
    for (int s = 0; s < PL; ++s) {
        const uint32_t e = lane + 64 * s;
        const uint32_t ee = e < pieces ? e : 0u;
        const uint32_t c16 = ee % c16n, dy = ee / (c16n * L.xw);
        uint32_t xin = (ee / c16n) % L.xw;
        const uint32_t grp = 2 * L.wpair, gb = xin - xin % grp;
        if (gb + grp <= L.xw) xin = gb + (xin - gb) / 2 + ((xin - gb) % 2) * L.wpair;
        uint32_t xp = x0 * L.stride + xin;
        xp = xp < L.wp ? xp : L.wp - 1;
        poff[s] = ((img * L.hp + row * L.stride + dy) * L.wp + xp) * L.cp + 16 * c16;
        const uint32_t lo = e < pieces ? dy * rowb + xin * L.xstride + 16 * c16 : 0xffffu;
        loff2[s / 2] |= lo << (16 * (s % 2));
    }
    auto loff = [&](int s) -> uint32_t { return (loff2[s / 2] >> (16 * (s % 2))) & 0xffffu; };
    uint32_t colb[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) colb[cb] = (cb * 16 + lane % 16) * L.stride * L.xstride;

    // residue (w, j) (field j of packed word w) is in plane pn(w, j) of the
    // modulus; the halo of the next residue is staged after the operations
    // of this one from registers that hold its plane's pieces, and a plane
    // is loaded into them one residue before its first residue is staged
    auto g_of = [&](uint32_t w) { return (w + 1 == M.W) ? M.glast : M.g; };
    auto pn = [&](uint32_t w, uint32_t j) { return w * M.ppw + (j >> M.lgf); };
    v4i pf[PL];
    auto load = [&](uint32_t pl) {
        const uint8_t *plane = planes + static_cast<uint64_t>(M.pl_off + pl) * L.plane_bytes;
#pragma unroll
        for (int s = 0; s < PL; ++s) pf[s] = load16(plane, lane + 64 * s < pieces ? poff[s] : 0u);
    };
    auto stage = [&](uint32_t j) {
#pragma unroll
        for (int s = 0; s < PL; ++s)
            if (lane + 64 * s < pieces) *reinterpret_cast<v4i *>(Bw + loff(s)) = plane_field(pf[s], M, j);
    };
    load(pn(w_lo, 0));
    stage(0);
    // (nw, nj): the next residue to stage; its plane is in pf once staged
    uint32_t nw = w_lo, nj = 1;
    if (nj == g_of(w_lo)) nw = w_lo + 1, nj = 0;
    if (nw < w_hi && pn(nw, nj) != pn(w_lo, 0)) load(pn(nw, nj));

    uint32_t part[4][NCB][4];
    v4i acc[4][NCB];
#pragma unroll
    for (int ob = 0; ob < 4; ++ob)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int r = 0; r < 4; ++r) part[ob][cb][r] = 0;

    for (uint32_t w = w_lo; w < w_hi; ++w) {
        const uint32_t g = g_of(w);
        uint32_t Rw = 0;
        if constexpr (GARBLE) Rw = offsets[M.woff + w];
        for (uint32_t j = 0; j < g; ++j) {
            const int32_t Rj = GARBLE ? static_cast<int32_t>((Rw >> (M.b * j)) & ((1u << M.b) - 1u)) : 0;
            // the seeds of this lane's 4 output channels of each row block
            // (the C operand of the first K step)
            v4i b0[4];
#pragma unroll
            for (int ob = 0; ob < 4; ++ob) {
                b0[ob] = *reinterpret_cast<const v4i *>(seed + ob * 16 + 4 * (lane / 16));
                if constexpr (GARBLE) b0[ob] += *reinterpret_cast<const v4i *>(negb + ob * 16 + 4 * (lane / 16)) * Rj;
            }
            if constexpr (K33 > 0) {
                // K step kk = 3 dy + dx; the fragments of step kk + 1 are
                // loaded before the matrix-core operations of step kk
                const uint8_t *Ar = Al + (lane % 16) * (576 + 32) + kg;
                auto frag = [&](int kk, v4i(&a)[4], v4i(&bq)[NCB]) {
#pragma unroll
                    for (int ob = 0; ob < 4; ++ob)
                        a[ob] = *reinterpret_cast<const v4i *>(Ar + ob * 16 * (576 + 32) + kk * 64);
                    const uint8_t *Br = Bw + (kk / 3) * rowb + kg + (kk % 3) * K33;
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb) bq[cb] = *reinterpret_cast<const v4i *>(Br + colb[cb]);
                };
                auto mma = [&](int kk, const v4i(&a)[4], const v4i(&bq)[NCB]) {
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                        for (int ob = 0; ob < 4; ++ob)
                            acc[ob][cb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[ob], bq[cb], kk == 0 ? b0[ob] : acc[ob][cb],
                                                                                0, 0, 0);
                };
                v4i fa0[4], fb0[NCB], fa1[4], fb1[NCB];
                frag(0, fa0, fb0);
                // the wave's priority is raised while it issues its
                // matrix-core steps and lowered for the staging and epilogue
                __builtin_amdgcn_s_setprio(1);
#pragma unroll
                for (int kk = 0; kk < 9; ++kk) {
                    // (scheduling barriers keep the loads of step kk + 1
                    // ahead of the operations of step kk)
                    if (kk % 2 == 0) {
                        if (kk + 1 < 9) frag(kk + 1, fa1, fb1);
                        __builtin_amdgcn_sched_barrier(0);
                        mma(kk, fa0, fb0);
                    } else {
                        if (kk + 1 < 9) frag(kk + 1, fa0, fb0);
                        __builtin_amdgcn_sched_barrier(0);
                        mma(kk, fa1, fb1);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
                __builtin_amdgcn_s_setprio(0);
            } else {
#pragma unroll
                for (int ob = 0; ob < 4; ++ob)
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb) acc[ob][cb] = b0[ob];
                const uint32_t ksteps = L.kc / 64;
                for (uint32_t kk = 0; kk < ksteps; ++kk) {
                    v4i a[4];
#pragma unroll
                    for (int ob = 0; ob < 4; ++ob)
                        a[ob] = *reinterpret_cast<const v4i *>(Al + (ob * 16 + lane % 16) * L.astride + kk * 64 + kg);
                    const uint32_t kidx = kk * 64 + kg;
                    uint32_t tap = kidx >> L.lg_ck;
                    if (tap >= L.taps) tap = 0;  // K padding: the weights there are 0
                    const uint32_t dy = __umul24(tap, L.kw_magic) >> 16, dx = tap - dy * L.kw;
                    const uint32_t boff = dy * rowb + dx * L.xstride + (kidx & (L.ck - 1u));
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb) {
                        const v4i bf = *reinterpret_cast<const v4i *>(Bw + boff + colb[cb]);
#pragma unroll
                        for (int ob = 0; ob < 4; ++ob)
                            acc[ob][cb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[ob], bf, acc[ob][cb], 0, 0, 0);
                    }
                }
            }
            // the next residue's halo over this one (after this wave's reads,
            // in LDS order), then the plane of the one after into the
            // registers if it is a new plane
            if (nw < w_hi) {
                stage(nj);
                uint32_t mw = nw, mj = nj + 1;
                if (mj == g_of(mw)) mw += 1, mj = 0;
                if (mw < w_hi && pn(mw, mj) != pn(nw, nj)) load(pn(mw, mj));
                nw = mw;
                nj = mj;
            }
            // epilogue: residue of u mod m into field j
            const uint32_t sh = M.b * j;
            auto epilogue = [&](auto shifts) {
#pragma unroll
                for (int ob = 0; ob < 4; ++ob)
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const uint32_t u = static_cast<uint32_t>(acc[ob][cb][r]);
                            uint32_t q = __umulhi(u, M.divM);  // < 2^23
                            if constexpr (decltype(shifts)::value) q >>= M.divS;
                            const uint32_t res =
                                static_cast<uint32_t>(__mul24(static_cast<int32_t>(q), -static_cast<int32_t>(M.m))) + u;
                            part[ob][cb][r] |= res << sh;
                        }
            };
            if (M.divS == 0)
                epilogue(std::integral_constant<bool, false>{});
            else
                epilogue(std::integral_constant<bool, true>{});
        }
        // word w complete: store it.  Element (ob, cb, r) of this lane is
        // output channel og 64 + ob 16 + 4 (lane / 16) + r at position
        // x0 + cb 16 + lane % 16: a per-lane offset plus a uniform step.
        uint32_t *dstp = out + (static_cast<uint64_t>(M.woff) + w) * L.n_out + img * L.oN + row * L.oY +
                         x0 * L.oX + og * kLinOTile * L.oO;
        const uint32_t lo = 4 * (lane / 16) * L.oO + (lane % 16) * L.oX;
        if (full_tile) {
#pragma unroll
            for (int ob = 0; ob < 4; ++ob)
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        uint32_t *d = dstp + (ob * 16 + r) * L.oO + cb * 16 * L.oX;
                        d[lo] = part[ob][cb][r];
                        part[ob][cb][r] = 0;
                    }
        } else {
#pragma unroll
            for (int ob = 0; ob < 4; ++ob)
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const uint32_t o = og * kLinOTile + o_local(ob, r), x = x0 + cb * 16 + lane % 16;
                        uint32_t *d = dstp + (ob * 16 + r) * L.oO + cb * 16 * L.oX;
                        if (o < L.c_out && x < L.cols) d[lo] = part[ob][cb][r];
                        part[ob][cb][r] = 0;
                    }
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

template <int NCB, bool GARBLE, int K33>
int launch_gemm(const LinPlan &L, const uint8_t *planes, const uint8_t *prep, const int64_t *bias,
                const uint32_t *offsets, uint32_t *out, hipStream_t stream) {
    int rc = lin_allow_lds(reinterpret_cast<const void *>(&k_linear_gemm<NCB, GARBLE, K33>), L.lds_bytes);
    if (rc) return rc;
    const uint64_t tiles = static_cast<uint64_t>(L.nimg) * L.tile_rows * L.xtiles;
    if (tiles >= (1ull << 31)) return REDASH_E_PARAM;
    hipLaunchKernelGGL((k_linear_gemm<NCB, GARBLE, K33>),
                       L.word_split ? dim3(static_cast<uint32_t>(tiles), L.ogroups, L.npairs)
                                    : dim3(static_cast<uint32_t>(tiles), L.k, L.ogroups),
                       dim3(kLinBlock), L.lds_bytes, stream, L, planes, prep, bias, offsets, out);
    return lin_launched();
}

template <int NCB, bool GARBLE, int K33>
int launch_gemm_w(const LinPlan &L, const uint8_t *planes, const uint8_t *prep, const int64_t *bias,
                  const uint32_t *offsets, uint32_t *out, hipStream_t stream) {
    constexpr int PL = K33 > 0 ? 7 : kWavePieces;
    if (L.kh * L.xw * (L.ck / 16) > 64u * PL || L.halo > 0xffffu) return REDASH_E_PARAM;  // not reached
    const uint32_t lds = L.lds_a + 4 * L.halo + 2 * kLinOTile * 4;
    int rc = lin_allow_lds(reinterpret_cast<const void *>(&k_linear_gemm_w<NCB, GARBLE, K33, PL>), lds);
    if (rc) return rc;
    const uint64_t tiles = static_cast<uint64_t>(L.nimg) * L.rows * L.xtiles;
    if (tiles >= (1ull << 31)) return REDASH_E_PARAM;
    const uint32_t nb = static_cast<uint32_t>((tiles + 3) / 4);
    hipLaunchKernelGGL((k_linear_gemm_w<NCB, GARBLE, K33, PL>),
                       L.word_split ? dim3(nb, L.ogroups, L.npairs) : dim3(nb, L.k, L.ogroups),
                       dim3(kLinBlock), lds, stream, L, planes, prep, bias, offsets, out);
    return lin_launched();
}

template <int NCB, bool GARBLE>
int launch_gemm_k(const LinPlan &L, const uint8_t *planes, const uint8_t *prep, const int64_t *bias,
                  const uint32_t *offsets, uint32_t *out, hipStream_t stream) {
    // one channel chunk (and a halo of at most 8 pieces per lane): independent waves
    if (L.ncc == 1 && L.kh * L.xw * (L.ck / 16) <= 64 * kWavePieces &&
        L.lds_a + 4 * L.halo + 2 * kLinOTile * 4 <= kLinMaxLds) {
        const bool k33 = L.kh == 3 && L.kw == 3 && L.ck == 64 && 3 * L.xw * 4 <= 7 * 64;
        if (k33 && L.xstride == 96) return launch_gemm_w<NCB, GARBLE, 96>(L, planes, prep, bias, offsets, out, stream);
        if (k33 && L.xstride == 80) return launch_gemm_w<NCB, GARBLE, 80>(L, planes, prep, bias, offsets, out, stream);
        return launch_gemm_w<NCB, GARBLE, 0>(L, planes, prep, bias, offsets, out, stream);
    }
    if (L.kh == 3 && L.kw == 3 && L.ck == 64 && L.xstride == 96)
        return launch_gemm<NCB, GARBLE, 96>(L, planes, prep, bias, offsets, out, stream);
    if (L.kh == 3 && L.kw == 3 && L.ck == 64 && L.xstride == 80)
        return launch_gemm<NCB, GARBLE, 80>(L, planes, prep, bias, offsets, out, stream);
    return launch_gemm<NCB, GARBLE, 0>(L, planes, prep, bias, offsets, out, stream);
}

template <bool GARBLE>
int launch_linear(const LinPlan &L, const uint32_t *in, const uint8_t *prep, const int64_t *bias,
                  const uint32_t *offsets, uint8_t *work, uint32_t *out, hipStream_t stream) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess) return REDASH_E_HIP;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) return REDASH_E_HIP;
    if (L.lds_bytes > static_cast<uint32_t>(v)) return REDASH_E_HIP;
    const uint64_t npos = static_cast<uint64_t>(L.nimg) * L.hp * L.wp;
    if (npos >= (1ull << 32)) return REDASH_E_PARAM;
    hipLaunchKernelGGL(k_linear_unpack, dim3(static_cast<uint32_t>((npos + 63) / 64), L.npairs, (L.cp + 63) / 64),
                       dim3(256), 0, stream, L, in, work);
    if (lin_launched()) return REDASH_E_HIP;
    if (L.xt == 32) return launch_gemm_k<2, GARBLE>(L, work, prep, bias, offsets, out, stream);
    return launch_gemm_k<1, GARBLE>(L, work, prep, bias, offsets, out, stream);
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
    out->work_bytes = work_bytes(L);
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
                       uint8_t *d_work, uint32_t *d_out_labels, hipStream_t stream) {
    LinPlan L;
    const int rc = build_lin_plan(p, &L);
    if (rc) return rc;
    if (!d_in_labels || !d_prepared || !d_work || !d_out_labels) return REDASH_E_NULL;
    return launch_linear<false>(L, d_in_labels, d_prepared, nullptr, nullptr, d_work, d_out_labels, stream);
}

int redash_linear_garble(const redash_linear_params *p, const uint32_t *d_in_zero, const uint8_t *d_prepared,
                         const int64_t *d_bias, const uint32_t *d_offsets, uint8_t *d_work, uint32_t *d_out_zero,
                         hipStream_t stream) {
    LinPlan L;
    const int rc = build_lin_plan(p, &L);
    if (rc) return rc;
    if (!d_in_zero || !d_prepared || !d_offsets || !d_work || !d_out_zero) return REDASH_E_NULL;
    return launch_linear<true>(L, d_in_zero, d_prepared, d_bias, d_offsets, d_work, d_out_zero, stream);
}

}  // extern "C"
