/*
 * redash.h -- C ABI of the MI355X (gfx950) library for the ReDASH garbled
 * scaling gadget (Maurer, Sander, Eisenbarth: "ReDASH", arXiv 2506.14489).
 *
 * The gadget maps an RNS-encoded activation, held as one arithmetic-garbled
 * wire label per base modulus, to floor(x / s) where s is one base modulus or
 * a product of base moduli.  It is ShiftUp by P/2, a division step per factor
 * of s (Sec. 3.2), the generalized base extension (Sec. 3.3, Eq. rns_to_mrs)
 * and ShiftDown by P/(2s) (Sec. 3.4).  Every step that is not free label
 * arithmetic (Sec. 2.3) is a projection gate: hash the digit label, select a
 * ciphertext row by the label's colour, decrypt.
 *
 * Roles (Sec. 2.1): the garbler garbles offline (redash_garble_scale), hands
 * the evaluator its input labels (redash_encode stands in for the oblivious
 * transfer) and decodes the returned labels (redash_decode).  The evaluator
 * runs redash_eval_scale online; that call is the hot path.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers named d_* are DEVICE pointers on the current HIP device.  The
 *    caller allocates and owns every buffer, sized from redash_plan(); the
 *    library never allocates or frees device memory and keeps no state
 *    between calls beyond read-only constants, host-side caches (per host
 *    thread, the plan of the last redash_params it passed; per device, its
 *    compute-unit count and LDS limit) and the fixed buffer of
 *    redash_eval_scale_noalloc.
 *  - Calls are asynchronous on `stream` (0 = the null stream); they return
 *    after the launches are queued.  Buffers must stay valid until the stream
 *    reaches the work.  Calls that write the same buffers must be ordered by
 *    the caller.
 *  - Return codes: REDASH_OK (0) or a negative REDASH_E* value; nothing is
 *    launched when a call returns an error.  Device kernels never trap.
 *  - Label encoding ("PK32"): a label over Z_m has lambda_m residues, lambda_m
 *    the least integer with m^lambda_m >= 2^128 (128-bit security, Sec. 2.3
 *    leaves the length open).  With b_m = bit length of (m-1) and
 *    g_m = floor(32 / b_m), residue r sits in 32-bit word r / g_m at bit
 *    b_m * (r % g_m); unused bits are zero.  W_m = ceil(lambda_m / g_m) words.
 *  - LabelTensor layout (structure of arrays): for base modulus i in base
 *    order, a block of W_{m_i} * n words; word w of gadget a is at
 *    block_i + w * n + a.  label_words = n * sum_i W_{m_i}.
 *  - Offsets (the garbler's global offsets R_m, Sec. 2.3: l_v = l_0 + v R):
 *    one PK32 label per modulus in base order, offset_words = sum_i W_{m_i}.
 *  - Garbled tables: one block per projection gate in gate order; gate g with
 *    input modulus q and output modulus m holds n * (q-1) * W_m words (row
 *    reduction, Sec. 2.3: the colour-0 row is implicit).  The row of colour
 *    c in 1..q-1 of gadget a starts at word (a * (q-1) + c - 1) * W_m of the
 *    gate block.
 *  - Gate order (the same for every gadget): Phase A (division, Sec. 3.2):
 *    for each scaling modulus S[a] in ascending order, one gate onto every
 *    later scaling modulus and then onto every remaining modulus R.  Phase B
 *    (base extension, Sec. 3.3): for each remaining modulus R[b] in ascending
 *    order, one gate onto every later remaining modulus and then onto every
 *    scaling modulus.  gates = k(k-1)/2 + t(k-t).
 *  - Hash of a projection gate (the paper fixes none): fixed-key AES-128 in
 *    Matyas-Meyer-Oseas form with the key 00 01 .. 0f, applied to the linear
 *    orthomorphism sigma(x) = ((x_hi ^ x_lo) << 64) | x_hi of the XOR-fold
 *    of the input label's PK32 words, tweaked with
 *    T_j = gadget_id * 2^96 + ((4 tau + j) mod 2^64), tau = a * gates + g, and
 *    gadget_id = seed mod 2^32; two blocks (one when m = 2) give a 256-bit
 *    (128-bit) fraction whose first lambda_m base-m digits are the pad.
 */
#ifndef REDASH_H
#define REDASH_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define REDASH_OK 0
#define REDASH_E_PARAM (-1) /* invalid parameters (see redash_params)             */
#define REDASH_E_NULL (-2)  /* a required pointer is NULL                          */
#define REDASH_E_HIP (-3)   /* a HIP launch or runtime call failed                 */
#define REDASH_E_LABEL (-4) /* reported by callers that read d_bad_count > 0       */
#define REDASH_E_SIZE (-5)  /* the call needs more than the library's fixed buffer */

/* Words of the fixed working buffer of redash_eval_scale_noalloc (64 MiB). */
#define REDASH_NOALLOC_WORK_WORDS (16ull << 20)

#define REDASH_MAX_K 15

/*
 * One gadget call: n independent gadget instances with the same base and
 * scaling factor.
 *   k           number of base moduli, 2..15.
 *   moduli      the RNS base (Sec. 2.2): primes or powers of two (Sec. 4
 *               uses one 2^l modulus), 2..255, strictly ascending, pairwise
 *               coprime, with P = prod(moduli) < 2^63.
 *   t           number of scaling moduli, 1..k-1.
 *   scale_idx   indices into moduli of the scaling moduli S, strictly
 *               ascending; s = prod of those moduli (Sec. 3.4: s may be one
 *               base modulus or a product of several).  ShiftUp adds
 *               U = floor(P/2) and ShiftDown subtracts floor(U/s) (Sec. 3.4's
 *               P/2 and P/(2s) where those are integers), so the gadget
 *               returns floor((x + (U mod s)) / s): floor(x/s) whenever
 *               P/(2s) is an integer, round-half-up of x/s for a base whose
 *               only even modulus 2^l is scaled by.
 *   n           number of gadget instances held in the buffers (may be 0).
 *   seed        garbler seed: keys the garbling PRG; gadget_id = seed mod 2^32.
 *   a0          global index of the first gadget held in the buffers.  The
 *               hash tweaks and the PRG are addressed by a0 + local index, so
 *               any slice of a larger call can be garbled or evaluated alone.
 * The struct is passed by pointer; unused array entries are ignored.
 */
typedef struct {
    uint32_t k;
    uint32_t moduli[16];
    uint32_t t;
    uint32_t scale_idx[16];
    uint64_t n;
    uint64_t seed;
    uint64_t a0;
} redash_params;

/* Buffer sizes in 32-bit words for a given redash_params. */
typedef struct {
    uint64_t label_words;  /* one LabelTensor (inputs, outputs, zero-labels) */
    uint64_t table_words;  /* all garbled tables of the n gadgets            */
    uint32_t offset_words; /* the k offsets R_m                              */
    uint32_t gates;        /* projection gates per gadget                    */
    uint64_t work_words;   /* evaluator working storage (redash_eval_scale)  */
} redash_sizes;

/*
 * Host only, no device work.  Validates `p` and reports the buffer sizes.
 * Returns REDASH_E_NULL if p or out is NULL, REDASH_E_PARAM if p is invalid.
 */
int redash_plan(const redash_params *p, redash_sizes *out);

/*
 * Garbler, offline phase (Sec. 2.1; Sec. 2.3 projection gates with row
 * reduction; Sec. 3.4 free ShiftUp/ShiftDown applied to zero-labels).
 * Writes:
 *   d_offsets   offset_words: R_m for every modulus (R_m[0] a unit of Z_m,
 *               so the m colours of a wire are distinct).
 *   d_in_zero   label_words: input zero-labels Z of gadgets a0..a0+n-1.
 *   d_out_zero  label_words: output zero-labels (value 0 after ShiftDown);
 *               also holds intermediate zero-labels while the call runs.
 *   d_tables    table_words: every garbled row (may be NULL when n = 0).
 *   d_work      work_words of working storage, as for redash_eval_scale
 *               (may be NULL when n = 0 or work_words = 0).
 * Deterministic in (moduli, scale set, seed, global gadget index).
 * REDASH_E_PARAM also when n >= 2^30.
 */
int redash_garble_scale(const redash_params *p, uint32_t *d_offsets, uint32_t *d_in_zero,
                        uint32_t *d_out_zero, uint32_t *d_tables, uint32_t *d_work, hipStream_t stream);

/*
 * Garbler on given input zero-labels: as redash_garble_scale, except that the
 * input zero-labels Z are read from d_in_zero (label_words, read only) instead
 * of being drawn from the PRG.  This chains a gadget after free operations
 * (Sec. 2.3: sums and public multiples of labels, e.g. the output
 * zero-labels of redash_linear_garble) whose labels were built on the same
 * offsets: d_offsets is written from the seed exactly as redash_garble_scale
 * writes it, so the seed must be the one whose offsets the zero-labels use.
 * The tweaks are (seed, global gadget index a0 + a) as in
 * redash_garble_scale: gadgets garbled under one seed must use disjoint
 * ranges a0..a0+n-1, including the gadgets whose PRG zero-labels fed the
 * free operations.  d_in_zero may not alias d_out_zero, d_tables or d_work.
 * Return codes as for redash_garble_scale.
 */
int redash_garble_scale_given(const redash_params *p, uint32_t *d_offsets, const uint32_t *d_in_zero,
                              uint32_t *d_out_zero, uint32_t *d_tables, uint32_t *d_work,
                              hipStream_t stream);

/*
 * Stand-in for the oblivious transfer of input labels (Sec. 2.1):
 * X_{a,i} = Z_{a,i} + ((x_a mod P) mod m_i) * R_{m_i}, residue-wise mod m_i.
 *   d_x         n signed activations (int64), any value (reduced mod P; the
 *               result is as stated under redash_params for x in the signed
 *               range [-floor(P/2), ceil(P/2) - 1], Sec. 2.4, 3.2, 3.4).
 *   d_in_zero   label_words, from redash_garble_scale.
 *   d_offsets   offset_words, from redash_garble_scale.
 *   d_in_labels label_words, written.
 */
int redash_encode(const redash_params *p, const int64_t *d_x, const uint32_t *d_in_zero,
                  const uint32_t *d_offsets, uint32_t *d_in_labels, hipStream_t stream);

/*
 * Evaluator, online phase: THE HOT PATH.  Runs the scaling gadget of
 * Sec. 3.4 on n LabelTensors: per projection gate, colour c = residue 0 of
 * the digit label, pad = hash (see conventions), E = row[c] + pad (row 0 is
 * zero), then the free operation of the gate -- Phase A and the recursion of
 * Phase B: L_dst <- q^{-1} (L_dst - E) mod m (Sec. 3.2 display equation,
 * Eq. rns_to_mrs); Phase B onto the scaling moduli: Acc_dst <- Acc_dst +
 * w * E with the mixed-radix weight w = prod of the earlier remaining moduli
 * (the missing residue of Sec. 3.3 written as the mixed-radix value of the
 * digits).
 *   d_in_labels  label_words (read only).
 *   d_tables     table_words from redash_garble_scale with the same params.
 *   d_out_labels label_words, written; also holds intermediate labels while
 *                the call runs.  May not alias d_in_labels or d_work.
 *   d_work       work_words of working storage: the Phase-B copies of the
 *                remaining moduli (Sec. 3.3 consumes them while the Phase-A
 *                values are outputs).  Contents on entry are ignored and on
 *                return unspecified; may be NULL when work_words is 0.
 * Output labels carry floor(x/s) (see redash_params) under the garbler's
 * output zero-labels.
 * REDASH_E_PARAM also when n >= 2^30 (a gadget's byte offset must fit in
 * 32 bits).
 */
int redash_eval_scale(const redash_params *p, const uint32_t *d_in_labels, const uint32_t *d_tables,
                      uint32_t *d_out_labels, uint32_t *d_work, hipStream_t stream);

/*
 * redash_eval_scale for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, results and return codes as redash_eval_scale,
 * without d_work: the working storage is a buffer of
 * REDASH_NOALLOC_WORK_WORDS words inside the library, one per GPU, which
 * each GPU holds from the loading of the library's kernels onto it until the
 * process ends.  The
 * call allocates and frees nothing (no hipMalloc, hipFree or allocating
 * library routine).
 *   Limit: n * work_words (from redash_plan) <= REDASH_NOALLOC_WORK_WORDS,
 *   else REDASH_E_SIZE and nothing is launched (the 12-prime base scaled by
 *   one modulus needs 54 words per gadget: up to 310,689 gadgets per call).
 *   Sharing: every call on a GPU uses that GPU's one buffer.  Calls that can
 *   overlap on one GPU (different streams without ordering between them, or
 *   several host threads) race on it and give wrong labels; order them on one
 *   stream.  Nothing in the buffer has to start at zero, and its contents
 *   after a call are unspecified.
 */
int redash_eval_scale_noalloc(const redash_params *p, const uint32_t *d_in_labels, const uint32_t *d_tables,
                              uint32_t *d_out_labels, hipStream_t stream);

/*
 * Garbler decodes the returned labels (Sec. 2.1): v_i = (Y_i[0] - O_i[0]) *
 * R_i[0]^{-1} mod m_i, y = CRT(v) in the signed range
 * [-floor(P/2), ceil(P/2) - 1] (Sec. 2.4).  A gadget whose label differs from O_i + v_i R_i in any residue
 * is counted as bad (its d_y entry is still written).
 *   d_out_labels, d_out_zero  label_words; d_offsets offset_words.
 *   d_y          n int64, written.
 *   d_bad_count  one uint64, overwritten with the number of bad gadgets.
 * Callers that want an error on bad labels read d_bad_count after the stream
 * completes and report REDASH_E_LABEL when it is nonzero.
 */
int redash_decode(const redash_params *p, const uint32_t *d_out_labels, const uint32_t *d_out_zero,
                  const uint32_t *d_offsets, int64_t *d_y, uint64_t *d_bad_count, hipStream_t stream);

/*
 * The projection-gate hash alone (Sec. 2.3; construction in the conventions
 * above), for tests.
 *   q, m        input and output modulus (2..255, prime or a power of two).
 *   count       number of labels.
 *   d_labels    W_q * count words, SoA: word w of label a at w * count + a.
 *   gadget_id   tweak high word.
 *   d_tau       count uint64 tweaks.
 *   d_out       W_m * count words, SoA, written.
 */
int redash_hash_labels(uint32_t q, uint32_t m, uint64_t count, const uint32_t *d_labels,
                       uint32_t gadget_id, const uint64_t *d_tau, uint32_t *d_out, hipStream_t stream);

/*
 * The AES of the projection-gate hash alone, for measuring the device's AES
 * rate with the evaluator's round-table code (Sec. 2.3 leaves the hash to the
 * implementation; the conventions above fix AES-128 under K = 00 01 .. 0f):
 * counter mode, d_out[4i .. 4i+3] = AES_K(c0 + i) for i < count, the counter
 * block being the 128-bit little-endian integer c0 + i and each output block
 * four little-endian words.
 *   count   number of blocks, at most 2^40 (else REDASH_E_PARAM).
 *   d_out   4 * count words, written.
 */
int redash_aes_ctr(uint64_t count, uint64_t c0, uint32_t *d_out, hipStream_t stream);

/*
 * The same counter-mode output as redash_aes_ctr from a bitsliced AES-128 (32
 * blocks per 32-bit lane word, the S-box as the Boyar-Peralta circuit, no
 * table lookups), to compare the two formulations' rates on the device.
 * Same arguments, layout and return codes.
 */
int redash_aes_ctr_bitsliced(uint64_t count, uint64_t c0, uint32_t *d_out, hipStream_t stream);

/* Static text for a return code. */
const char *redash_strerror(int code);

/* ========================================================================
 * Garbled linear layers on LabelTensors (the layer that feeds the gadget)
 * ========================================================================
 *
 * Arithmetic garbling makes addition and multiplication by a public constant
 * free (Sec. 2.3): a dense or 2-D convolution layer with public integer
 * weights w and bias b, y = W x + b, is evaluated on labels residue by
 * residue, Y_o = sum_j w_oj X_j mod m, and the garbler, who knows the
 * offsets R, sets the output zero-labels Z_o = sum_j w_oj Z_j - b_o R, so
 * that Y_o carries y_o.  The paper runs these layers on LabelTensors with
 * 32-bit residue arithmetic (Sec. 3.6); here the contraction runs on int8
 * matrix cores (each residue and each weight reduced mod m fits a signed
 * byte): the input residues are unpacked once into byte planes in a
 * caller-provided working buffer, and the reduction mod m and the PK32
 * packing are fused into the contraction.
 *
 * Layer: input NCHW (batch, c_in, h_in, w_in) of activations, weights OIHW
 * (c_out, c_in, kh, kw), stride, zero padding `pad` (a padded input is the
 * public constant 0, whose label is the all-zero label), output NCHW
 * (batch, c_out, h_out, w_out) with h_out = (h_in + 2 pad - kh)/stride + 1,
 * w_out likewise.  A dense layer (batch, in) -> (batch, out) is the case
 * h_in = w_in = kh = kw = 1 (the NCHW and row-major layouts coincide).
 * Activations are numbered in NCHW order; label tensors use the LabelTensor
 * layout of the conventions above with n = the number of activations.
 *
 *   k, moduli   the RNS base, as in redash_params (primes or powers of two,
 *               2..255, ascending, pairwise coprime, P < 2^63).
 *   batch, c_in, h_in, w_in, c_out, kh, kw, stride, pad  the layer, with
 *               every size >= 1, pad < kh and pad < kw, c_in kh kw <= 16384,
 *               kh kw <= 64, and at most 2^30 - 1 input and output
 *               activations.
 */
typedef struct {
    uint32_t k;
    uint32_t moduli[16];
    uint32_t batch, c_in, h_in, w_in;
    uint32_t c_out, kh, kw;
    uint32_t stride, pad;
} redash_linear_params;

typedef struct {
    uint64_t in_label_words;  /* input LabelTensor: batch c_in h_in w_in sum_i W_i   */
    uint64_t out_label_words; /* output LabelTensor: batch c_out h_out w_out sum_i W_i */
    uint64_t prepared_bytes;  /* prepared weights (redash_linear_prepare)          */
    uint64_t work_bytes;      /* working buffer of redash_linear_eval / _garble    */
    uint32_t h_out, w_out;
    uint32_t offset_words;    /* the k offsets R_m (redash_linear_garble)          */
} redash_linear_sizes;

/* Host only.  Validates `p` and reports the sizes.  REDASH_E_NULL, REDASH_E_PARAM. */
int redash_linear_plan(const redash_linear_params *p, redash_linear_sizes *out);

/*
 * Once per layer and base (weights are constants of the model): reduces every
 * weight mod each m_i into the signed range of Z_m_i and lays it out for the
 * layer kernels (the layout is private to the library; only its size,
 * prepared_bytes, is public).
 *   d_weights   c_out c_in kh kw int32 weights, OIHW (any int32 values).
 *   d_prepared  prepared_bytes, written.
 */
int redash_linear_prepare(const redash_linear_params *p, const int32_t *d_weights, uint8_t *d_prepared,
                          hipStream_t stream);

/*
 * Evaluator, online: Y = sum w X, every residue of every modulus (Sec. 2.3).
 *   d_in_labels   in_label_words (read only).
 *   d_prepared    from redash_linear_prepare with the same params.
 *   d_work        work_bytes of working storage: the input residues in
 *                 zero-padded channel-last byte planes (one residue per
 *                 byte, or 8, 4 or 2 residues of a modulus m <= 16 in 1-,
 *                 2- or 4-bit fields).  Contents on entry are ignored and on
 *                 return unspecified.
 *   d_out_labels  out_label_words, written; may not alias d_in_labels.
 */
int redash_linear_eval(const redash_linear_params *p, const uint32_t *d_in_labels, const uint8_t *d_prepared,
                       uint8_t *d_work, uint32_t *d_out_labels, hipStream_t stream);

/*
 * Garbler: output zero-labels Z_o = sum w Z - b_o R (Sec. 2.3), so that the
 * evaluator's output label of activation o carries sum w x + b_o.
 *   d_in_zero   in_label_words: zero-labels of the layer's inputs.
 *   d_prepared  from redash_linear_prepare with the same params.
 *   d_bias      c_out int64 biases, or NULL for none.
 *   d_offsets   offset_words: the offsets R_m (as from redash_garble_scale).
 *   d_work      work_bytes of working storage, as for redash_linear_eval.
 *   d_out_zero  out_label_words, written; may not alias d_in_zero.
 */
int redash_linear_garble(const redash_linear_params *p, const uint32_t *d_in_zero, const uint8_t *d_prepared,
                         const int64_t *d_bias, const uint32_t *d_offsets, uint8_t *d_work, uint32_t *d_out_zero,
                         hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* REDASH_H */
