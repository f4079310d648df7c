/*
 * mxq.h -- C ABI of libmxq, mixed-mantissa MXINT (4/6/8-bit) activation
 * quantization and MXINT GEMM on AMD MI355X (gfx950).
 *
 * The operations follow MXSens (arXiv 2607.17733):
 *   - MXINT (Section 2): blocks of 32 consecutive values along the reduction
 *     dimension K share one power-of-two scale stored as an 8-bit exponent
 *     (Section 5.1: +0.25 bit per element); elements are fixed-point
 *     integers, so a block dot product is an integer multiply-accumulate
 *     followed by a power-of-two scaling.
 *   - Mixed mantissas (Section 4.1, Algorithm 2): each block has exactly one
 *     mantissa width out of {4, 6, 8} (or {3, 6, 8}, the Section 5
 *     template); columns are permuted so that
 *     same-width columns fill whole blocks.  The widths and the permutation
 *     are the output of the offline sensitivity analysis (Algorithms 1-3,
 *     Theorem A.1) and are inputs here.  Weights and activations of a linear
 *     share one width map (Section 3.1: one sensitivity metric for both).
 *
 * Quantization of one block x[0..31] with width m (m counts the sign bit):
 *   e = floor(log2(max|x|)) clamped to [-127, 127], stored as E = e + 127;
 *   s = e - (m - 2) is the weight of the mantissa LSB;
 *   q = clamp(round(x / 2^s)) with round = nearest-even (default) or
 *   nearest-away, clamp = symmetric +-(2^(m-1)-1) (default) or full
 *   [-2^(m-1), 2^(m-1)-1].
 *   A block whose maximum is zero or subnormal has E = 0 (e clamps to
 *   -127); a block holding Inf or NaN has E = 255 and zero mantissas.
 * GEMM: Y[i][j] = sum_b P[i][j][b] * 2^(sa[i][b] + sw[j][b]) with
 *   P[i][j][b] = sum_t qa[i][32b+t] * qw[j][32b+t] and s = E - 127 - (m - 2),
 *   accumulated in fp32.  Every elementary product is exact: both kernels
 *   turn each mantissa into one or two FP6/FP8 "digits" whose sum is
 *   q * 2^-(m - 2), multiply them on the block-scaled matrix cores with each
 *   block's E as its E8M0 hardware scale, and accumulate in fp32.  Any block
 *   with E == 255 on either side makes
 *   the outputs it touches NaN.  Results whose magnitude is below fp32's
 *   range (2^-149) flush towards zero.
 *
 * Conventions for every entry point:
 *   - All functions are thread-safe and reentrant.  Device work is enqueued
 *     on `stream` (a hipStream_t; NULL = the default stream) and runs
 *     asynchronously; nothing synchronizes, allocates or frees memory.
 *   - The caller owns every buffer.  "DEVICE" pointers are device memory of
 *     the current HIP device; "HOST" pointers are read during the call only.
 *   - Device pointers must be 16-byte aligned.  Leading dimensions (lda,
 *     ldw, ldy) are in elements.
 *   - On invalid arguments a nonzero mxq_status is returned before anything
 *     is enqueued and no output is touched.  A failed kernel launch returns
 *     MXQ_ERR_DEVICE.  No C++ exception crosses the ABI.
 *   - M == 0 or N == 0 is valid and enqueues nothing.
 */
#ifndef MXQ_H
#define MXQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MXQ_ABI_VERSION 12
#define MXQ_BLOCK 32
/* mxq_gemm uses the weight-streaming decode kernel for M <= this (up to
 * four 16-row activation tiles per weight read). */
#define MXQ_DECODE_MAX_M 64

typedef enum {
  MXQ_OK = 0,
  MXQ_ERR_NULL = 1,        /* a required pointer is NULL */
  MXQ_ERR_SHAPE = 2,       /* K % 32 != 0, K <= 0, negative sizes, ld < K/N */
  MXQ_ERR_WIDTHS = 3,      /* a width not in {3,4,6,8}, or widths not non-decreasing */
  MXQ_ERR_PERM = 4,        /* reserved: permutations are not validated (see below) */
  MXQ_ERR_ALIGN = 5,       /* a device pointer is not 16-byte aligned */
  MXQ_ERR_UNSUPPORTED = 6, /* block != 32, unknown round/clamp mode */
  MXQ_ERR_DEVICE = 7,      /* kernel launch or device query failed */
  MXQ_ERR_SCRATCH = 8      /* sizes exceed an allocation-free entry point's static scratch */
} mxq_status;

typedef enum { MXQ_ROUND_NEAREST_EVEN = 0, MXQ_ROUND_NEAREST_AWAY = 1 } mxq_round;
typedef enum { MXQ_CLAMP_SYMMETRIC = 0, MXQ_CLAMP_FULL = 1 } mxq_clamp;

/*
 * Format of one quantized linear (shared by its activations and weights).
 *   K       reduction length, a positive multiple of 32.
 *   block   must be 32.
 *   round   mxq_round.   clamp   mxq_clamp.
 *   widths  HOST, K/32 entries, each 3, 4, 6 or 8, non-decreasing (3-bit,
 *           then 4-bit, 6-bit and 8-bit blocks; any count may be zero).
 *           Width 3 is the floor of the paper's 3-6-8 template (Section 5,
 *           the average-bitwidth study): |q| <= 3 (symmetric) or -4..3
 *           (full), LSB weight 2^(e - 1).  3-bit blocks form their own
 *           segment in every layout below and take 3 bits per mantissa in
 *           the packed rows and in the symmetric-clamp weights;
 *           mxq_unpack_* and mxq_gemm_partials report their mantissas q.
 *   perm    DEVICE int32[K] or NULL (identity).  Position p of the quantized
 *           row holds source column perm[p].  Entries outside [0, K) are read
 *           as +0.0 (never dereferenced); duplicates are allowed.
 */
typedef struct {
  int64_t K;
  int32_t block;
  int32_t round;
  int32_t clamp;
  int32_t reserved;        /* must be 0 */
  const uint8_t *widths;
  const int32_t *perm;
} mxq_fmt;

int mxq_abi_version(void);
const char *mxq_status_str(int status);

/*
 * Sizes (bytes) of the buffers; negative mxq_status on a bad format or a
 * negative count.  The algorithmic size of a quantized row is Section 2's
 * MXINT storage: m bits per element of an m-bit block plus one 8-bit shared
 * exponent per 32-element block (the 0.25 bits per element that Section 5.1
 * adds to the average bitwidth).  The packed rows (C) hold exactly that,
 * rounded up to 16 bytes, and the symmetric-clamp weights (B) within a few
 * percent; the operand image (A) holds matrix-core digits instead (6 or 8
 * bits per element and digit plane).
 *
 * Steps and lanes (shared by the GEMM layouts below).  The K-blocks of a
 * width map form four segments in order: the 3-bit, 4-bit, 6-bit and 8-bit
 * blocks.  Each segment is walked in steps, four blocks per step for 3- and
 * 4-bit blocks and two for 6- and 8-bit blocks (s' = step index within the
 * segment, blocks counted within the segment; a segment's last step is
 * completed with zero blocks: mantissas 0, E = 0).  The steps of a segment
 * form groups of four (the last may be shorter) that share scale words; the
 * groups of all segments are numbered in order.  A step holds 64 "lanes"
 * l = 16 g + r (lane group g = 0..3; r = row of a 16-row tile or column of a
 * 16-column slab): the lane order of the gfx950 block-scaled 16x16x128
 * matrix-core instruction.
 *
 * (A) mxq_quantize_act's output for M rows, the matrix-core operand image:
 *   a_mant, mxq_act_bytes(fmt, M): ceil(M / 16) tiles of 16 rows (rows past
 *   M are zero rows), each the steps in order, a step being 64 lanes of 24
 *   bytes (3-, 4- and 6-bit steps) or 32 bytes (8-bit steps), lane l at
 *   l * 24 (or 32).  FP6 lanes hold 32 e3m2 codes, element t at bits
 *   6t..6t+5 of the 24 little-endian bytes; FP8 bytes are e4m3 codes.
 *     3/4-bit step: lane (g, r) holds block 4s'+g of row r: the e3m2 codes
 *       of the values q (4-bit) or 2q (3-bit);
 *     6-bit step: with q = 8h + l, h = floor(q / 8): lane (2j, r) holds the
 *       codes of h/2 and lane (2j+1, r) those of l/16 for block 2s'+j;
 *     8-bit step: with q = 16h + l, h = floor(q / 16): for block 2s'+j,
 *       lane (e, r) bytes 16j..16j+15 hold the codes of 2h and lane
 *       (2+e, r) bytes 16j..16j+15 those of l/8, for elements 16e..16e+15
 *       (e = 0, 1).
 *   a_exp, mxq_act_exp_bytes(fmt, M): per tile, per group, 256 bytes: lane
 *   l's byte for step k of the group at 4 l + k, the E of the block whose
 *   codes the lane holds (block 4s'+g, or 2s'+(g >> 1) for 6/8-bit steps),
 *   0 for zero blocks and for the missing steps of a short group.
 *   So a lane's codes times 2^(E - 127) are q * 2^(E - 127) times 1 (4-bit),
 *   2 (3-bit), 1/16 (6-bit, h/2 + l/16) or 1/8 (8-bit, 2h + l/8); the
 *   weights' digits below carry the rest of 2^-(m - 2) per operand.
 *
 * (B) mxq_pack_weights' output for N columns, mxq_weight_bytes(fmt, N): the
 *   one copy of the weights both GEMMs read, at the size of the mantissas
 *   under the symmetric clamp (3, 4, 6 and 8 bits per element; the full
 *   clamp's wider ranges take 4, 6, 8 and 8).
 *   ceil(N / 128) super-slabs of 128 columns (padding columns are zero),
 *   each the steps in order, a step being the chunks of its eight 16-column
 *   slabs (slab n at n * C) of C bytes.  Weight codes: a 3/4-bit mantissa
 *   is the FP6 code s|k (s = 32 if q < 0, k = |q|), e2m3 for 3-bit blocks
 *   (the value q/8) and e3m2 for 4-bit blocks (q/16); a 6-bit mantissa,
 *   |q| = 8h + l, is two e3m2 codes s|h and s|l (h/16 and l/16, the GEMM
 *   scaling the high plane by 2^3); an 8-bit mantissa is one byte, sign-
 *   magnitude s|(|q|) (s = 128) under the symmetric clamp and two's
 *   complement under the full clamp, read as the e4m3 codes of its high
 *   nibble h (signed, scaled by 2^4) and its low nibble l (sign-magnitude:
 *   |q| = 16h + l; two's complement: q = 16h + l, 0 <= l <= 15), h/512 and
 *   l/512.  With D0..D5 the six FP6 words of a lane (32 codes, element t at
 *   bits 6t of D0..D5), symmetric-clamp codes keep only a few bits per
 *   field and are stored "folded":
 *     fold4(D) = D0 | (D1 & 0x18618618), D2 | (D1 & 0x61861861),
 *                D3 | (D4 & 0x18618618), D5 | (D4 & 0x61861861)  (16 bytes)
 *     fold3(D) = D0 | D1 >> 1, D3 | D4 >> 1, D2 | D5 << 3 | D5 >> 31
 *     fold2(D) = D0 | D1 | D2, D3 | D4 | D5  (codes 0|h, h <= 3)
 *   and the chunks are, for lane l = 16 g + c (column c of the slab):
 *     3-bit, symmetric (C = 768): fold3 of block 4s'+g: its first two words
 *       at 8 l, its third at 512 + 4 l; full (C = 1024): fold4 at 16 l;
 *     4-bit, symmetric (C = 1024): fold4 of block 4s'+g at 16 l; full
 *       (C = 1536): D0..D3 at 16 l, D4, D5 at 1024 + 8 l;
 *     6-bit, for block 2s'+j and u = 16 j + c: fold4 of the low codes at
 *       16 u, then, symmetric (C = 768), fold2 of the high codes without
 *       their sign at 512 + 8 u (the sign is the low code's), full
 *       (C = 1024), fold4 of the high codes at 512 + 16 u;
 *     8-bit (C = 1024): block 2s'+j's 32 bytes at 32 (16 j + c).
 *   w_exp, mxq_weight_exp_bytes(fmt, N): per super-slab, per group, 2048
 *   bytes: lane l's 32 bytes at 32 l, slab n's byte for step k of the group
 *   at 8 k + n: the E of block 4s'+g (3/4-bit) or 2s'+(g >> 1) (6/8-bit) of
 *   column 16 n + c, 0 for zero blocks and missing steps.
 *   Read it back with mxq_unpack_weights.
 *
 * (C) Packed rows (mxq_quantize_rows; the KV cache of mxq_attn_decode):
 *   mxq_act_packed_bytes(fmt) bytes per row: the blocks in permuted order,
 *   block b taking 4 * m_b bytes, zero padded to a multiple of 16:
 *     3-bit: element t's 3-bit two's complement field at bits 3t..3t+2 of
 *            the block's 96-bit little-endian integer (12 bytes);
 *     4-bit: byte j holds element 2j in bits 0-3 and element 2j+1 in bits 4-7;
 *     6-bit: 16 bytes of low nibbles in the 4-bit layout, then two 32-bit
 *            words of the signed top two bits: word d covers elements
 *            16d..16d+15, its byte j holds element 16d+2j in bits 6-7,
 *            16d+2j+1 in bits 4-5, 16d+8+2j in bits 2-3, 16d+9+2j in bits 0-1;
 *     8-bit: one two's-complement byte per element.
 *   Exponent rows of mxq_exp_row_bytes(fmt) bytes: byte b = the E of block
 *   b, zero padded to a multiple of 16.
 */
int64_t mxq_act_packed_bytes(const mxq_fmt *fmt);
int64_t mxq_exp_row_bytes(const mxq_fmt *fmt);
int64_t mxq_act_bytes(const mxq_fmt *fmt, int64_t M);
int64_t mxq_act_exp_bytes(const mxq_fmt *fmt, int64_t M);
int64_t mxq_weight_bytes(const mxq_fmt *fmt, int64_t N);
int64_t mxq_weight_exp_bytes(const mxq_fmt *fmt, int64_t N);

/*
 * Online activation quantization (paper: Section 5, activations of every
 * decoder linear are quantized to MXINT; Section 4.1 widths), into the
 * GEMM's operand image (layout (A) above).
 *   a       DEVICE bf16 [M][lda], lda >= K, read only.
 *   a_mant  DEVICE uint8 [mxq_act_bytes(fmt, M)], written.
 *   a_exp   DEVICE uint8 [mxq_act_exp_bytes(fmt, M)], written.
 */
mxq_status mxq_quantize_act(const mxq_fmt *fmt, const uint16_t *a, int64_t M,
                            int64_t lda, uint8_t *a_mant, uint8_t *a_exp,
                            void *stream);

/*
 * The same quantizer writing packed rows (layout (C) above; paper Appendix
 * A.2: the KV cache is quantized to MXINT as well): the rows that
 * mxq_attn_decode reads, and the input of mxq_unpack_act and
 * mxq_gemm_partials.
 *   a       DEVICE bf16 [M][lda], lda >= K, read only.
 *   rows    DEVICE uint8 [M * mxq_act_packed_bytes(fmt)], written.
 *   exps    DEVICE uint8 [M * mxq_exp_row_bytes(fmt)], written.
 * Errors: as mxq_quantize_act.
 */
mxq_status mxq_quantize_rows(const mxq_fmt *fmt, const uint16_t *a, int64_t M,
                             int64_t lda, uint8_t *rows, uint8_t *exps,
                             void *stream);

/*
 * The activation quantizer fused with its producer, RMS normalisation (the
 * paper keeps normalisation layers in 16-bit floating point, Appendix A.2,
 * and quantizes the inputs of every decoder linear): the rows of x are
 * normalised and then quantized exactly as mxq_quantize_act quantizes its
 * input.  Per row, ms = sum of x^2 / K in float64 (each 32-element block in
 * order, then the blocks in order); r = float32(1 / sqrt(ms + eps)) with the
 * root and the division in IEEE float64; y = bf16(gain * bf16(x * r)) with
 * float32 products and round-to-nearest-even.  The normalised rows are not
 * written.
 *   x     DEVICE bf16 [M][ldx], ldx >= K, read only.
 *   gain  DEVICE bf16 [K], 16-byte aligned, read only.
 *   eps   >= 0.
 *   a_mant, a_exp as for mxq_quantize_act, written.
 * Errors: as mxq_quantize_act, plus MXQ_ERR_NULL for a null gain and
 * MXQ_ERR_SHAPE for a negative or NaN eps.
 */
mxq_status mxq_quantize_act_rmsnorm(const mxq_fmt *fmt, const uint16_t *x,
                                    int64_t M, int64_t ldx,
                                    const uint16_t *gain, float eps,
                                    uint8_t *a_mant, uint8_t *a_exp,
                                    void *stream);

/*
 * The activation quantizer fused with the down projection's producer,
 * SiLU(gate) * up: the rows y = bf16(bf16(silu(g)) * u) (float32 product,
 * round-to-nearest-even) are quantized exactly as mxq_quantize_act
 * quantizes its input, without being written.  silu(g) = g / (1 + e^-g) in
 * float32 with a fixed evaluation of e^t, so that every machine gets the same
 * bits: t clamped to [-120, 120], k = rint(t * 0x3FB8AA3B), r = (t - k *
 * 0x3F317200) - k * 0x35BFBE8E (float32 bit patterns of 1/ln2 and of ln2
 * split in two), the degree-7 Taylor polynomial of e^r by Horner's rule,
 * then 2^k; every operation rounded on its own, no fused multiply-add.  A
 * NaN gate gives a NaN.
 *   gate, up  DEVICE bf16 [M][ld], ld >= K, 16-byte aligned, read only.
 *   a_mant, a_exp as for mxq_quantize_act, written.
 * Errors: as mxq_quantize_act, plus MXQ_ERR_NULL for a null up.
 */
mxq_status mxq_quantize_act_swiglu(const mxq_fmt *fmt, const uint16_t *gate,
                                   const uint16_t *up, int64_t M, int64_t ld,
                                   uint8_t *a_mant, uint8_t *a_exp,
                                   void *stream);

/*
 * Offline weight quantization and packing (same quantizer as the
 * activations; paper Section 5: weights of every decoder linear).
 *   w       DEVICE bf16 [N][ldw] (torch.nn.Linear layout: row j is output
 *           column j), ldw >= K.
 *   w_mant  DEVICE uint8 [mxq_weight_bytes(fmt, N)], written.
 *   w_exp   DEVICE uint8 [mxq_weight_exp_bytes(fmt, N)], written.
 */
mxq_status mxq_pack_weights(const mxq_fmt *fmt, const uint16_t *w, int64_t N,
                            int64_t ldw, uint8_t *w_mant, uint8_t *w_exp,
                            void *stream);

/*
 * MXINT GEMM, Y = Ahat * What^T in fp32 (paper Sections 2 and 6: integer
 * block products, power-of-two block scales).
 *   a_mant/a_exp  DEVICE, from mxq_quantize_act (or its fused variants) with
 *                 the same fmt and at least M rows.
 *   w_mant/w_exp  DEVICE, from mxq_pack_weights with the same fmt and N.
 *   y             DEVICE float [M][ldy], ldy >= N; every y[i][j] with i < M,
 *                 j < N is written, nothing else.
 * M <= MXQ_DECODE_MAX_M runs the weight-streaming decode kernel (each
 * weight step read once for all ceil(M / 16) activation tiles), larger M
 * the tiled prefill kernel; both read the same buffers.  The weights' high
 * digit planes take the scale E + 3 (6-bit) or E + 4 (8-bit), which the
 * E8M0 format holds up to 254: a 6-bit weight block with E >= 252 or an
 * 8-bit one with E >= 251 (|w| >= 2^124) makes the outputs it touches NaN.
 * Errors: MXQ_ERR_SHAPE also when sixteen 16-row activation tiles or a
 * weight super-slab exceed 2^31 - 1 bytes (K of about four million or more).
 */
mxq_status mxq_gemm(const mxq_fmt *fmt, int64_t M, int64_t N,
                    const uint8_t *a_mant, const uint8_t *a_exp,
                    const uint8_t *w_mant, const uint8_t *w_exp, float *y,
                    int64_t ldy, void *stream);

/*
 * Debug / parity entry points (not on the hot path; they restate Section 2's
 * block arithmetic one element at a time).
 * mxq_unpack_act: packed rows and exponent rows (mxq_quantize_rows) ->
 *   mantissas q DEVICE int8 [rows][K] (permuted order) and exponents e
 *   DEVICE uint8 [rows][K/32].
 * mxq_unpack_weights: the same from mxq_pack_weights' buffers.
 * mxq_gemm_partials: the exact per-block integer sums
 *   P[i][j][b] = sum_t qa[i][32b+t] * qw[j][32b+t] (Section 2's integer
 *   block product) as p DEVICE int32 [M][N][K/32], one thread per sum, from
 *   packed rows (a_mant/a_exp as written by mxq_quantize_rows for M rows)
 *   and the packed weights.
 */
mxq_status mxq_unpack_act(const mxq_fmt *fmt, int64_t rows,
                          const uint8_t *a_mant, const uint8_t *a_exp,
                          int8_t *q, uint8_t *e, void *stream);
mxq_status mxq_unpack_weights(const mxq_fmt *fmt, int64_t N,
                              const uint8_t *w_mant, const uint8_t *w_exp,
                              int8_t *q, uint8_t *e, void *stream);
mxq_status mxq_gemm_partials(const mxq_fmt *fmt, int64_t M, int64_t N,
                             const uint8_t *a_mant, const uint8_t *a_exp,
                             const uint8_t *w_mant, const uint8_t *w_exp,
                             int32_t *p, void *stream);

/*
 * Calibration: the offline step that produces a linear's permutation and
 * width map from calibration activations (paper: Section 3, Algorithm 1;
 * Section 4.2, Algorithm 2; Appendix A, Theorem A.1).
 *   mxq_calib_colsq: column sensitivities of one calibration sample,
 *     diag(X^T X): s[k] = sum over the rows of x[r][k]^2 in float64, the
 *     rows summed in row order from zero; with `accumulate` the sample's sum
 *     is added to s[k] (samples in call order), else it replaces it.
 *     x DEVICE bf16 [rows][ldx], ldx >= K, read; s DEVICE double [K].
 *   mxq_calib_colsq_samples: the same for n_samples samples at once (sample
 *     i at x + i * sample_stride elements, sample_stride >= rows * ldx):
 *     each sample's sums go to row i of `work` (DEVICE double
 *     [n_samples][K], caller-owned scratch), then are added to s in sample
 *     order, so the result equals n_samples calls of mxq_calib_colsq.
 *     n_samples in [1, 65535].
 *   mxq_calib_ratio (HOST only): Theorem A.1's control parameter
 *     R = ((B - 4) * sum d_i - 4 * 32 * n) / sum(2 * S_i * (d_i - 32)) for n
 *     layers of input widths d_in[i] (multiples of 32) and layer
 *     sensitivities s_layer[i], so that 32 8-bit columns per layer and
 *     R * S_i * (d_i - 32) 6-bit ones average B bits.  Sums in layer order.
 *   mxq_calib_counts (HOST only): Algorithm 2's split of a layer of d_in
 *     columns into 32-column blocks: n8 = n8_blocks (the paper: 1), n6 =
 *     floor(R * s_layer * (d_in - 32)) columns rounded down to whole blocks
 *     and clamped to [0, d_in / 32 - n8], n4 the rest.
 *   mxq_calib_perm: the permutation of Algorithm 2: columns sorted by
 *     descending s (equal values in column order, NaN as +inf); the first
 *     32 * n8_blocks are 8-bit, the next 32 * n6_blocks 6-bit, the rest
 *     4-bit; perm lists the 4-bit columns, then the 6-bit, then the 8-bit,
 *     each in sorted order, matching the width map [4]*n4 + [6]*n6 + [8]*n8.
 *     s DEVICE double [K], read; perm DEVICE int32 [K], written; K a
 *     multiple of 32.
 * Errors: MXQ_ERR_NULL (null pointer), MXQ_ERR_SHAPE (rows < 0, K <= 0,
 * ldx < K, widths not multiples of 32, block counts out of range, or a zero
 * denominator in R), MXQ_ERR_DEVICE (launch).  Device work is enqueued on
 * `stream`; nothing is allocated.
 */
mxq_status mxq_calib_colsq(const uint16_t *x, int64_t rows, int64_t ldx,
                           int64_t K, double *s, int accumulate, void *stream);
mxq_status mxq_calib_colsq_samples(const uint16_t *x, int64_t n_samples,
                                   int64_t rows, int64_t ldx,
                                   int64_t sample_stride, int64_t K,
                                   double *work, double *s, int accumulate,
                                   void *stream);
mxq_status mxq_calib_ratio(int32_t n, const int64_t *d_in,
                           const double *s_layer, double B, double *R);
mxq_status mxq_calib_counts(int64_t d_in, double R, double s_layer,
                            int32_t n8_blocks, int32_t *n4, int32_t *n6,
                            int32_t *n8);
mxq_status mxq_calib_perm(const double *s, int64_t K, int32_t n6_blocks,
                          int32_t n8_blocks, int32_t *perm, void *stream);

/*
 * Achievable-peak microbenchmarks, for the benchmark's roofline figures (not
 * part of the quantize / GEMM path; the paper states no peaks, these price
 * the kernels against what the same box reaches).
 *   mxq_peak_sink_words: length, in 4-byte words, of the sink both take.
 *   mxq_peak_stream_read: reads each of the `bytes` (a positive multiple of
 *     16) of DEVICE buffer `buf` once, with 16-byte non-temporal loads;
 *     `sink` DEVICE uint32 [mxq_peak_sink_words()], written (a checksum).
 *   mxq_peak_mfma: register-resident matrix-core loop, `iters` products per
 *     accumulator, eight accumulators per wave, sixteen waves per CU; kind
 *     0 = dense int8 32x32x32, 1 = block-scaled FP6 e3m2 32x32x64, 2 =
 *     block-scaled FP8 e4m3 32x32x64.  `*ops` (HOST) receives the
 *     multiply-add ops (2 per product term) one launch performs; `sink`
 *     DEVICE float [mxq_peak_sink_words()], written.
 * Errors: MXQ_ERR_NULL (null pointer), MXQ_ERR_SHAPE (bytes not a positive
 * multiple of 16, iters < 1, kind outside 0..2), MXQ_ERR_DEVICE (launch).
 * Enqueued on `stream`; nothing is allocated.
 */
int64_t mxq_peak_sink_words(void);
mxq_status mxq_peak_stream_read(const void *buf, int64_t bytes, uint32_t *sink,
                                void *stream);
mxq_status mxq_peak_mfma(int kind, int64_t iters, float *sink, int64_t *ops,
                         void *stream);

/*
 * Decode attention over an MXINT KV cache (MXSens Appendix A.2: K and V are
 * quantized to MXINT with 32-element blocks along the head dimension, 4 to 8
 * bits per block, and attention reads them).  One new token per sequence:
 * for sequence b and query head h, with KV head k = h / G (G = Hq / Hkv),
 *   s_t = scale * sum_d q[b][h][d] * K[b][t][k][d]   (t = 0..T-1),
 *   o[b][h][d] = sum_t softmax(s)_t * V[b][t][k][d],
 * where K and V are the dequantized cache values q * 2^(E - 127 - (m - 2)).
 * Arithmetic is float32: each block's dot product, then its scale; an
 * online softmax over chunks of 64 tokens; partial results merged in a
 * fixed order, so repeated calls give identical results.
 *   fmt     the cache format: K = 128 (the head dimension), perm NULL,
 *           widths as for mxq_quantize_act (round and clamp do not matter
 *           here).
 *   q       DEVICE bf16 [B][Hq][128], 16-byte aligned, read only.
 *   B >= 0 (0: nothing to do), Hkv >= 1, Hq a multiple of Hkv with
 *   Hq / Hkv <= 16, T >= 1.
 *   scale   finite (usually 1 / sqrt(128)).
 *   k_mant, v_mant   DEVICE, 16-byte aligned: packed rows of
 *           mxq_act_packed_bytes(fmt) bytes (layout (C) above), row
 *           (b * T + t) * Hkv + k; the rows written by mxq_quantize_rows
 *           for M = B * T * Hkv rows of [.][128] serve as they are.  Read
 *           only.
 *   k_exp, v_exp     DEVICE, 16-byte aligned: exponent rows of
 *           mxq_exp_row_bytes(fmt) bytes, same row order (mxq_quantize_rows'
 *           exps).  Read only.
 *   o       DEVICE float32 [B][Hq][128], written.
 *   work    DEVICE, 16-byte aligned, work_bytes >= mxq_attn_work_bytes(...):
 *           the caller's scratch for per-split partial results; its
 *           contents need no initialisation and are overwritten.
 * Errors: check_fmt's errors; MXQ_ERR_SHAPE for K != 128, a bad count, a
 * non-finite scale or a short work buffer; MXQ_ERR_UNSUPPORTED for a
 * permutation; MXQ_ERR_NULL; MXQ_ERR_ALIGN; MXQ_ERR_DEVICE on a failed
 * launch.  Asynchronous on `stream`.
 * mxq_attn_work_bytes returns the work size in bytes, or a negative
 * mxq_status for invalid arguments.
 */
int64_t mxq_attn_work_bytes(const mxq_fmt *fmt, int64_t B, int64_t Hq, int64_t Hkv, int64_t T);
mxq_status mxq_attn_decode(const mxq_fmt *fmt, const uint16_t *q, int64_t B, int64_t Hq,
                           int64_t Hkv, int64_t T, float scale, const uint8_t *k_mant,
                           const uint8_t *k_exp, const uint8_t *v_mant, const uint8_t *v_exp,
                           float *o, float *work, int64_t work_bytes, void *stream);

/*
 * mxq_attn_decode without a work buffer, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Arguments, results and errors are those
 * of mxq_attn_decode (the same kernels, split the same way, so the outputs
 * are identical), except that the per-split partial results live in a
 * static device array of MXQ_ATTN_STATIC_WORK_BYTES per GPU, held from the
 * library's first such call on that GPU until the process ends.  Calls whose
 * mxq_attn_work_bytes exceeds MXQ_ATTN_STATIC_WORK_BYTES return
 * MXQ_ERR_SCRATCH before anything is enqueued (B * Hq * splits * 520 bytes;
 * about 2.1 MB for 64 query heads at any batch up to 16).  Every call on one
 * GPU shares that GPU's array: calls that may overlap in time on one GPU
 * (different streams, or different threads without ordering) race and must
 * be serialised by the caller.  Nothing is allocated or freed, and no
 * memory is set: the kernels overwrite the scratch they read.
 */
#define MXQ_ATTN_STATIC_WORK_BYTES (8LL << 20)
mxq_status mxq_attn_decode_static(const mxq_fmt *fmt, const uint16_t *q, int64_t B, int64_t Hq,
                                  int64_t Hkv, int64_t T, float scale, const uint8_t *k_mant,
                                  const uint8_t *k_exp, const uint8_t *v_mant,
                                  const uint8_t *v_exp, float *o, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* MXQ_H */
