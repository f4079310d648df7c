/*
 * mxq_oracle.c -- reference CPU implementation of mixed-mantissa MXINT
 * quantization and the blockwise MXINT GEMM.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file.  Its only users are the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark.  It shares no code, header, table or
 * helper with the GPU library: every step below is written out from the
 * paper's description of the format, in double precision, with plain loops.
 *
 * Paper: MXSens -- Sensitivity-Aware Mixed-Precision Quantization (arXiv
 * 2607.17733).
 *   - Section 2 (Background): a microscaling block of 32 values shares one
 *     power-of-two scale encoded as an exponent; MXINT elements are
 *     fixed-point integers, so a block dot product is an integer
 *     multiply-accumulate followed by a power-of-two scaling.
 *   - Section 1 (Introduction): shared power-of-two scale per block of 32.
 *   - Section 4.1 (Triplet quantization): each block carries exactly one
 *     mantissa width out of {4, 6, 8}; same-width columns fill whole blocks.
 *   - Section 5 (average-bitwidth study, the LLaMA-2-7B table): a second
 *     template uses MXINT3 in place of MXINT4 (widths {3, 6, 8}); a 3-bit
 *     block follows the same rules with m = 3.  Its storage follows its
 *     bits (the table's average bitwidths count 3 bits per element): 12
 *     bytes per block in the packed-row layout.
 *   - Section 5.1 (MXSens results): the exponent is 8 bits per 32 elements,
 *     i.e. +0.25 bit per element; the widths therefore count storage bits,
 *     sign included (also the bit accounting in the proof of Theorem A.1).
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - shared exponent e = floor(log2(max |x|)) over the block, clamped to
 *     [-127, 127] and stored as E = e + 127 (E8M0); an all-zero block has
 *     E = 0 and zero mantissas; a block holding NaN or Inf has E = 255 and
 *     zero mantissas, and every GEMM output touching it is NaN;
 *   - the least significant mantissa bit weighs 2^(e - (m - 2)), i.e. one
 *     integer bit before the binary point as in OCP MXINT8;
 *   - rounding to nearest with ties to even (default) or ties away from zero;
 *   - clamping to the symmetric range +-(2^(m-1) - 1) (default) or to the
 *     full two's-complement range [-2^(m-1), 2^(m-1) - 1].
 *
 * The oracle never uses log2(): the exponent comes from frexp(), which is
 * exact, and the scaling by 2^-s is ldexp(), also exact in double for every
 * bf16 input.
 */
#include <fenv.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_BLOCK 32

/* bf16 bit pattern -> exact double. */
static double bf16_to_double(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Quantize one block of 32 values (already gathered in permuted order).
 * Writes 32 mantissas and returns the stored exponent byte E. */
static uint8_t quantize_block(const double *x, int m, int round_mode,
                              int clamp_mode, int8_t *q) {
  double amax = 0.0;
  int special = 0;
  for (int t = 0; t < ORACLE_BLOCK; ++t) {
    if (isnan(x[t]) || isinf(x[t])) special = 1;
    double a = fabs(x[t]);
    if (a > amax) amax = a;
  }
  if (special) {                 /* E8M0 NaN encoding; mantissas zero */
    for (int t = 0; t < ORACLE_BLOCK; ++t) q[t] = 0;
    return 255;
  }
  if (amax == 0.0) {             /* zero block */
    for (int t = 0; t < ORACLE_BLOCK; ++t) q[t] = 0;
    return 0;
  }
  int ex;
  (void)frexp(amax, &ex);        /* amax = f * 2^ex, f in [0.5, 1) */
  int e = ex - 1;                /* floor(log2(amax)) */
  if (e < -127) e = -127;
  if (e > 127) e = 127;
  int s = e - (m - 2);           /* weight of the mantissa LSB */
  long qmax = (1L << (m - 1)) - 1;
  long qmin = clamp_mode == 1 ? -(1L << (m - 1)) : -qmax;
  for (int t = 0; t < ORACLE_BLOCK; ++t) {
    double v = ldexp(x[t], -s);  /* exact */
    double r = round_mode == 1 ? round(v) : nearbyint(v);
    long qi = (long)r;
    if (qi > qmax) qi = qmax;
    if (qi < qmin) qi = qmin;
    q[t] = (int8_t)qi;
  }
  return (uint8_t)(e + 127);
}

static int width_ok(int m) { return m == 3 || m == 4 || m == 6 || m == 8; }

/*
 * Quantize `rows` rows of a bf16 matrix (row stride `ld` elements) along K.
 * perm[p] is the source column placed at position p (NULL = identity).
 * widths[b] is the mantissa width of block b (K/32 entries).
 * Outputs: q[rows][K] mantissas in permuted order, e[rows][K/32] exponents.
 * Returns 0 on success, nonzero on invalid arguments.
 */
int oracle_quantize(const uint16_t *x, int64_t rows, int64_t ld, int64_t K,
                    const int32_t *perm, const uint8_t *widths, int round_mode,
                    int clamp_mode, int8_t *q, uint8_t *e) {
  if (K <= 0 || K % ORACLE_BLOCK != 0 || rows < 0 || ld < K) return 1;
  int64_t nb = K / ORACLE_BLOCK;
  for (int64_t b = 0; b < nb; ++b)
    if (!width_ok(widths[b])) return 2;
  fesetround(FE_TONEAREST);
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    double blk[ORACLE_BLOCK];
    for (int64_t b = 0; b < nb; ++b) {
      for (int t = 0; t < ORACLE_BLOCK; ++t) {
        int64_t p = b * ORACLE_BLOCK + t;
        int64_t col = perm ? perm[p] : p;
        blk[t] = bf16_to_double(x[r * ld + col]);
      }
      e[r * nb + b] = quantize_block(blk, widths[b], round_mode, clamp_mode,
                                     q + r * K + b * ORACLE_BLOCK);
    }
  }
  return 0;
}

/* Dequantize: xhat[r][p] = q * 2^(E - 127 - (m - 2)); NaN for E == 255. */
int oracle_dequantize(const int8_t *q, const uint8_t *e, int64_t rows,
                      int64_t K, const uint8_t *widths, double *xhat) {
  if (K <= 0 || K % ORACLE_BLOCK != 0) return 1;
  int64_t nb = K / ORACLE_BLOCK;
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t b = 0; b < nb; ++b) {
      int E = e[r * nb + b];
      int s = E - 127 - (widths[b] - 2);
      for (int t = 0; t < ORACLE_BLOCK; ++t) {
        int64_t p = b * ORACLE_BLOCK + t;
        xhat[r * K + p] = E == 255 ? NAN : ldexp((double)q[r * K + p], s);
      }
    }
  return 0;
}

/*
 * Per-block integer partial sums P[i][j][b] = sum_t qa[i][32b+t]*qw[j][32b+t]
 * (exact; |P| <= 32 * 128 * 128 = 2^19, stored as int32).
 */
int oracle_block_partials(const int8_t *qa, const int8_t *qw, int64_t M,
                          int64_t N, int64_t K, int32_t *P) {
  if (K <= 0 || K % ORACLE_BLOCK != 0) return 1;
  int64_t nb = K / ORACLE_BLOCK;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < M; ++i)
    for (int64_t j = 0; j < N; ++j)
      for (int64_t b = 0; b < nb; ++b) {
        int64_t acc = 0;
        for (int t = 0; t < ORACLE_BLOCK; ++t)
          acc += (int64_t)qa[i * K + b * ORACLE_BLOCK + t] *
                 (int64_t)qw[j * K + b * ORACLE_BLOCK + t];
        P[(i * N + j) * nb + b] = (int32_t)acc;
      }
  return 0;
}

/*
 * Blockwise MXINT GEMM, Y = Ahat * What^T, for a subset of outputs:
 * Y[a][c] for output row rows_idx[a] and output column cols_idx[c]
 * (NULL index arrays mean 0..nr-1 / 0..nc-1).
 *   Y[i][j] = sum_b P[i][j][b] * 2^(sa[i][b] + sw[j][b]),
 *   s = E - 127 - (m_b - 2),
 * accumulated in double in block order.  A block with E == 255 on either
 * side makes the output NaN.
 */
int oracle_gemm(const int8_t *qa, const uint8_t *ea, const int8_t *qw,
                const uint8_t *ew, const uint8_t *widths, int64_t K,
                const int64_t *rows_idx, int64_t nr, const int64_t *cols_idx,
                int64_t nc, double *Y) {
  if (K <= 0 || K % ORACLE_BLOCK != 0) return 1;
  int64_t nb = K / ORACLE_BLOCK;
#pragma omp parallel for schedule(static)
  for (int64_t a = 0; a < nr; ++a) {
    int64_t i = rows_idx ? rows_idx[a] : a;
    for (int64_t c = 0; c < nc; ++c) {
      int64_t j = cols_idx ? cols_idx[c] : c;
      double y = 0.0;
      for (int64_t b = 0; b < nb; ++b) {
        int EA = ea[i * nb + b], EW = ew[j * nb + b];
        int64_t acc = 0;
        for (int t = 0; t < ORACLE_BLOCK; ++t)
          acc += (int64_t)qa[i * K + b * ORACLE_BLOCK + t] *
                 (int64_t)qw[j * K + b * ORACLE_BLOCK + t];
        if (EA == 255 || EW == 255) {
          y = NAN;
          continue;
        }
        int sa = EA - 127 - (widths[b] - 2);
        int sw = EW - 127 - (widths[b] - 2);
        y += ldexp((double)acc, sa + sw);
      }
      Y[a * nc + c] = y;
    }
  }
  return 0;
}

/*
 * Sum over blocks of |P[i][j][b]| * 2^(sa + sw) for the same subset of
 * outputs: the magnitude that bounds any fp32 summation order of the
 * blockwise products (used for the rounding-error bound in the tests).
 */
int oracle_gemm_absbound(const int8_t *qa, const uint8_t *ea, const int8_t *qw,
                         const uint8_t *ew, const uint8_t *widths, int64_t K,
                         const int64_t *rows_idx, int64_t nr,
                         const int64_t *cols_idx, int64_t nc, double *S) {
  if (K <= 0 || K % ORACLE_BLOCK != 0) return 1;
  int64_t nb = K / ORACLE_BLOCK;
#pragma omp parallel for schedule(static)
  for (int64_t a = 0; a < nr; ++a) {
    int64_t i = rows_idx ? rows_idx[a] : a;
    for (int64_t c = 0; c < nc; ++c) {
      int64_t j = cols_idx ? cols_idx[c] : c;
      double s = 0.0;
      for (int64_t b = 0; b < nb; ++b) {
        int64_t acc = 0;
        for (int t = 0; t < ORACLE_BLOCK; ++t)
          acc += (int64_t)qa[i * K + b * ORACLE_BLOCK + t] *
                 (int64_t)qw[j * K + b * ORACLE_BLOCK + t];
        int sa = ea[i * nb + b] - 127 - (widths[b] - 2);
        int sw = ew[j * nb + b] - 127 - (widths[b] - 2);
        s += ldexp((double)(acc < 0 ? -acc : acc), sa + sw);
      }
      S[a * nc + c] = s;
    }
  }
  return 0;
}

/*
 * Packed storage of quantized activations, written byte by byte from the
 * documented layout (the GPU's packed output is compared to this):
 *   row r starts at r * row_bytes, row_bytes = 16*n4 + 24*n6 + 32*n8
 *   rounded up to a multiple of 16; blocks follow the permuted order;
 *   - 4-bit block (16 bytes): byte j holds element 2j in bits 0-3 and
 *     element 2j+1 in bits 4-7 (two's complement nibbles);
 *   - 6-bit block (24 bytes): bytes 0-15 hold the low 4 bits of each element
 *     in the 4-bit layout; bytes 16-23 hold the signed top 2 bits as two
 *     words, word d (d = 0, 1) covering elements 16d..16d+15: byte j of word
 *     d has element 16d+2j in bits 6-7, 16d+2j+1 in bits 4-5, 16d+8+2j in
 *     bits 2-3 and 16d+9+2j in bits 0-1;
 *   - 8-bit block (32 bytes): one two's-complement byte per element.
 * Padding bytes are zero.
 */
int64_t oracle_act_row_bytes(const uint8_t *widths, int64_t nb) {
  int64_t bytes = 0;
  /* 32 mantissas of m bits: 4 m bytes per block (12 for the 3-bit blocks) */
  for (int64_t b = 0; b < nb; ++b) bytes += 4 * (int64_t)widths[b];
  return (bytes + 15) / 16 * 16;
}

int oracle_pack_act(const int8_t *q, int64_t rows, int64_t K,
                    const uint8_t *widths, uint8_t *out) {
  if (K <= 0 || K % ORACLE_BLOCK != 0) return 1;
  int64_t nb = K / ORACLE_BLOCK;
  int64_t rb = oracle_act_row_bytes(widths, nb);
  memset(out, 0, (size_t)(rows * rb));
  for (int64_t r = 0; r < rows; ++r) {
    uint8_t *row = out + r * rb;
    int64_t off = 0;
    for (int64_t b = 0; b < nb; ++b) {
      const int8_t *v = q + r * K + b * ORACLE_BLOCK;
      int m = widths[b];
      uint8_t *blk = row + off;
      if (m == 8) {
        for (int t = 0; t < 32; ++t) blk[t] = (uint8_t)v[t];
      } else if (m == 3) {
        /* 96 bits, little-endian: element t's 3-bit two's complement field
           at bits 3t .. 3t + 2 */
        for (int t = 0; t < 32; ++t) {
          unsigned f = (unsigned)v[t] & 7u;
          for (int k = 0; k < 3; ++k)
            if ((f >> k) & 1u) blk[(3 * t + k) / 8] |= (uint8_t)(1u << ((3 * t + k) % 8));
        }
      } else {
        /* low nibble plane (the whole mantissa when m == 4) */
        for (int j = 0; j < 16; ++j) {
          unsigned lo = (unsigned)v[2 * j] & 15u;
          unsigned hi = (unsigned)v[2 * j + 1] & 15u;
          blk[j] = (uint8_t)(lo | (hi << 4));
        }
        if (m == 6) {
          for (int d = 0; d < 2; ++d)
            for (int j = 0; j < 4; ++j) {
              /* top two bits of the 6-bit two's complement field */
              unsigned h0 = ((unsigned)v[16 * d + 2 * j] & 63u) >> 4;
              unsigned h1 = ((unsigned)v[16 * d + 2 * j + 1] & 63u) >> 4;
              unsigned h2 = ((unsigned)v[16 * d + 8 + 2 * j] & 63u) >> 4;
              unsigned h3 = ((unsigned)v[16 * d + 9 + 2 * j] & 63u) >> 4;
              blk[16 + 4 * d + j] =
                  (uint8_t)((h0 << 6) | (h1 << 4) | (h2 << 2) | h3);
            }
        }
      }
      off += 4 * m;
    }
  }
  return 0;
}

/* Number of threads the OpenMP loops above use (1 without OpenMP). */
int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads for the OpenMP loops above (timing of the oracle at a stated core
 * count); a no-op without OpenMP. */
void oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
