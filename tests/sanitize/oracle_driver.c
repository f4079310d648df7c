/* Driver of the C oracle for the sanitizer build (test infrastructure).
 * Built with gcc -fsanitize=address,undefined and run on small inputs of
 * every width, round and clamp mode, ragged row and column counts, special
 * values (zero, subnormal, huge, Inf, NaN blocks) and the rejection of bad
 * shapes: any out-of-bounds access, overflow or undefined shift aborts. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_quantize(const uint16_t *x, int64_t rows, int64_t ld, int64_t K, const int32_t *perm,
                    const uint8_t *widths, int round_mode, int clamp_mode, int8_t *q, uint8_t *e);
int oracle_dequantize(const int8_t *q, const uint8_t *e, int64_t rows, int64_t K,
                      const uint8_t *widths, double *xhat);
int oracle_block_partials(const int8_t *qa, const int8_t *qw, int64_t M, int64_t N, int64_t K,
                          int32_t *P);
int oracle_gemm(const int8_t *qa, const uint8_t *ea, const int8_t *qw, const uint8_t *ew,
                const uint8_t *widths, int64_t K, const int64_t *rows_idx, int64_t nr,
                const int64_t *cols_idx, int64_t nc, double *Y);
int oracle_gemm_absbound(const int8_t *qa, const uint8_t *ea, const int8_t *qw,
                         const uint8_t *ew, const uint8_t *widths, int64_t K,
                         const int64_t *rows_idx, int64_t nr, const int64_t *cols_idx,
                         int64_t nc, double *S);
int64_t oracle_act_row_bytes(const uint8_t *widths, int64_t nb);
int oracle_pack_act(const int8_t *q, int64_t rows, int64_t K, const uint8_t *widths,
                    uint8_t *out);

static uint32_t rng = 12345u;
static uint32_t next(void) {
  rng ^= rng << 13;
  rng ^= rng >> 17;
  rng ^= rng << 5;
  return rng;
}

static int run(int64_t M, int64_t N, const uint8_t *widths, int64_t nb, int round_mode,
               int clamp_mode, int with_perm) {
  const int64_t K = 32 * nb, ld = K + 3;
  uint16_t *a = malloc(sizeof(uint16_t) * M * ld), *w = malloc(sizeof(uint16_t) * N * ld);
  int32_t *perm = malloc(sizeof(int32_t) * K);
  int8_t *qa = malloc(M * K), *qw = malloc(N * K);
  uint8_t *ea = malloc(M * nb), *ew = malloc(N * nb);
  double *xa = malloc(sizeof(double) * M * K), *Y = malloc(sizeof(double) * M * N),
         *S = malloc(sizeof(double) * M * N);
  int32_t *P = malloc(sizeof(int32_t) * M * N * nb);
  uint8_t *packed = malloc(M * oracle_act_row_bytes(widths, nb));
  int64_t *ri = malloc(sizeof(int64_t) * M), *ci = malloc(sizeof(int64_t) * N);
  for (int64_t i = 0; i < M * ld; ++i) a[i] = (uint16_t)next();      /* any bit pattern */
  for (int64_t i = 0; i < N * ld; ++i) w[i] = (uint16_t)(next() & 0xBFFFu);
  if (M > 2) {
    for (int64_t k = 0; k < K; ++k) a[0 * ld + k] = 0;                /* a zero row */
    a[1 * ld + 3] = 0x7F80u;                                          /* +Inf */
    a[2 * ld + 5] = 0x7FC1u;                                          /* NaN */
  }
  for (int64_t k = 0; k < K; ++k) perm[k] = (int32_t)((k * 7 + 3) % K);
  int rc = 0;
  rc |= oracle_quantize(a, M, ld, K, with_perm ? perm : NULL, widths, round_mode, clamp_mode,
                        qa, ea);
  rc |= oracle_quantize(w, N, ld, K, with_perm ? perm : NULL, widths, round_mode, clamp_mode,
                        qw, ew);
  rc |= oracle_dequantize(qa, ea, M, K, widths, xa);
  rc |= oracle_block_partials(qa, qw, M, N, K, P);
  rc |= oracle_gemm(qa, ea, qw, ew, widths, K, NULL, M, NULL, N, Y);
  rc |= oracle_gemm_absbound(qa, ea, qw, ew, widths, K, NULL, M, NULL, N, S);
  for (int64_t i = 0; i < M; ++i) ri[i] = M - 1 - i;
  for (int64_t j = 0; j < N; ++j) ci[j] = (j * 5) % N;
  rc |= oracle_gemm(qa, ea, qw, ew, widths, K, ri, M, ci, N, Y);
  rc |= oracle_gemm_absbound(qa, ea, qw, ew, widths, K, ri, M, ci, N, S);
  rc |= oracle_pack_act(qa, M, K, widths, packed);
  free(a); free(w); free(perm); free(qa); free(qw); free(ea); free(ew); free(xa); free(Y);
  free(S); free(P); free(packed); free(ri); free(ci);
  return rc;
}

int main(void) {
  static const uint8_t maps[][8] = {{3, 3, 4, 6, 8, 8, 8, 8}, {4, 4, 4, 4, 4, 4, 6, 8},
                                    {3, 3, 3, 3, 3, 3, 3, 3}, {8, 8, 8, 8, 8, 8, 8, 8},
                                    {6, 6, 6, 6, 6, 6, 6, 6}};
  int failures = 0;
  for (int m = 0; m < 5; ++m)
    for (int nb = 1; nb <= 8; nb += 3)
      for (int mode = 0; mode < 4; ++mode)
        failures += run(5 + nb, 3 + mode, maps[m], nb, mode & 1, mode >> 1, (m + nb) & 1) != 0;
  /* rejected shapes touch nothing */
  uint8_t w4[1] = {4};
  failures += oracle_quantize(NULL, 1, 31, 31, NULL, w4, 0, 0, NULL, NULL) == 0;
  failures += oracle_pack_act(NULL, 1, 33, w4, NULL) == 0;
  if (failures) {
    fprintf(stderr, "%d oracle run(s) failed\n", failures);
    return 1;
  }
  printf("oracle driver: ok\n");
  return 0;
}
