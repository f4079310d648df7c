// api.cpp -- the C ABI of libmxq (declared in include/mxq.h): argument
// validation, width-map segment derivation and kernel dispatch.  Every check
// happens before anything is enqueued; nothing here allocates, frees or
// synchronizes.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "../../include/mxq.h"
#include "mxq_device.h"
#include "mxq_internal.h"

namespace {

using mxq::Segs;

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

constexpr int64_t kWeightTailPad = 64;

// Validate a format and derive its width segments (MXSens Section 4.1: one
// width per block; the permutation groups same-width columns, ordered
// 4-bit, 6-bit, 8-bit).
mxq_status check_fmt(const mxq_fmt *f, Segs *s) {
  if (!f) return MXQ_ERR_NULL;
  if (f->block != MXQ_BLOCK) return MXQ_ERR_UNSUPPORTED;
  if (f->round != MXQ_ROUND_NEAREST_EVEN && f->round != MXQ_ROUND_NEAREST_AWAY)
    return MXQ_ERR_UNSUPPORTED;
  if (f->clamp != MXQ_CLAMP_SYMMETRIC && f->clamp != MXQ_CLAMP_FULL)
    return MXQ_ERR_UNSUPPORTED;
  if (f->reserved != 0) return MXQ_ERR_UNSUPPORTED;
  if (f->K <= 0 || f->K % MXQ_BLOCK != 0) return MXQ_ERR_SHAPE;
  if (f->K / MXQ_BLOCK > (int64_t)(1 << 24)) return MXQ_ERR_SHAPE;
  if (!f->widths) return MXQ_ERR_NULL;
  if (f->perm && !aligned16(f->perm)) return MXQ_ERR_ALIGN;
  const int64_t nb = f->K / MXQ_BLOCK;
  int n[3] = {0, 0, 0};
  int n3 = 0;
  int prev = 0;
  for (int64_t b = 0; b < nb; ++b) {
    const int m = f->widths[b];
    if (m != 3 && m != 4 && m != 6 && m != 8) return MXQ_ERR_WIDTHS;
    if (m < prev) return MXQ_ERR_WIDTHS;
    prev = m;
    if (m == 3) ++n3;
    ++n[m == 3 ? 0 : (m - 4) / 2];
  }
  s->n4 = n[0];
  s->n6 = n[1];
  s->n8 = n[2];
  s->n3 = n3;
  return MXQ_OK;
}

int64_t row_used(const Segs &s) { return mxq::packed_row_used(s); }
// packed section and per-row exponent section
int64_t canon_rb(const Segs &s) { return round_up(row_used(s), 16); }
int64_t exp_rb(const mxq_fmt *f) { return round_up(f->K / MXQ_BLOCK, 16); }
mxq::LGeo l_geo(const Segs &s) { return mxq::LGeo(s.n3, s.n4, s.n6, s.n8); }
bool full_clamp(const mxq_fmt *f) { return f->clamp == MXQ_CLAMP_FULL; }
// activation operand image: 16-row tiles, and their scale words
int64_t act_tiles(int64_t M) { return (M + mxq::kATileRows - 1) / mxq::kATileRows; }
int64_t act_bytes(const Segs &s, int64_t M) { return act_tiles(M) * mxq::a_tile_bytes(l_geo(s)); }
int64_t act_exp_bytes(const Segs &s, int64_t M) {
  return act_tiles(M) * mxq::a_tile_scale_bytes(l_geo(s));
}
// weights: 128-column super-slabs, and their scale words
int64_t w_supers(int64_t N) { return (N + mxq::kWCols - 1) / mxq::kWCols; }
int64_t w_bytes(const mxq_fmt *f, const Segs &s, int64_t N) {
  return w_supers(N) * mxq::w_super_bytes(l_geo(s), full_clamp(f));
}
int64_t w_exp_bytes(const Segs &s, int64_t N) {
  return w_supers(N) * mxq::w_super_scale_bytes(l_geo(s));
}

mxq_status launched(hipError_t e) { return e == hipSuccess ? MXQ_OK : MXQ_ERR_DEVICE; }

enum QuantKind { kWeights, kImage, kRows };

mxq_status quantize_common(const mxq_fmt *fmt, const uint16_t *src, int64_t rows,
                           int64_t ld, uint8_t *mant, uint8_t *exp, void *stream,
                           QuantKind kind, const uint16_t *gain = nullptr, float eps = 0.f,
                           const uint16_t *src2 = nullptr) {
  Segs s;
  mxq_status st = check_fmt(fmt, &s);
  if (st != MXQ_OK) return st;
  if (rows < 0 || ld < fmt->K) return MXQ_ERR_SHAPE;
  if (rows == 0) return MXQ_OK;
  if (!src || !mant || !exp) return MXQ_ERR_NULL;
  if (!aligned16(src) || !aligned16(mant) || !aligned16(exp)) return MXQ_ERR_ALIGN;
  if (gain && !aligned16(gain)) return MXQ_ERR_ALIGN;
  if (src2 && !aligned16(src2)) return MXQ_ERR_ALIGN;
  mxq::QuantArgs a{};
  a.rmsnorm = gain != nullptr;
  a.gain = gain;
  a.eps = eps;
  a.swiglu = src2 != nullptr;
  a.src2 = src2;
  a.src = src;
  a.ld = ld;
  a.src_rows = rows;
  a.K = fmt->K;
  a.perm = fmt->perm;
  a.n4 = s.n4;
  a.n6 = s.n6;
  a.n8 = s.n8;
  a.n3 = s.n3;
  a.ties_away = fmt->round == MXQ_ROUND_NEAREST_AWAY;
  a.full_clamp = full_clamp(fmt);
  a.vec16 = (ld % 8 == 0) ? 1 : 0;
  if (kind == kWeights) {
    a.out_rows = round_up(rows, mxq::kWCols);
    a.mant = mant;
    a.exp = exp;
    return launched(mxq::launch_quantize(a, true, (hipStream_t)stream));
  }
  a.canon_rb = canon_rb(s);
  a.canon_erb = exp_rb(fmt);
  a.row_used = row_used(s);
  if (kind == kRows) {
    a.write_rows = 1;
    a.out_rows = rows;
    a.mant = mant;
    a.exp = exp;
    a.out_rb = canon_rb(s);
    a.out_erb = exp_rb(fmt);
  } else {
    a.write_image = 1;
    a.out_rows = round_up(rows, mxq::kATileRows);
    a.img = mant;
    a.img_exp = exp;
    a.a_tile = mxq::a_tile_bytes(l_geo(s));
    a.a_tile_sc = mxq::a_tile_scale_bytes(l_geo(s));
  }
  // the activation quantizer stages its rows in LDS: one row must fit
  if (mxq::quantize_act_lds(fmt->K, mxq::quantize_act_padded_blocks(s.n3, s.n4, s.n6, s.n8),
                            fmt->perm != nullptr, gain != nullptr) > mxq::kMaxLds)
    return MXQ_ERR_UNSUPPORTED;
  return launched(mxq::launch_quantize_act(a, (hipStream_t)stream));
}

mxq_status gemm_args(const mxq_fmt *fmt, int64_t M, int64_t N, const uint8_t *a_mant,
                     const uint8_t *a_exp, const uint8_t *w_mant, const uint8_t *w_exp,
                     const void *out, mxq::GemmArgs *g) {
  Segs s;
  mxq_status st = check_fmt(fmt, &s);
  if (st != MXQ_OK) return st;
  if (M < 0 || N < 0) return MXQ_ERR_SHAPE;
  if (M == 0 || N == 0) return MXQ_OK;
  if (!a_mant || !a_exp || !w_mant || !w_exp || !out) return MXQ_ERR_NULL;
  if (!aligned16(a_mant) || !aligned16(a_exp) || !aligned16(w_mant) ||
      !aligned16(w_exp) || !aligned16(out))
    return MXQ_ERR_ALIGN;
  const mxq::LGeo lg = l_geo(s);
  // The prefill kernel addresses a workgroup's 256 activation rows (16
  // tiles) and one weight super-slab with 32-bit buffer offsets from a
  // 64-bit base.
  if (16 * mxq::a_tile_bytes(lg) > INT32_MAX ||
      mxq::w_super_bytes(lg, full_clamp(fmt)) > INT32_MAX)
    return MXQ_ERR_SHAPE;
  *g = mxq::GemmArgs{};
  g->a_mant = a_mant;
  g->a_exp = a_exp;
  g->w_mant = w_mant;
  g->w_exp = w_exp;
  g->M = M;
  g->N = N;
  g->a_rb = canon_rb(s);
  g->a_erb = exp_rb(fmt);
  g->a_tile = mxq::a_tile_bytes(lg);
  g->a_tile_sc = mxq::a_tile_scale_bytes(lg);
  g->w_super = mxq::w_super_bytes(lg, full_clamp(fmt));
  g->w_super_sc = mxq::w_super_scale_bytes(lg);
  g->n3 = s.n3;
  g->n4 = s.n4;
  g->n6 = s.n6;
  g->n8 = s.n8;
  g->full = full_clamp(fmt) ? 1 : 0;
  return MXQ_OK;
}

}  // namespace

static mxq_status attn_common(const mxq_fmt *fmt, const uint16_t *q, int64_t B, int64_t Hq,
                              int64_t Hkv, int64_t T, float scale, const uint8_t *k_mant,
                              const uint8_t *k_exp, const uint8_t *v_mant, const uint8_t *v_exp,
                              float *o, float *work, int64_t work_bytes, bool use_static,
                              void *stream);

extern "C" {

int mxq_abi_version(void) { return MXQ_ABI_VERSION; }

const char *mxq_status_str(int status) {
  switch (status) {
    case MXQ_OK: return "ok";
    case MXQ_ERR_NULL: return "null pointer";
    case MXQ_ERR_SHAPE: return "invalid shape or leading dimension";
    case MXQ_ERR_WIDTHS: return "invalid width map (widths must be 3, 4, 6 or 8, non-decreasing)";
    case MXQ_ERR_PERM: return "invalid permutation";
    case MXQ_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case MXQ_ERR_UNSUPPORTED: return "unsupported block size, rounding or clamp mode";
    case MXQ_ERR_DEVICE: return "device launch failure";
    case MXQ_ERR_SCRATCH:
      return "sizes exceed the static scratch of the allocation-free entry point";
    default: return "unknown status";
  }
}

int64_t mxq_act_bytes(const mxq_fmt *fmt, int64_t M) {
  Segs s;
  const mxq_status st = check_fmt(fmt, &s);
  if (st != MXQ_OK) return -(int64_t)st;
  if (M < 0) return -(int64_t)MXQ_ERR_SHAPE;
  return act_bytes(s, M);
}

int64_t mxq_act_exp_bytes(const mxq_fmt *fmt, int64_t M) {
  Segs s;
  const mxq_status st = check_fmt(fmt, &s);
  if (st != MXQ_OK) return -(int64_t)st;
  if (M < 0) return -(int64_t)MXQ_ERR_SHAPE;
  return act_exp_bytes(s, M);
}

int64_t mxq_exp_row_bytes(const mxq_fmt *fmt) {
  Segs s;
  const mxq_status st = check_fmt(fmt, &s);
  return st == MXQ_OK ? exp_rb(fmt) : -(int64_t)st;
}

int64_t mxq_act_packed_bytes(const mxq_fmt *fmt) {
  Segs s;
  const mxq_status st = check_fmt(fmt, &s);
  return st == MXQ_OK ? canon_rb(s) : -(int64_t)st;
}

int64_t mxq_weight_bytes(const mxq_fmt *fmt, int64_t N) {
  Segs s;
  const mxq_status st = check_fmt(fmt, &s);
  if (st != MXQ_OK) return -(int64_t)st;
  if (N < 0) return -(int64_t)MXQ_ERR_SHAPE;
  return w_bytes(fmt, s, N);
}

int64_t mxq_weight_exp_bytes(const mxq_fmt *fmt, int64_t N) {
  Segs s;
  const mxq_status st = check_fmt(fmt, &s);
  if (st != MXQ_OK) return -(int64_t)st;
  if (N < 0) return -(int64_t)MXQ_ERR_SHAPE;
  return w_exp_bytes(s, N);
}

mxq_status mxq_quantize_act(const mxq_fmt *fmt, const uint16_t *a, int64_t M,
                            int64_t lda, uint8_t *a_mant, uint8_t *a_exp,
                            void *stream) {
  return quantize_common(fmt, a, M, lda, a_mant, a_exp, stream, kImage);
}

mxq_status mxq_quantize_rows(const mxq_fmt *fmt, const uint16_t *a, int64_t M, int64_t lda,
                             uint8_t *rows, uint8_t *exps, void *stream) {
  return quantize_common(fmt, a, M, lda, rows, exps, stream, kRows);
}

mxq_status mxq_quantize_act_rmsnorm(const mxq_fmt *fmt, const uint16_t *x, int64_t M,
                                    int64_t ldx, const uint16_t *gain, float eps,
                                    uint8_t *a_mant, uint8_t *a_exp, void *stream) {
  if (M > 0 && !gain) return MXQ_ERR_NULL;
  if (!(eps >= 0.f)) return MXQ_ERR_SHAPE;
  return quantize_common(fmt, x, M, ldx, a_mant, a_exp, stream, kImage, gain, eps);
}

mxq_status mxq_quantize_act_swiglu(const mxq_fmt *fmt, const uint16_t *gate,
                                   const uint16_t *up, int64_t M, int64_t ld,
                                   uint8_t *a_mant, uint8_t *a_exp, void *stream) {
  if (M > 0 && !up) return MXQ_ERR_NULL;
  return quantize_common(fmt, gate, M, ld, a_mant, a_exp, stream, kImage, nullptr, 0.f, up);
}

mxq_status mxq_pack_weights(const mxq_fmt *fmt, const uint16_t *w, int64_t N,
                            int64_t ldw, uint8_t *w_mant, uint8_t *w_exp,
                            void *stream) {
  return quantize_common(fmt, w, N, ldw, w_mant, w_exp, stream, kWeights);
}

mxq_status mxq_gemm(const mxq_fmt *fmt, int64_t M, int64_t N, const uint8_t *a_mant,
                    const uint8_t *a_exp, const uint8_t *w_mant, const uint8_t *w_exp,
                    float *y, int64_t ldy, void *stream) {
  mxq::GemmArgs g;
  mxq_status st = gemm_args(fmt, M, N, a_mant, a_exp, w_mant, w_exp, y, &g);
  if (st != MXQ_OK) return st;
  if (M == 0 || N == 0) return MXQ_OK;
  if (ldy < N) return MXQ_ERR_SHAPE;
  g.y = y;
  g.ldy = ldy;
  hipStream_t s = (hipStream_t)stream;
  return launched(M <= MXQ_DECODE_MAX_M ? mxq::launch_gemm_decode(g, s)
                                        : mxq::launch_gemm_prefill(g, s));
}

mxq_status mxq_gemm_partials(const mxq_fmt *fmt, int64_t M, int64_t N,
                             const uint8_t *a_mant, const uint8_t *a_exp,
                             const uint8_t *w_mant, const uint8_t *w_exp, int32_t *p,
                             void *stream) {
  mxq::GemmArgs g;
  mxq_status st = gemm_args(fmt, M, N, a_mant, a_exp, w_mant, w_exp, p, &g);
  if (st != MXQ_OK) return st;
  if (M == 0 || N == 0) return MXQ_OK;
  g.p = p;
  return launched(mxq::launch_gemm_partials(g, (hipStream_t)stream));
}

static mxq_status unpack_common(const mxq_fmt *fmt, int64_t rows, const uint8_t *mant,
                                const uint8_t *exp, int8_t *q, uint8_t *e, void *stream,
                                bool weights) {
  Segs s;
  mxq_status st = check_fmt(fmt, &s);
  if (st != MXQ_OK) return st;
  if (rows < 0) return MXQ_ERR_SHAPE;
  if (rows == 0) return MXQ_OK;
  if (!mant || !exp || !q || !e) return MXQ_ERR_NULL;
  if (!aligned16(mant) || !aligned16(exp)) return MXQ_ERR_ALIGN;
  mxq::UnpackArgs a{};
  a.mant = mant;
  a.exp = exp;
  a.q = q;
  a.e = e;
  a.rows = rows;
  a.K = fmt->K;
  a.a_rb = canon_rb(s);
  a.a_erb = exp_rb(fmt);
  a.w_super = mxq::w_super_bytes(l_geo(s), full_clamp(fmt));
  a.w_super_sc = mxq::w_super_scale_bytes(l_geo(s));
  a.n3 = s.n3;
  a.n4 = s.n4;
  a.n6 = s.n6;
  a.n8 = s.n8;
  a.full = full_clamp(fmt) ? 1 : 0;
  return launched(mxq::launch_unpack(a, weights, (hipStream_t)stream));
}

mxq_status mxq_unpack_act(const mxq_fmt *fmt, int64_t rows, const uint8_t *a_mant,
                          const uint8_t *a_exp, int8_t *q, uint8_t *e, void *stream) {
  return unpack_common(fmt, rows, a_mant, a_exp, q, e, stream, false);
}

mxq_status mxq_unpack_weights(const mxq_fmt *fmt, int64_t N, const uint8_t *w_mant,
                              const uint8_t *w_exp, int8_t *q, uint8_t *e, void *stream) {
  return unpack_common(fmt, N, w_mant, w_exp, q, e, stream, true);
}

mxq_status mxq_calib_colsq(const uint16_t *x, int64_t rows, int64_t ldx, int64_t K, double *s,
                           int accumulate, void *stream) {
  if (!x || !s) return MXQ_ERR_NULL;
  if (rows < 0 || K <= 0 || ldx < K) return MXQ_ERR_SHAPE;
  return launched(mxq::launch_calib_colsq(x, rows, ldx, K, s, accumulate != 0,
                                          (hipStream_t)stream));
}

mxq_status mxq_calib_colsq_samples(const uint16_t *x, int64_t n_samples, int64_t rows,
                                   int64_t ldx, int64_t sample_stride, int64_t K, double *work,
                                   double *s, int accumulate, void *stream) {
  if (!x || !s || !work) return MXQ_ERR_NULL;
  if (n_samples < 1 || n_samples > 65535 || rows < 0 || K <= 0 || ldx < K ||
      (n_samples > 1 && sample_stride < rows * ldx))
    return MXQ_ERR_SHAPE;
  return launched(mxq::launch_calib_colsq_samples(x, n_samples, rows, ldx, sample_stride, K,
                                                  work, s, accumulate != 0, (hipStream_t)stream));
}

mxq_status mxq_calib_ratio(int32_t n, const int64_t *d_in, const double *s_layer, double B,
                           double *R) {
  if (!d_in || !s_layer || !R) return MXQ_ERR_NULL;
  if (n < 1) return MXQ_ERR_SHAPE;
  double total = 0.0, den = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    if (d_in[i] < 32 || d_in[i] % 32) return MXQ_ERR_SHAPE;
    total += (double)d_in[i];
    den += 2.0 * s_layer[i] * (double)(d_in[i] - 32);
  }
  if (!(den != 0.0)) return MXQ_ERR_SHAPE;   // every layer insensitive (or only 8-bit)
  *R = ((B - 4.0) * total - 4.0 * 32.0 * (double)n) / den;
  return MXQ_OK;
}

mxq_status mxq_calib_counts(int64_t d_in, double R, double s_layer, int32_t n8_blocks,
                            int32_t *n4, int32_t *n6, int32_t *n8) {
  if (!n4 || !n6 || !n8) return MXQ_ERR_NULL;
  if (d_in < 32 || d_in % 32 || n8_blocks < 0) return MXQ_ERR_SHAPE;
  const int64_t nb = d_in / 32;
  const int64_t e = n8_blocks < nb ? n8_blocks : nb;
  const double cols = floor(R * s_layer * (double)(d_in - 32));
  int64_t six = 0;
  if (cols > 0) six = cols >= (double)(nb * 32) ? nb : (int64_t)cols / 32;
  if (six > nb - e) six = nb - e;
  *n8 = (int32_t)e;
  *n6 = (int32_t)six;
  *n4 = (int32_t)(nb - e - six);
  return MXQ_OK;
}

mxq_status mxq_calib_perm(const double *s, int64_t K, int32_t n6_blocks, int32_t n8_blocks,
                          int32_t *perm, void *stream) {
  if (!s || !perm) return MXQ_ERR_NULL;
  if (K <= 0 || K % 32 || K > INT32_MAX || n6_blocks < 0 || n8_blocks < 0 ||
      (int64_t)n6_blocks + n8_blocks > K / 32)
    return MXQ_ERR_SHAPE;
  return launched(mxq::launch_calib_perm(s, K, n6_blocks, n8_blocks, perm, (hipStream_t)stream));
}

int64_t mxq_peak_sink_words(void) { return mxq::peak_sink_words(); }

mxq_status mxq_peak_stream_read(const void *buf, int64_t bytes, uint32_t *sink, void *stream) {
  if (!buf || !sink) return MXQ_ERR_NULL;
  if (bytes <= 0 || bytes % 16) return MXQ_ERR_SHAPE;
  return launched(mxq::launch_peak_stream(buf, bytes, sink, (hipStream_t)stream));
}

mxq_status mxq_peak_mfma(int kind, int64_t iters, float *sink, int64_t *ops, void *stream) {
  if (!sink || !ops) return MXQ_ERR_NULL;
  if (kind < 0 || kind > 2 || iters < 1) return MXQ_ERR_SHAPE;
  *ops = mxq::peak_mfma_ops(kind, iters);
  return launched(mxq::launch_peak_mfma(kind, iters, sink, (hipStream_t)stream));
}

// Decode attention over the MXINT KV cache (MXSens Appendix A.2).
static mxq_status attn_shape(const mxq_fmt *fmt, int64_t B, int64_t Hq, int64_t Hkv, int64_t T,
                             Segs *sg) {
  const mxq_status st = check_fmt(fmt, sg);
  if (st != MXQ_OK) return st;
  if (fmt->K != 128) return MXQ_ERR_SHAPE;
  if (fmt->perm) return MXQ_ERR_UNSUPPORTED;
  if (B < 0 || Hkv < 1 || Hq < Hkv || Hq % Hkv || Hq / Hkv > 16 || T < 1) return MXQ_ERR_SHAPE;
  if (B > 65535 || Hkv > 65535 || Hq > INT32_MAX || T > (int64_t)1 << 40) return MXQ_ERR_SHAPE;
  return MXQ_OK;
}

int64_t mxq_attn_work_bytes(const mxq_fmt *fmt, int64_t B, int64_t Hq, int64_t Hkv, int64_t T) {
  Segs sg;
  const mxq_status st = attn_shape(fmt, B, Hq, Hkv, T, &sg);
  if (st != MXQ_OK) return -(int64_t)st;
  if (B == 0) return 0;
  const int64_t tps = mxq::attn_tokens_per_split(B, Hkv, T);
  return B * Hq * ((T + tps - 1) / tps) * 130 * (int64_t)sizeof(float);
}

mxq_status mxq_attn_decode(const mxq_fmt *fmt, const uint16_t *q, int64_t B, int64_t Hq,
                           int64_t Hkv, int64_t T, float scale, const uint8_t *k_mant,
                           const uint8_t *k_exp, const uint8_t *v_mant, const uint8_t *v_exp,
                           float *o, float *work, int64_t work_bytes, void *stream) {
  return attn_common(fmt, q, B, Hq, Hkv, T, scale, k_mant, k_exp, v_mant, v_exp, o, work,
                     work_bytes, false, stream);
}

mxq_status mxq_attn_decode_static(const mxq_fmt *fmt, const uint16_t *q, int64_t B, int64_t Hq,
                                  int64_t Hkv, int64_t T, float scale, const uint8_t *k_mant,
                                  const uint8_t *k_exp, const uint8_t *v_mant,
                                  const uint8_t *v_exp, float *o, void *stream) {
  return attn_common(fmt, q, B, Hq, Hkv, T, scale, k_mant, k_exp, v_mant, v_exp, o, nullptr,
                     0, true, stream);
}

}  // extern "C"

static mxq_status attn_common(const mxq_fmt *fmt, const uint16_t *q, int64_t B, int64_t Hq,
                              int64_t Hkv, int64_t T, float scale, const uint8_t *k_mant,
                              const uint8_t *k_exp, const uint8_t *v_mant, const uint8_t *v_exp,
                              float *o, float *work, int64_t work_bytes, bool use_static,
                              void *stream) {
  Segs sg;
  const mxq_status st = attn_shape(fmt, B, Hq, Hkv, T, &sg);
  if (st != MXQ_OK) return st;
  if (!(scale == scale) || scale == INFINITY || scale == -INFINITY) return MXQ_ERR_SHAPE;
  if (B == 0) return MXQ_OK;
  if (!q || !k_mant || !k_exp || !v_mant || !v_exp || !o || (!use_static && !work))
    return MXQ_ERR_NULL;
  if (!aligned16(k_mant) || !aligned16(k_exp) || !aligned16(v_mant) || !aligned16(v_exp) ||
      (!use_static && !aligned16(work)) || !aligned16(q) || ((uintptr_t)o & 3u))
    return MXQ_ERR_ALIGN;
  const int64_t tps = mxq::attn_tokens_per_split(B, Hkv, T);
  const int64_t splits = (T + tps - 1) / tps;
  const int64_t need = B * Hq * splits * 130 * (int64_t)sizeof(float);
  if (splits > mxq::kAttnMaxSplits) return MXQ_ERR_SHAPE;
  if (use_static) {
    if (need > mxq::kAttnStaticWorkBytes) return MXQ_ERR_SCRATCH;
    if (mxq::attn_static_scratch(&work) != hipSuccess) return MXQ_ERR_DEVICE;
  } else if (work_bytes < need) {
    return MXQ_ERR_SHAPE;
  }
  mxq::AttnArgs a{};
  a.q = q;
  a.k_mant = k_mant;
  a.k_exp = k_exp;
  a.v_mant = v_mant;
  a.v_exp = v_exp;
  a.o = o;
  a.work = work;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.T = T;
  a.G = (int)(Hq / Hkv);
  a.scale = scale;
  a.exp_bytes = exp_rb(fmt);
  a.tokens_per_split = tps;
  a.splits = (int)splits;
  a.n3 = sg.n3;
  a.n4 = sg.n4;
  a.n6 = sg.n6;
  a.n8 = sg.n8;
  return launched(mxq::launch_attn_decode(a, (hipStream_t)stream));
}
