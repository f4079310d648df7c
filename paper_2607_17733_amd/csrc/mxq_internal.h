// mxq_internal.h -- argument blocks and launchers shared between the host
// API (api.cpp) and the kernel translation units.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mxq.h"

namespace mxq {

struct QuantArgs {
  const uint16_t *src;     // bf16 rows [src_rows][ld]
  int64_t ld;
  int64_t src_rows;        // rows with data (M, or N for weights)
  int64_t out_rows;        // rows written (activations: M, or M rounded up to
                           // 16 for the operand image; weights: N rounded up
                           // to 128)
  int64_t K;
  const int32_t *perm;     // device, K entries, or nullptr
  int n4, n6, n8;
  int n3;                  // the first n3 of the n4 blocks are 3-bit
  int ties_away, full_clamp;
  uint8_t *mant;           // canonical packed rows (activations), weight data
  uint8_t *exp;            // exponent rows (activations), weight scale words
  int64_t out_rb;          // packed row stride (activations)
  int64_t out_erb;         // exponent row stride
  int64_t canon_rb;        // packed section bytes per row
  int64_t canon_erb;       // exponent bytes per row
  int64_t row_used;        // unpadded packed bytes per row
  // activations: which outputs to write
  int write_rows, write_image;
  uint8_t *img;            // operand image (16-row tiles)
  uint8_t *img_exp;        // its scale words
  int64_t a_tile, a_tile_sc;  // bytes per 16-row tile of each
  int stage;               // weights: stage source rows in LDS before the gather
  int vec16;               // 16-byte source loads are aligned
  int rows_per_wg;         // filled by the launcher
  int lg_rows;             // activations: log2 of the rows per group
  int perm_table;          // activations: gather through the LDS offset table
  // activations: RMS-normalise each row before quantizing (y = g * x / rms)
  int rmsnorm;
  const uint16_t *gain;    // bf16 [K]
  float eps;
  // activations: the rows are SiLU(src) * src2 (gate and up, same layout)
  int swiglu;
  const uint16_t *src2;
};

struct GemmArgs {
  const uint8_t *a_mant;   // operand image (gemm) or packed rows (partials)
  const uint8_t *a_exp;    // its scale words (gemm) or exponent rows (partials)
  const uint8_t *w_mant;   // weight data
  const uint8_t *w_exp;    // weight scale words
  float *y;                // [M][ldy] (gemm)
  int32_t *p;              // [M][N][nb] (partials)
  int64_t M, N, ldy;
  int64_t a_rb, a_erb;     // packed activation row / exponent row strides (partials)
  int64_t a_tile, a_tile_sc;      // operand image bytes per 16-row tile
  int64_t w_super, w_super_sc;    // weight bytes per 128-column super-slab
  int n3, n4, n6, n8;
  int full;                // full clamp: the weights' full-range encodings
};

struct UnpackArgs {
  const uint8_t *mant;
  const uint8_t *exp;
  int8_t *q;               // [rows][K]
  uint8_t *e;              // [rows][nb]
  int64_t rows, K;
  int64_t a_rb, a_erb;     // activation layout
  int64_t w_super, w_super_sc;  // weight layout
  int n3, n4, n6, n8;
  int full;
};

constexpr int64_t kMaxLds = 160 * 1024;   // LDS per workgroup on gfx950

hipError_t launch_quantize(const QuantArgs &args, bool weights, hipStream_t s);
hipError_t launch_quantize_act(const QuantArgs &args, hipStream_t s);
int quantize_act_padded_blocks(int n3, int n4, int n6, int n8);
int quantize_act_rows(int64_t K, int padded_blocks, bool perm, bool rmsnorm = false);
int64_t quantize_act_lds(int64_t K, int padded_blocks, bool perm, bool rmsnorm = false);
// Compute units of the current device (256 if the query fails).
int device_cu_count();
hipError_t launch_gemm_prefill(const GemmArgs &args, hipStream_t s);
hipError_t launch_gemm_partials(const GemmArgs &args, hipStream_t s);
hipError_t launch_gemm_decode(const GemmArgs &args, hipStream_t s);
hipError_t launch_unpack(const UnpackArgs &args, bool weights, hipStream_t s);

// Calibration (calib.hip).
hipError_t launch_calib_colsq(const uint16_t *x, int64_t rows, int64_t ld, int64_t K, double *s,
                              bool accumulate, hipStream_t s_);
hipError_t launch_calib_colsq_samples(const uint16_t *x, int64_t n, int64_t rows, int64_t ld,
                                      int64_t sample_stride, int64_t K, double *part, double *s,
                                      bool accumulate, hipStream_t stream);
hipError_t launch_calib_perm(const double *s, int64_t K, int64_t n6, int64_t n8, int32_t *perm,
                             hipStream_t stream);

// Achievable-peak microbenchmarks (peaks.hip).
int64_t peak_sink_words();
int64_t peak_mfma_ops(int kind, int64_t iters);
hipError_t launch_peak_stream(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t s);
hipError_t launch_peak_mfma(int kind, int64_t iters, float *sink, hipStream_t s);

// Decode attention over an MXINT KV cache (attn.hip).
struct AttnArgs {
  const uint16_t *q;       // bf16 [B][Hq][128]
  const uint8_t *k_mant, *k_exp, *v_mant, *v_exp;
  float *o;                // [B][Hq][128]
  float *work;             // [B][Hkv][splits][G][130]
  int64_t B, Hq, Hkv, T;
  int G;
  float scale;
  int64_t exp_bytes;       // exponent row stride
  int64_t tokens_per_split;
  int splits;
  int n3, n4, n6, n8;
};

constexpr int kAttnMaxSplits = 512;    // attn_tokens_per_split never asks for more
// Static per-device scratch of mxq_attn_decode_static (include/mxq.h).
constexpr int64_t kAttnStaticWorkBytes = MXQ_ATTN_STATIC_WORK_BYTES;
// The device address of this device's static scratch (looked up once per
// device, with that device current).
hipError_t attn_static_scratch(float **ptr);
int64_t attn_tokens_per_split(int64_t B, int64_t Hkv, int64_t T);
hipError_t launch_attn_decode(const AttnArgs &args, hipStream_t s);

}  // namespace mxq
