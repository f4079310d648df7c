// quantize.hip -- offline MXINT quantize + pack of bf16 weight rows.
//
// MXSens (arXiv 2607.17733) Section 2 and Section 4.1: every 32-element
// block of the permuted weight row (one output column) gets one shared
// exponent and one mantissa width, the same quantizer as the activations.
//
// Work decomposition: a thread owns 8 consecutive elements of a block (a
// "quarter"), so the 4 threads of a block are adjacent lanes; the block
// maximum is a 2-step xor-shuffle reduction of integer |bf16| bit patterns.
// A workgroup owns one row (K >= 2048) or several whole rows (short K).
// With a column permutation the workgroup first stages its source rows in
// LDS with 16-byte coalesced loads and gathers from LDS.
//
// Output: the weight layout of both GEMMs (LGeo in mxq_device.h), one copy
// at the MXINT size: the folded FP6 codes of 3- and 4-bit blocks, the two
// digit planes of 6-bit blocks, the mantissa bytes of 8-bit blocks, and the
// scale words (each block's exponent E).  The four quarters of a block
// assemble its FP6 operand words by xor-shuffles before folding them.  The
// padding of the segments (up to whole steps) and of the columns (up to
// whole 128-column super-slabs) is written as zeros.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

constexpr int kThreads = 256;

// OR of the words of the 4 quarters of a block (adjacent lanes).
__device__ inline void or4(uint32_t *d, int n) {
  for (int k = 0; k < n; ++k) {
    d[k] |= __shfl_xor(d[k], 1);
    d[k] |= __shfl_xor(d[k], 2);
  }
}

// The six operand words of 8 six-bit codes at elements 8kg..8kg+7 (the
// other quarters' bits zero): the 48 bits start at bit 48 kg.
__device__ inline void quarter_words(const uint32_t *c, int kg, uint32_t *d) {
  uint64_t v = 0;
#pragma unroll
  for (int u = 0; u < 8; ++u) v |= (uint64_t)(c[u] & 63u) << (6 * u);
  v <<= 16 * (kg & 1);
  const int w0 = (kg >> 1) * 3 + (kg & 1);
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
#pragma unroll
  for (int j = 0; j < 6; ++j) d[j] = (j == w0 ? lo : 0u) | (j == w0 + 1 ? hi : 0u);
}

__global__ __launch_bounds__(kThreads) void quantize_kernel(QuantArgs q) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int t = threadIdx.x;
  const int64_t K = q.K;
  const LGeo lg(q.n3, q.n4, q.n6, q.n8);
  const bool full = q.full_clamp != 0;
  int npb = 0;                               // padded blocks of a column
  for (int s = 0; s < kSegs; ++s) npb += lg.S[s] * (s < 2 ? 4 : 2);
  const int G = 4 * npb;                     // quarters per column
  const int R = q.rows_per_wg;
  const int64_t row0 = (int64_t)blockIdx.x * R;
  uint16_t *srow = (uint16_t *)smem;         // [R][K] staged source rows

  if (q.stage) {
    const int64_t total = (int64_t)R * K;
    if (q.vec16) {
      for (int64_t v = t; v < total / 8; v += kThreads) {
        const int lr = (int)(v * 8 / K);
        const int64_t col = v * 8 - (int64_t)lr * K;
        const int64_t row = row0 + lr;
        uint4 d = make_uint4(0, 0, 0, 0);
        if (row < q.src_rows) d = *(const uint4 *)(q.src + row * q.ld + col);
        *(uint4 *)(srow + (int64_t)lr * K + col) = d;
      }
    } else {
      for (int64_t v = t; v < total; v += kThreads) {
        const int lr = (int)(v / K);
        const int64_t col = v - (int64_t)lr * K;
        const int64_t row = row0 + lr;
        srow[v] = row < q.src_rows ? q.src[row * q.ld + col] : (uint16_t)0;
      }
    }
    __syncthreads();
  }

  for (int64_t f = t; f < (int64_t)R * G; f += kThreads) {
    const int lr = (int)(f / G);
    const int gq = (int)(f - (int64_t)lr * G);
    const int64_t row = row0 + lr;           // the weight column
    // the last workgroup's rows may pass the padded column count (a block's
    // four quarters skip together, so the shuffles stay within live lanes)
    if (row >= q.out_rows) continue;
    const int pb = gq >> 2, kg = gq & 3;
    // segment, step, position within the step, and the width-map block
    int s = 0, rem = pb;
    while (s < kSegs - 1 && rem >= lg.S[s] * (s < 2 ? 4 : 2)) {
      rem -= lg.S[s] * (s < 2 ? 4 : 2);
      ++s;
    }
    const int per = s < 2 ? 4 : 2;
    const int st = lg.st0[s] + rem / per, pos = rem % per;
    const bool real = rem < lg.nb[s];
    const int b = lg.b0[s] + rem;
    const int m = s == 0 ? 3 : s == 1 ? 4 : s == 2 ? 6 : 8;
    const bool live = real && row < q.src_rows;

    uint32_t bits[8];
    const int64_t p0 = (int64_t)b * kBlock + 8 * kg;
    if (!live) {
#pragma unroll
      for (int u = 0; u < 8; ++u) bits[u] = 0;
    } else if (q.perm) {
      const int4 pa = *(const int4 *)(q.perm + p0);
      const int4 pc = *(const int4 *)(q.perm + p0 + 4);
      const int src[8] = {pa.x, pa.y, pa.z, pa.w, pc.x, pc.y, pc.z, pc.w};
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bool ok = src[u] >= 0 && (int64_t)src[u] < K;
        uint32_t v = 0;
        if (ok) v = q.stage ? srow[(int64_t)lr * K + src[u]] : q.src[row * q.ld + src[u]];
        bits[u] = v;
      }
    } else if (q.vec16) {
      const uint4 d = *(const uint4 *)(q.src + row * q.ld + p0);
      const uint32_t w[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        bits[2 * u] = w[u] & 0xFFFFu;
        bits[2 * u + 1] = w[u] >> 16;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 8; ++u) bits[u] = q.src[row * q.ld + p0 + u];
    }

    uint32_t amax = 0;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t mag = bits[u] & 0x7FFFu;
      amax = mag > amax ? mag : amax;
    }
    uint32_t o = __shfl_xor(amax, 1);
    amax = o > amax ? o : amax;
    o = __shfl_xor(amax, 2);
    amax = o > amax ? o : amax;
    const int E = live ? block_exponent(amax) : 0;
    int qv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) qv[u] = live ? quant_elem(bits[u], E, m, q.ties_away, q.full_clamp) : 0;

    // where the block goes
    const int64_t col = row;
    const int n = (int)((col % kWCols) >> 4), c = (int)(col & 15);
    uint8_t *chunk = q.mant + (col / kWCols) * w_super_bytes(lg, full) + w_step_off(lg, st, full) +
                     (int64_t)n * w_chunk_bytes(s, full);
    uint8_t *scl = q.exp + (col / kWCols) * w_super_scale_bytes(lg) +
                   (int64_t)lg.group_of(st) * 2048 + 8 * lg.byte_of(st) + n;

    if (s <= 1) {
      uint32_t codes[8], d[6], x[4];
#pragma unroll
      for (int u = 0; u < 8; ++u) codes[u] = w_code34(qv[u]);
      quarter_words(codes, kg, d);
      or4(d, 6);
      const int l = 16 * pos + c;
      if (s == 0 && !full) {
        fold3(d, x);
        if (kg < 2) *(uint32_t *)(chunk + 8 * l + 4 * kg) = x[kg];
        else if (kg == 2) *(uint32_t *)(chunk + 512 + 4 * l) = x[2];
      } else if (s == 1 && full) {
        *(uint32_t *)(chunk + 16 * l + 4 * kg) = d[kg];
        if (kg < 2) *(uint32_t *)(chunk + 1024 + 8 * l + 4 * kg) = d[4 + kg];
      } else {
        fold4(d, x);
        *(uint32_t *)(chunk + 16 * l + 4 * kg) = x[kg];
      }
      if (kg == 0) scl[32 * l] = (uint8_t)E;
    } else if (s == 2) {
      uint32_t ch[8], cl[8], dh[6], dl[6], x[4];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        w_code6(qv[u], ch[u], cl[u]);
        if (!full) ch[u] &= 31u;             // the high plane keeps no sign
      }
      quarter_words(cl, kg, dl);
      quarter_words(ch, kg, dh);
      or4(dl, 6);
      or4(dh, 6);
      const int jc = 16 * pos + c;
      fold4(dl, x);
      *(uint32_t *)(chunk + 16 * jc + 4 * kg) = x[kg];
      if (full) {
        fold4(dh, x);
        *(uint32_t *)(chunk + 512 + 16 * jc + 4 * kg) = x[kg];
      } else {
        fold2(dh, x);
        if (kg < 2) *(uint32_t *)(chunk + 512 + 8 * jc + 4 * kg) = x[kg];
      }
      if (kg == 0) {
        scl[32 * (16 * (2 * pos) + c)] = (uint8_t)E;
        scl[32 * (16 * (2 * pos + 1) + c)] = (uint8_t)E;
      }
    } else {
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        w0 |= w_code8(qv[u], full) << (8 * u);
        w1 |= w_code8(qv[4 + u], full) << (8 * u);
      }
      const int jc = 16 * pos + c;
      *(uint2 *)(chunk + 32 * jc + 8 * kg) = make_uint2(w0, w1);
      if (kg == 0) {
        scl[32 * (16 * (2 * pos) + c)] = (uint8_t)E;
        scl[32 * (16 * (2 * pos + 1) + c)] = (uint8_t)E;
      }
    }
    // the unused scale bytes of a segment's short last group
    if (kg == 0 && rem == 0) {
      const int S = lg.S[s];
      for (int k = S; k < (S + kGroupSteps - 1) / kGroupSteps * kGroupSteps; ++k) {
        uint8_t *z = q.exp + (col / kWCols) * w_super_scale_bytes(lg) +
                     (int64_t)(lg.G0[s] + k / kGroupSteps) * 2048 + 8 * (k % kGroupSteps) + n;
        for (int gg = 0; gg < 4; ++gg) z[32 * (16 * gg + c)] = 0;
      }
    }
  }
}

}  // namespace

hipError_t launch_quantize(const QuantArgs &args, bool weights, hipStream_t stream) {
  if (!weights) return hipErrorInvalidValue;     // activations: launch_quantize_act
  const LGeo lg(args.n3, args.n4, args.n6, args.n8);
  int npb = 0;
  for (int s = 0; s < kSegs; ++s) npb += lg.S[s] * (s < 2 ? 4 : 2);
  const int G = 4 * npb;
  QuantArgs a = args;
  a.rows_per_wg = G >= kThreads ? 1 : kThreads / G;
  const int64_t grid = (a.out_rows + a.rows_per_wg - 1) / a.rows_per_wg;
  if (grid <= 0) return hipSuccess;
  // stage the source rows in LDS for the permutation gather when they fit;
  // longer rows gather straight from global memory
  a.stage = (a.perm && (int64_t)a.rows_per_wg * a.K * 2 <= kMaxLds) ? 1 : 0;
  const int64_t lds = a.stage ? (int64_t)a.rows_per_wg * a.K * 2 : 0;
  if (lds > kMaxLds) return hipErrorInvalidValue;
  (void)hipFuncSetAttribute((const void *)quantize_kernel,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  hipLaunchKernelGGL(quantize_kernel, dim3((unsigned)grid), dim3(kThreads), (size_t)lds, stream,
                     a);
  return hipGetLastError();
}

}  // namespace mxq
