// decode.hip -- MXINT GEMM for decode shapes (M <= 16), streaming the
// packed weights at HBM rate.
//
// Y[i][j] = sum_b 2^(sa[i][b] + sw[j][b]) * sum_t qa qw  (MXSens, arXiv
// 2607.17733, Section 2: integer block products with power-of-two block
// scales; Section 6: the memory cost is the packed weights).
//
// The weights stay packed in HBM (4m bits per element, stream layout in
// mxq_device.h) and become FP8 e4m3 digits in registers: a nibble is looked
// up in a 16-entry byte table with three V_PERM_B32.  With the block's E as
// the E8M0 scale the digits must sum to q * 2^-(m-2): a 4-bit mantissa q
// becomes e4m3(q/4), a 6-bit q = 16h + l the digits e4m3(h) and
// e4m3(l/16), an 8-bit q = 16h + l the digits e4m3(h/4) and e4m3(l/64).
// The activations arrive as ready FP6/FP8 digits (decode image).
// V_MFMA_SCALE_F32_16X16X128_F8F6F4 multiplies 16 rows by
// 16 columns over four K-blocks and applies every block's E8M0 scale in
// hardware, so no per-block rescale runs on the VALU.  Digit products are
// exact; a 6/8-bit block pair takes two instructions (the second with the
// weight digits' halves swapped: h*h + l*l, then h*l + l*h).
//
// Work decomposition: one workgroup per 16-column slab, four waves taking
// every fourth step of each width segment, four steps per iteration with
// all loads issued first; the waves' fp32 accumulators meet in LDS in a
// fixed order.  Activation loads of rows >= M are predicated off.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef unsigned u2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kUnroll = 4;

// FP8 e4m3 code of num / den (den a power of two; the value must be exact).
constexpr uint32_t e4m3_exact(int num, int den) {
  if (num == 0) return 0;
  const uint32_t sign = num < 0 ? 0x80u : 0u;
  int a = num < 0 ? -num : num;
  int e = 0;                               // a / den = (a / 2^p) * 2^(p - log2 den)
  while ((a >> e) > 1) ++e;                // a in [2^e, 2^(e+1))
  int lg = 0;
  while ((1 << lg) < den) ++lg;
  const int ue = e - lg;                   // unbiased exponent of the value
  const uint32_t mant = (uint32_t)(((a << 3) >> e) & 7);
  return sign | ((uint32_t)(ue + 7) << 3) | mant;
}

// 16-entry byte table (entry n = f(n)) as four dwords
template <int KIND>
constexpr uint32_t table_dword(int d) {
  uint32_t v = 0;
  for (int k = 0; k < 4; ++k) {
    const int n = 4 * d + k;
    const int sn = n < 8 ? n : n - 16;     // two's-complement nibble
    uint32_t c = 0;
    if (KIND == 0) c = e4m3_exact(sn, 4);        // 4-bit q -> q/4; 8-bit high h -> h/4
    if (KIND == 1) c = e4m3_exact(n, 16);        // 6-bit low digit l -> l/16
    if (KIND == 2) c = e4m3_exact(n, 64);        // 8-bit low digit l -> l/64
    v |= c << (8 * k);
  }
  return v;
}

// 2-bit signed high digit h of a 6-bit mantissa -> e4m3(h): h = 0, 1, -2, -1
constexpr uint32_t kTop6 = e4m3_exact(0, 1) | (e4m3_exact(1, 1) << 8) |
                           (e4m3_exact(-2, 1) << 16) | (e4m3_exact(-1, 1) << 24);

// Byte-wise lookup: byte k of s holds an index in its low nibble.
template <int KIND>
__device__ inline uint32_t lut16(uint32_t s) {
  const uint32_t s7 = s & 0x07070707u;
  const uint32_t lo = __builtin_amdgcn_perm(table_dword<KIND>(1), table_dword<KIND>(0), s7);
  const uint32_t hi = __builtin_amdgcn_perm(table_dword<KIND>(3), table_dword<KIND>(2), s7);
  const uint32_t sel = ((s >> 1) & 0x04040404u) | 0x03020100u;
  return __builtin_amdgcn_perm(hi, lo, sel);
}

struct Step4 {
  u4 w;
  u4 a0;
  u2 a1;
  uint32_t ws, as;
};
struct Step68 {
  u4 w;            // 8-bit: 16 bytes; 6-bit: nibbles in .x/.y, top-bit dword in .z
  u4 a0, a1;
  uint32_t ws, as;
};

__device__ inline v4f mfma(const v8i &a, const v8i &b, v4f acc, int fa, uint32_t as,
                           uint32_t ws) {
  if (fa == 3)
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, acc, 3, 0, 0, (int)as, 0,
                                                            (int)ws);
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, acc, 0, 0, 0, (int)as, 0,
                                                          (int)ws);
}

__global__ __launch_bounds__(kThreads) void gemm_decode_kernel(GemmArgs g) {
  __shared__ v4f red[kWaves][64];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int line = lane & 15;
  const DGeo d(g.n4, g.n6, g.n8);
  const int64_t slab = blockIdx.x;
  const uint8_t *wslab = g.w_mant + slab * wd_slab_bytes(d);
  const uint8_t *aimg = g.a_mant + g.a_op;
  const bool arow = line < g.M;
  v4f acc = {0.f, 0.f, 0.f, 0.f};

  // 4-bit steps: A e3m2 (format 3) x W e4m3 (format 0), one instruction
  for (int s0 = wave; s0 < d.S4; s0 += kWaves * kUnroll) {
    Step4 st[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const int s = s0 + kWaves * k;
      st[k].w = u4{0u, 0u, 0u, 0u};
      st[k].a0 = u4{0u, 0u, 0u, 0u};
      st[k].a1 = u2{0u, 0u};
      st[k].ws = st[k].as = 0;
      if (s < d.S4) {
        const uint8_t *wc = wslab + wd_step_off(d, s);
        st[k].w = *(const u4 *)(wc + 16 * lane);
        st[k].ws = wc[1024 + lane];
        if (arow) {
          const uint8_t *ac = aimg + ad_step_off(d, s);
          st[k].a0 = *(const u4 *)(ac + 16 * lane);
          st[k].a1 = *(const u2 *)(ac + 1024 + 8 * lane);
          st[k].as = ac[1536 + lane];
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      v8i b;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        b[2 * i] = (int)lut16<0>(st[k].w[i]);
        b[2 * i + 1] = (int)lut16<0>(st[k].w[i] >> 4);
      }
      const v8i a = {(int)st[k].a0[0], (int)st[k].a0[1], (int)st[k].a0[2], (int)st[k].a0[3],
                     (int)st[k].a1[0], (int)st[k].a1[1], 0, 0};
      acc = mfma(a, b, acc, 3, st[k].as, st[k].ws);
    }
  }

  // 6-bit and 8-bit steps: FP8 digits on both sides, two instructions
#pragma unroll
  for (int seg = 1; seg <= 2; ++seg) {
    const int sb = seg == 1 ? d.S4 : d.S4 + d.S6;
    const int se = seg == 1 ? d.S4 + d.S6 : d.nsteps;
    const int lb = wd_lane_bytes(seg);
    for (int s0 = sb + wave; s0 < se; s0 += kWaves * kUnroll) {
      Step68 st[kUnroll];
#pragma unroll
      for (int k = 0; k < kUnroll; ++k) {
        const int s = s0 + kWaves * k;
        st[k].w = u4{0u, 0u, 0u, 0u};
        st[k].a0 = st[k].a1 = u4{0u, 0u, 0u, 0u};
        st[k].ws = st[k].as = 0;
        if (s < se) {
          const uint8_t *wc = wslab + wd_step_off(d, s);
          if (seg == 1) {
            const u2 nb = *(const u2 *)(wc + 8 * lane);
            st[k].w = u4{nb[0], nb[1], *(const uint32_t *)(wc + 512 + 4 * lane), 0u};
          } else {
            st[k].w = *(const u4 *)(wc + 16 * lane);
          }
          st[k].ws = wc[64 * lb + lane];
          if (arow) {
            const uint8_t *ac = aimg + ad_step_off(d, s);
            st[k].a0 = *(const u4 *)(ac + 32 * lane);
            st[k].a1 = *(const u4 *)(ac + 32 * lane + 16);
            st[k].as = ac[2048 + lane];
          }
        }
      }
#pragma unroll
      for (int k = 0; k < kUnroll; ++k) {
        uint32_t hd[4], ld[4];
        if (seg == 1) {
          // low digits from the nibbles, high digits from the 2-bit plane
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            ld[2 * i] = lut16<1>(st[k].w[i]);
            ld[2 * i + 1] = lut16<1>(st[k].w[i] >> 4);
          }
#pragma unroll
          for (int q = 0; q < 4; ++q)
            hd[q] = __builtin_amdgcn_perm(0u, kTop6, (st[k].w[2] >> (2 * q)) & 0x03030303u);
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            ld[i] = lut16<2>(st[k].w[i]);
            hd[i] = lut16<0>(st[k].w[i] >> 4);
          }
        }
        const v8i a = {(int)st[k].a0[0], (int)st[k].a0[1], (int)st[k].a0[2], (int)st[k].a0[3],
                       (int)st[k].a1[0], (int)st[k].a1[1], (int)st[k].a1[2], (int)st[k].a1[3]};
        const v8i bhl = {(int)hd[0], (int)hd[1], (int)hd[2], (int)hd[3],
                         (int)ld[0], (int)ld[1], (int)ld[2], (int)ld[3]};
        const v8i blh = {(int)ld[0], (int)ld[1], (int)ld[2], (int)ld[3],
                         (int)hd[0], (int)hd[1], (int)hd[2], (int)hd[3]};
        acc = mfma(a, bhl, acc, 0, st[k].as, st[k].ws);
        acc = mfma(a, blh, acc, 0, st[k].as, st[k].ws);
      }
    }
  }

  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    v4f y = red[0][lane];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) y += red[w][lane];
    const int64_t col = slab * 16 + line;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * (lane >> 4) + i;
      if (row < g.M && col < g.N) g.y[row * g.ldy + col] = y[i];
    }
  }
}

}  // namespace

hipError_t launch_gemm_decode(const GemmArgs &a, hipStream_t stream) {
  dim3 grid((unsigned)(a.npad / 16));
  hipLaunchKernelGGL(gemm_decode_kernel, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
