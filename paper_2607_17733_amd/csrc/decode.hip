// decode.hip -- MXINT GEMM for decode shapes (M <= 16), streaming the
// packed weights at HBM rate.
//
// Y[i][j] = sum_b 2^(sa[i][b] + sw[j][b]) * sum_t qa qw  (MXSens, arXiv
// 2607.17733, Section 2: integer block products with power-of-two block
// scales; Section 6: the memory cost is the packed weights).
//
// The weights stay packed in HBM (4m bits per element, stream layout in
// mxq_device.h) and become FP8 e4m3 digits in registers.  With the block's
// E as the E8M0 scale the digits must sum to q * 2^-(m-2): a 4-bit q becomes
// e4m3(q/4); a 6-bit q two digits summing to q/16; an 8-bit q = 16h + l the
// digits e4m3(h/4) and e4m3(l/64).  Sign-magnitude codes (symmetric clamp)
// take one V_PERM_B32 over an 8-entry magnitude table plus the sign bit per
// four codes; two's-complement nibbles a 16-entry table (three permutes).
// The activations arrive as ready FP6/FP8 digits (decode image).
// V_MFMA_SCALE_F32_16X16X128_F8F6F4 multiplies 16 rows by
// 16 columns over four K-blocks and applies every block's E8M0 scale in
// hardware, so no per-block rescale runs on the VALU.  Digit products are
// exact; a 6/8-bit block pair takes two instructions (the second with the
// weight digits' halves swapped: h*h + l*l, then h*l + l*h).
//
// Work decomposition: one workgroup per 16-column slab, its nw waves taking
// every nw-th step of each width segment (nw from 2 to 8, so that every slab
// of the grid is resident at once at about 16 waves per CU).  Each wave
// keeps two stages of loads in flight: the next stage (four 4-bit or two
// 6/8-bit steps) is issued before the current one is converted and
// multiplied.  The waves' fp32 accumulators meet in LDS in a fixed order.
// Activation loads of rows >= M are predicated off.
#include <type_traits>

#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef unsigned u2 __attribute__((ext_vector_type(2)));


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

// Sign-magnitude codes (symmetric clamp): 8-entry magnitude tables, entry
// k = e4m3(k / den), as two dwords; the 2-bit high part of a 6-bit
// magnitude (|q| div 8) -> e4m3(h/2).
constexpr uint32_t mag_dword(int den, int d) {
  uint32_t v = 0;
  for (int k = 0; k < 4; ++k) v |= e4m3_exact(4 * d + k, den) << (8 * k);
  return v;
}
constexpr uint32_t kTop6m = e4m3_exact(0, 2) | (e4m3_exact(1, 2) << 8) |
                            (e4m3_exact(2, 2) << 16) | (e4m3_exact(3, 2) << 24);

// e4m3 digits of the low / high nibble codes of x (sign at bit 3 of each
// nibble, magnitude index in bits 0-2): one byte permute and the sign bit.
template <int DEN>
__device__ inline uint32_t mag_lo(uint32_t x) {
  const uint32_t c = __builtin_amdgcn_perm(mag_dword(DEN, 1), mag_dword(DEN, 0), x & 0x07070707u);
  return c | ((x & 0x08080808u) << 4);
}
template <int DEN>
__device__ inline uint32_t mag_hi(uint32_t x) {
  const uint32_t c =
      __builtin_amdgcn_perm(mag_dword(DEN, 1), mag_dword(DEN, 0), (x >> 4) & 0x07070707u);
  return c | (x & 0x80808080u);
}

// Byte-wise lookup: byte k of s holds an index in its low nibble.
template <int KIND>
__device__ inline uint32_t lut16(uint32_t s) {
  const uint32_t s7 = s & 0x07070707u;
  const uint32_t lo = __builtin_amdgcn_perm(table_dword<KIND>(1), table_dword<KIND>(0), s7);
  const uint32_t hi = __builtin_amdgcn_perm(table_dword<KIND>(3), table_dword<KIND>(2), s7);
  const uint32_t sel = ((s >> 1) & 0x04040404u) | 0x03020100u;
  return __builtin_amdgcn_perm(hi, lo, sel);
}

constexpr int kU4 = 4;     // 4-bit steps per pipeline stage
constexpr int kU68 = 2;    // 6/8-bit steps per pipeline stage
constexpr int kMaxWaves = 8;

__device__ inline v4f mfma(const v8i &a, const v8i &b, v4f acc, int fa, uint32_t as,
                           uint32_t ws) {
  if (fa == 3)
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, acc, 3, 0, 0, (int)as, 0,
                                                            (int)ws);
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, acc, 0, 0, 0, (int)as, 0,
                                                          (int)ws);
}

// FP8 digits of the 16 weight elements of a 4-bit lane (four nibble dwords).
template <bool SM>
__device__ inline v8i digits4(const u4 &w) {
  v8i b;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (SM) {
      b[2 * i] = (int)mag_lo<4>(w[i]);
      b[2 * i + 1] = (int)mag_hi<4>(w[i]);
    } else {
      b[2 * i] = (int)lut16<0>(w[i]);
      b[2 * i + 1] = (int)lut16<0>(w[i] >> 4);
    }
  }
  return b;
}

// High and low FP8 digits of the 16 elements of a 6- or 8-bit weight lane.
template <bool SM, int SEG>
__device__ inline void digits68(const u4 &w, uint32_t (&hd)[4], uint32_t (&ld)[4]) {
  if (SEG == 1 && SM) {
    // |q| = 8h + l: low digits l/16 from the nibble codes (with the sign),
    // high digits h/2 from the 2-bit codes plus the same sign
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      ld[2 * i] = mag_lo<16>(w[i]);
      ld[2 * i + 1] = mag_hi<16>(w[i]);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t x = w[q >> 1];
      const uint32_t sg = (q & 1) ? (x & 0x80808080u) : ((x & 0x08080808u) << 4);
      hd[q] = __builtin_amdgcn_perm(0u, kTop6m, (w[2] >> (2 * q)) & 0x03030303u) | sg;
    }
  } else if (SEG == 1) {
    // q = 16h + l: low digits from the nibbles, high from the 2-bit codes
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      ld[2 * i] = lut16<1>(w[i]);
      ld[2 * i + 1] = lut16<1>(w[i] >> 4);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q)
      hd[q] = __builtin_amdgcn_perm(0u, kTop6, (w[2] >> (2 * q)) & 0x03030303u);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ld[i] = lut16<2>(w[i]);
      hd[i] = lut16<0>(w[i] >> 4);
    }
  }
}

template <bool SM>
__global__ __launch_bounds__(64 * kMaxWaves) void gemm_decode_kernel(GemmArgs g) {
  __shared__ v4f red[kMaxWaves][64];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int nw = blockDim.x >> 6;
  const int line = lane & 15;
  const DGeo d(g.n4, g.n6, g.n8);
  const int64_t slab = blockIdx.x;
  const uint8_t *wslab = g.w_mant + slab * wd_slab_bytes(d);
  const uint8_t *aimg = g.a_mant + g.a_op;
  const bool arow = line < g.M;
  v4f acc = {0.f, 0.f, 0.f, 0.f};

  // Lanes of rows >= M read row 0's activation bytes (same addresses as a
  // live lane, so no extra traffic); their output rows are discarded.
  const int alane = arow ? lane : (lane & ~15);

  // Pipelined walk over the steps s0, s0 + nw, ... (< n) of one segment:
  // "full" stages of U steps (every step present) alternate between two
  // register buffers with no branch between a stage's loads and its use,
  // so each stage waits only for its own loads; the last prefetch is
  // clamped to the final stage.  The remaining steps run one at a time.
  auto pipeline = [&](int s0, int U, int n, auto &&load, auto &&comp, auto &&tail) {
    const int stride = nw * U;
    const int nf = s0 + (U - 1) * nw < n ? (n - 1 - s0 - (U - 1) * nw) / stride + 1 : 0;
    if (nf > 0) {
      load(0, s0);
      int i = 0;
      for (; i + 1 < nf; i += 2) {
        load(1, s0 + (i + 1) * stride);
        comp(0);
        load(0, s0 + (i + 2 < nf ? i + 2 : nf - 1) * stride);
        comp(1);
      }
      if (i < nf) comp(0);
    }
    for (int sk = s0 + nf * stride; sk < n; sk += nw) tail(sk);
  };

  // 4-bit steps: A e3m2 (format 3) x W e4m3 (format 0), one instruction per
  // step; the wave takes steps wave, wave + nw, ...
  {
    u4 w[2][kU4], a0[2][kU4];
    u2 a1[2][kU4];
    uint32_t ws[2][kU4], as[2][kU4];
    auto load = [&](int buf, int s) {
#pragma unroll
      for (int k = 0; k < kU4; ++k) {
        const uint8_t *wc = wslab + (int64_t)(s + k * nw) * wd_chunk(0);
        const uint8_t *ac = aimg + (int64_t)(s + k * nw) * ad_chunk(0);
        w[buf][k] = *(const u4 *)(wc + 16 * lane);
        ws[buf][k] = wc[1024 + lane];
        a0[buf][k] = *(const u4 *)(ac + 16 * alane);
        a1[buf][k] = *(const u2 *)(ac + 1024 + 8 * alane);
        as[buf][k] = ac[1536 + alane];
      }
    };
    auto comp = [&](int buf) {
#pragma unroll
      for (int k = 0; k < kU4; ++k) {
        const v8i b = digits4<SM>(w[buf][k]);
        const v8i a = {(int)a0[buf][k][0], (int)a0[buf][k][1], (int)a0[buf][k][2],
                       (int)a0[buf][k][3], (int)a1[buf][k][0], (int)a1[buf][k][1], 0, 0};
        acc = mfma(a, b, acc, 3, as[buf][k], ws[buf][k]);
      }
    };
    auto tail = [&](int sk) {
      const uint8_t *wc = wslab + (int64_t)sk * wd_chunk(0);
      const uint8_t *ac = aimg + (int64_t)sk * ad_chunk(0);
      const u4 x = *(const u4 *)(wc + 16 * lane);
      const u4 p = *(const u4 *)(ac + 16 * alane);
      const u2 q = *(const u2 *)(ac + 1024 + 8 * alane);
      const v8i a = {(int)p[0], (int)p[1], (int)p[2], (int)p[3], (int)q[0], (int)q[1], 0, 0};
      acc = mfma(a, digits4<SM>(x), acc, 3, ac[1536 + alane], wc[1024 + lane]);
    };
    pipeline(wave, kU4, d.S4, load, comp, tail);
  }

  // 6-bit and 8-bit steps: FP8 digits on both sides, two instructions per
  // step (the weight digits' halves swapped in the second)
  auto run68 = [&](auto segc) {
    constexpr int SEG = decltype(segc)::value;
    constexpr int lb = wd_lane_bytes(SEG);
    const int sb = SEG == 1 ? d.S4 : d.S4 + d.S6;
    const int n = SEG == 1 ? d.S6 : d.S8;
    const uint8_t *wseg = wslab + wd_step_off(d, sb);
    const uint8_t *aseg = aimg + ad_step_off(d, sb);
    u4 w[2][kU68], a0[2][kU68], a1[2][kU68];
    uint32_t ws[2][kU68], as[2][kU68];
    auto load1 = [&](int sk, u4 &wv, u4 &p0, u4 &p1, uint32_t &wsv, uint32_t &asv) {
      const uint8_t *wc = wseg + (int64_t)sk * wd_chunk(SEG);
      const uint8_t *ac = aseg + (int64_t)sk * ad_chunk(SEG);
      if (SEG == 1) {
        const u2 nb = *(const u2 *)(wc + 8 * lane);
        wv = u4{nb[0], nb[1], *(const uint32_t *)(wc + 512 + 4 * lane), 0u};
      } else {
        wv = *(const u4 *)(wc + 16 * lane);
      }
      wsv = wc[64 * lb + lane];
      p0 = *(const u4 *)(ac + 32 * alane);
      p1 = *(const u4 *)(ac + 32 * alane + 16);
      asv = ac[2048 + alane];
    };
    auto mul = [&](const u4 &wv, const u4 &p0, const u4 &p1, uint32_t wsv, uint32_t asv) {
      uint32_t hd[4], ld[4];
      digits68<SM, SEG>(wv, hd, ld);
      const v8i a = {(int)p0[0], (int)p0[1], (int)p0[2], (int)p0[3],
                     (int)p1[0], (int)p1[1], (int)p1[2], (int)p1[3]};
      const v8i bhl = {(int)hd[0], (int)hd[1], (int)hd[2], (int)hd[3],
                       (int)ld[0], (int)ld[1], (int)ld[2], (int)ld[3]};
      const v8i blh = {(int)ld[0], (int)ld[1], (int)ld[2], (int)ld[3],
                       (int)hd[0], (int)hd[1], (int)hd[2], (int)hd[3]};
      acc = mfma(a, bhl, acc, 0, asv, wsv);
      acc = mfma(a, blh, acc, 0, asv, wsv);
    };
    auto load = [&](int buf, int s) {
#pragma unroll
      for (int k = 0; k < kU68; ++k)
        load1(s + k * nw, w[buf][k], a0[buf][k], a1[buf][k], ws[buf][k], as[buf][k]);
    };
    auto comp = [&](int buf) {
#pragma unroll
      for (int k = 0; k < kU68; ++k) mul(w[buf][k], a0[buf][k], a1[buf][k], ws[buf][k], as[buf][k]);
    };
    auto tail = [&](int sk) {
      u4 wv, p0, p1;
      uint32_t wsv, asv;
      load1(sk, wv, p0, p1, wsv, asv);
      mul(wv, p0, p1, wsv, asv);
    };
    pipeline(wave, kU68, n, load, comp, tail);
  };
  run68(std::integral_constant<int, 1>());
  run68(std::integral_constant<int, 2>());

  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    v4f y = red[0][lane];
    for (int w = 1; w < nw; ++w) y += red[w][lane];
    const int64_t col = slab * 16 + line;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * (lane >> 4) + i;
      if (row < g.M && col < g.N) g.y[row * g.ldy + col] = y[i];
    }
  }
}

}  // namespace

// Waves per workgroup (one workgroup per 16-column slab): enough for about
// 16 waves per CU when every slab is resident at once (2 for 1792 slabs,
// 8 for 512 slabs).
static int decode_waves(int64_t slabs) {
  int cus = 256;
  int dev = 0;
  if (hipGetDevice(&dev) == hipSuccess) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        n > 0)
      cus = n;
  }
  int64_t w = (16LL * cus + slabs - 1) / slabs;
  if (w < 2) w = 2;
  if (w > kMaxWaves) w = kMaxWaves;
  return (int)w;
}

hipError_t launch_gemm_decode(const GemmArgs &a, hipStream_t stream) {
  const int64_t slabs = a.npad / 16;
  dim3 grid((unsigned)slabs), block((unsigned)(64 * decode_waves(slabs)));
  if (a.sm)
    hipLaunchKernelGGL(gemm_decode_kernel<true>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(gemm_decode_kernel<false>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
