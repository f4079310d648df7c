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
// Work decomposition: the kernel is bound by the number of vector memory
// loads, so each load serves as many products as possible.  A workgroup
// owns a pair of 16-column slabs (one activation load feeds both), its nw
// waves (2 to 16, about 16 waves per CU with every pair resident) taking
// every nw-th group of four steps of each width segment; a group's scale
// bytes are one dword per lane and operand (op_sel picks the step).  The
// waves' fp32 accumulators meet in LDS in a fixed order.
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

// The packed weights are read exactly once: non-temporal loads stream them
// past the caches (measured on gfx950: 6.9 TB/s for a plain streaming read
// against 6.2 TB/s with ordinary loads).  Activations stay cached; every
// workgroup reads them.
template <typename T>
__device__ inline T stream_load(const T *p) {
  return __builtin_nontemporal_load(p);
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

constexpr int kMaxWaves = 16;

// Block-scaled 16x16x128 product; the scale bytes of step K of a group sit
// in byte K of the scale dwords (op_sel).  FA: format of A (3 = e3m2 FP6,
// 0 = e4m3 FP8); B is e4m3.
template <int FA, int K>
__device__ inline v4f mfma(const v8i &a, const v8i &b, v4f acc, uint32_t as, uint32_t ws) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, acc, FA, 0, K, (int)as, K,
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
  __shared__ v4f red[kMaxWaves][2][64];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int nw = blockDim.x >> 6;
  const int line = lane & 15;
  const DGeo d(g.n4, g.n6, g.n8);
  const int64_t nslab = g.npad / 16;
  const int64_t slab0 = 2 * (int64_t)blockIdx.x;
  const bool two = slab0 + 1 < nslab;
  const int64_t sb = wd_slab_bytes(d);
  const uint8_t *wsl0 = g.w_mant + slab0 * sb;
  const uint8_t *wsl1 = two ? wsl0 + sb : wsl0;
  const uint8_t *aimg = g.a_mant + g.a_op;
  // Lanes of rows >= M read row 0's activation bytes (same addresses as a
  // live lane, so no extra traffic); their output rows are discarded.
  const int alane = line < g.M ? lane : (lane & ~15);
  v4f acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};

  // One group of up to four steps of a segment for both slabs: all loads
  // first, then the products.  FULL groups carry no per-step guards.
  auto group4 = [&](int gi, int nst) {
    constexpr int sd = wd_step_data(0), ad = ad_step_data(0);
    const uint8_t *g0 = wsl0 + grp_off(gi, sd), *g1 = wsl1 + grp_off(gi, sd);
    const uint8_t *ga = aimg + grp_off(gi, ad);
    const uint32_t sw0 = stream_load((const uint32_t *)(g0 + 4 * lane));
    const uint32_t sw1 = stream_load((const uint32_t *)(g1 + 4 * lane));
    const uint32_t sa = *(const uint32_t *)(ga + 4 * alane);
    u4 x0[4], x1[4], p[4];
    u2 q[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x0[k] = x1[k] = p[k] = u4{0u, 0u, 0u, 0u};
      q[k] = u2{0u, 0u};
      if (k < nst) {
        x0[k] = stream_load((const u4 *)(g0 + kScaleBlock + k * sd + 16 * lane));
        x1[k] = stream_load((const u4 *)(g1 + kScaleBlock + k * sd + 16 * lane));
        p[k] = *(const u4 *)(ga + kScaleBlock + k * ad + 16 * alane);
        q[k] = *(const u2 *)(ga + kScaleBlock + k * ad + 1024 + 8 * alane);
      }
    }
    // steps past a short group are skipped: their scale bytes are
    // unspecified (an E8M0 NaN would poison even zero products)
    auto step = [&](auto kc) {
      constexpr int k = decltype(kc)::value;
      if (k >= nst) return;
      const v8i a = {(int)p[k][0], (int)p[k][1], (int)p[k][2], (int)p[k][3],
                     (int)q[k][0], (int)q[k][1], 0, 0};
      acc0 = mfma<3, k>(a, digits4<SM>(x0[k]), acc0, sa, sw0);
      acc1 = mfma<3, k>(a, digits4<SM>(x1[k]), acc1, sa, sw1);
    };
    step(std::integral_constant<int, 0>());
    step(std::integral_constant<int, 1>());
    step(std::integral_constant<int, 2>());
    step(std::integral_constant<int, 3>());
  };

  // 4-bit steps: A e3m2 (FP6) x W e4m3, one instruction per step and slab;
  // the wave takes groups wave, wave + nw, ...
  {
    const int S = d.S[0], nfg = S / kStreamGroup, rem = S % kStreamGroup;
    for (int gi = wave; gi < nfg; gi += nw) group4(gi, kStreamGroup);
    if (rem && wave == nfg % nw) group4(nfg, rem);
  }

  // 6-bit and 8-bit steps: FP8 digits on both sides, two instructions per
  // step and slab (the weight digits' halves swapped in the second)
  auto run68 = [&](auto segc) {
    constexpr int SEG = decltype(segc)::value;
    constexpr int sd = wd_step_data(SEG), ad = ad_step_data(SEG);
    const uint8_t *w0 = wsl0 + wd_seg_off(d, SEG), *w1 = wsl1 + wd_seg_off(d, SEG);
    const uint8_t *a0 = aimg + ad_seg_off(d, SEG);
    auto group = [&](int gi, int nst) {
      const uint8_t *g0 = w0 + grp_off(gi, sd), *g1 = w1 + grp_off(gi, sd);
      const uint8_t *ga = a0 + grp_off(gi, ad);
      const uint32_t sw0 = stream_load((const uint32_t *)(g0 + 4 * lane));
      const uint32_t sw1 = stream_load((const uint32_t *)(g1 + 4 * lane));
      const uint32_t sa = *(const uint32_t *)(ga + 4 * alane);
      u4 x0[4], x1[4], p[4], r[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        x0[k] = x1[k] = p[k] = r[k] = u4{0u, 0u, 0u, 0u};
        if (k < nst) {
          const uint8_t *c0 = g0 + kScaleBlock + k * sd, *c1 = g1 + kScaleBlock + k * sd;
          if (SEG == 1) {
            const u2 n0 = stream_load((const u2 *)(c0 + 8 * lane));
            const u2 n1 = stream_load((const u2 *)(c1 + 8 * lane));
            x0[k] = u4{n0[0], n0[1], stream_load((const uint32_t *)(c0 + 512 + 4 * lane)), 0u};
            x1[k] = u4{n1[0], n1[1], stream_load((const uint32_t *)(c1 + 512 + 4 * lane)), 0u};
          } else {
            x0[k] = stream_load((const u4 *)(c0 + 16 * lane));
            x1[k] = stream_load((const u4 *)(c1 + 16 * lane));
          }
          const uint8_t *ca = ga + kScaleBlock + k * ad + 32 * alane;
          p[k] = *(const u4 *)ca;
          r[k] = *(const u4 *)(ca + 16);
        }
      }
      auto step = [&](auto kc) {
        constexpr int k = decltype(kc)::value;
        if (k >= nst) return;
        const v8i a = {(int)p[k][0], (int)p[k][1], (int)p[k][2], (int)p[k][3],
                       (int)r[k][0], (int)r[k][1], (int)r[k][2], (int)r[k][3]};
        uint32_t hd[4], ld[4];
        digits68<SM, SEG>(x0[k], hd, ld);
        v8i bhl = {(int)hd[0], (int)hd[1], (int)hd[2], (int)hd[3],
                   (int)ld[0], (int)ld[1], (int)ld[2], (int)ld[3]};
        v8i blh = {(int)ld[0], (int)ld[1], (int)ld[2], (int)ld[3],
                   (int)hd[0], (int)hd[1], (int)hd[2], (int)hd[3]};
        acc0 = mfma<0, k>(a, bhl, acc0, sa, sw0);
        acc0 = mfma<0, k>(a, blh, acc0, sa, sw0);
        digits68<SM, SEG>(x1[k], hd, ld);
        bhl = v8i{(int)hd[0], (int)hd[1], (int)hd[2], (int)hd[3],
                  (int)ld[0], (int)ld[1], (int)ld[2], (int)ld[3]};
        blh = v8i{(int)ld[0], (int)ld[1], (int)ld[2], (int)ld[3],
                  (int)hd[0], (int)hd[1], (int)hd[2], (int)hd[3]};
        acc1 = mfma<0, k>(a, bhl, acc1, sa, sw1);
        acc1 = mfma<0, k>(a, blh, acc1, sa, sw1);
      };
      step(std::integral_constant<int, 0>());
      step(std::integral_constant<int, 1>());
      step(std::integral_constant<int, 2>());
      step(std::integral_constant<int, 3>());
    };
    const int S = d.S[SEG], nfg = S / kStreamGroup, rem = S % kStreamGroup;
    for (int gi = wave; gi < nfg; gi += nw) group(gi, kStreamGroup);
    if (rem && wave == nfg % nw) group(nfg, rem);
  };
  run68(std::integral_constant<int, 1>());
  run68(std::integral_constant<int, 2>());

  red[wave][0][lane] = acc0;
  red[wave][1][lane] = acc1;
  __syncthreads();
  if (wave < 2 && (wave == 0 || two)) {
    v4f y = red[0][wave][lane];
    for (int w = 1; w < nw; ++w) y += red[w][wave][lane];
    const int64_t col = (slab0 + wave) * 16 + line;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * (lane >> 4) + i;
      if (row < g.M && col < g.N) g.y[row * g.ldy + col] = y[i];
    }
  }
}

}  // namespace

// Waves per workgroup (one workgroup per pair of 16-column slabs): enough
// for about 16 waves per CU when every pair is resident at once (4 for 896
// pairs, 16 for 256 pairs).
static int decode_waves(int64_t pairs) {
  int cus = 256;
  int dev = 0;
  if (hipGetDevice(&dev) == hipSuccess) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        n > 0)
      cus = n;
  }
  int64_t w = 16LL * cus / pairs;      // rounded down: every pair stays resident
  if (w < 2) w = 2;
  if (w > kMaxWaves) w = kMaxWaves;
  return (int)w;
}

hipError_t launch_gemm_decode(const GemmArgs &a, hipStream_t stream) {
  const int64_t pairs = (a.npad / 16 + 1) / 2;
  dim3 grid((unsigned)pairs), block((unsigned)(64 * decode_waves(pairs)));
  if (a.sm)
    hipLaunchKernelGGL(gemm_decode_kernel<true>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(gemm_decode_kernel<false>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
