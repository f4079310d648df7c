// decode.hip -- MXINT GEMM for decode shapes (M <= 16), streaming the
// weights at HBM rate.
//
// Y[i][j] = sum_b 2^(sa[i][b] + sw[j][b]) * sum_t qa qw  (MXSens, arXiv
// 2607.17733, Section 2: integer block products with power-of-two block
// scales; Section 6: the memory cost is the packed weights).
//
// The weights are read in the one layout both GEMMs share (LGeo in
// mxq_device.h): folded FP6 codes for 3- and 4-bit blocks, two digit planes
// for 6-bit blocks, mantissa bytes for 8-bit blocks, at the MXINT size.  The
// lane restores its FP6 operand with a few masks and shifts (FP8 digit codes
// of an 8-bit block from its bytes), and V_MFMA_SCALE_F32_16X16X128_F8F6F4
// multiplies 16 activation rows by 16 columns over four K-blocks, applying
// every block's E8M0 scale in hardware.  A 6- or 8-bit step (two blocks,
// each as its two digit planes) takes two instructions: the weights' high
// plane in every lane (scale E + 3 or E + 4), then their low plane.  The
// activations arrive as ready FP6/FP8 codes (the operand image).
//
// Work decomposition: the kernel is bound by the number of vector memory
// loads, so each load serves as many products as possible.  Each weight
// step is read once for all of the launch's 16-row activation tiles (up to
// four: M <= 64).  A workgroup
// owns a unit of four 16-column slabs, or two where four would leave CUs
// without a workgroup, or (M <= 16) one unit of 5 to 7 consecutive slabs
// per CU where that balances the CUs (one activation load feeds all of
// them); its nw waves
// (2 to 8, the most at which every unit is resident by the kernel's register
// occupancy) take every nw-th group of four steps; a group's scale bytes are
// one word per lane and operand.  The waves' fp32 accumulators meet in LDS
// in a fixed order.
#include <atomic>
#include <type_traits>

#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef unsigned u2 __attribute__((ext_vector_type(2)));
typedef unsigned u3 __attribute__((ext_vector_type(3)));

constexpr int kFmtE4M3 = 0, kFmtE2M3 = 2, kFmtE3M2 = 3;
constexpr int kMaxWaves = 8;
constexpr int kDecodeTiles = 4;             // 16-row activation tiles per launch
static_assert(16 * kDecodeTiles == MXQ_DECODE_MAX_M, "decode rows");

// The weights are read exactly once: non-temporal loads stream them past the
// caches.  Activations stay cached; every workgroup reads them.
template <typename T>
__device__ inline T stream_load(const T *p) {
  return __builtin_nontemporal_load(p);
}

template <int FA, int FB, int K>
__device__ inline v4f mfma(const v8i &a, const v8i &b, v4f acc, uint32_t as, uint32_t ws) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, acc, FA, FB, K, (int)as, K,
                                                          (int)ws);
}

// E8M0 scale e + n, saturating at 255 (NaN), per byte of a scale word.
template <int N>
__device__ inline uint32_t scale_plus(uint32_t w) {
  const uint32_t lo = (w & 0x00FF00FFu) + (N | (N << 16));
  const uint32_t hi = ((w >> 8) & 0x00FF00FFu) + (N | (N << 16));
  const uint32_t lo_s = lo | (((lo & 0x01000100u) >> 8) * 0xFFu);
  const uint32_t hi_s = hi | (((hi & 0x01000100u) >> 8) * 0xFFu);
  return (lo_s & 0x00FF00FFu) | ((hi_s & 0x00FF00FFu) << 8);
}

__device__ inline v8i six(const uint32_t *d) {
  const u4 a = u4{d[0], d[1], d[2], d[3]};
  const u2 b = u2{d[4], d[5]};
  const u4 b4 = __builtin_shufflevector(b, b, 0, 1, -1, -1);
  return (v8i)__builtin_shufflevector(a, b4, 0, 1, 2, 3, 4, 5, 6, 7);
}

// FP8 digit codes of 4 mantissa bytes: the high plane (+-h/512) and the low
// plane (+-l/512); sign-magnitude bytes (|q| = 16h + l) or, with FULL, two's
// complement (h = q >> 4 signed, l = q & 15).
template <bool FULL>
__device__ inline uint32_t hi_codes(uint32_t w) {
  if (!FULL) return ((w >> 4) & 0x07070707u) | (w & 0x80808080u);
  const uint32_t x = (w >> 4) & 0x0F0F0F0Fu;
  const uint32_t s = (x >> 3) & 0x01010101u;
  const uint32_t mag = (x ^ (s * 0x0Fu)) + s;
  return mag | (s << 7);
}
template <bool FULL>
__device__ inline uint32_t lo_codes(uint32_t w) {
  return FULL ? (w & 0x0F0F0F0Fu) : (w & 0x8F8F8F8Fu);
}

// T: 16-row activation tiles (M <= 16 T); SL: 16-column slabs per
// workgroup (one activation load feeds all of them).  A unit is SL
// consecutive slabs; with 2 or 4 it lies inside one 128-column super-slab,
// with 5 to 7 (one unit per CU where that balances the CUs) it may cross
// into the next super-slab.
template <bool FULL, int T, int SL>
__global__ __launch_bounds__(64 * kMaxWaves) void gemm_decode_kernel(GemmArgs g) {
  __shared__ v4f red[kMaxWaves][SL][64];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int nw = blockDim.x >> 6;
  const int grp = lane >> 4, line = lane & 15;
  const LGeo lg(g.n3, g.n4, g.n6, g.n8);
  // Aligned units: the units of a super-slab run on one XCD (workgroups b,
  // b + 8, ... of a round-robin dispatch), so its L2 reads each step record
  // of the super-slab and its scale block whole.  Crossing units: each XCD
  // takes a contiguous range of units, whose super-slabs it then shares.
  constexpr bool ALIGNED = kWSlabs % SL == 0;
  int64_t unit = blockIdx.x;
  if (ALIGNED) {
    constexpr int PPS = kWSlabs / SL;                // units per super-slab
    if ((gridDim.x % (8 * PPS)) == 0) {
      const int64_t x = unit & 7, i = unit >> 3;
      unit = ((i / PPS) * 8 + x) * PPS + (i % PPS);
    }
  } else if ((gridDim.x & 7) == 0) {
    unit = (unit & 7) * (gridDim.x >> 3) + (unit >> 3);
  }
  const int64_t gs0 = unit * SL;                     // first slab of the unit
  const int64_t ss = gs0 / kWSlabs;                  // its super-slab
  const int n0 = (int)(gs0 % kWSlabs);               // its slab in the super-slab
  // slabs past N (inside the padded super-slab) read the unit's first slab
  auto live = [&](int sl) { return gs0 * 16 + 16 * sl < g.N; };
  // slab sl lies in super-slab ss + 1 when n0 + sl >= 8 (at most one
  // crossing); cross: some live slab of the unit does
  const bool cross = !ALIGNED && n0 + SL > kWSlabs && (ss + 1) * kWCols < g.N;
  const uint8_t *wsup = g.w_mant + ss * g.w_super;
  const uint8_t *wsc = g.w_exp + ss * g.w_super_sc + 32 * lane;
  const uint8_t *wsc2 = cross ? wsc + g.w_super_sc : wsc;
  // Lanes of rows >= M read the first row of their tile (same addresses as a
  // live lane, so no extra traffic); their output rows are discarded.
  int alane[T];
#pragma unroll
  for (int t = 0; t < T; ++t) alane[t] = 16 * t + line < g.M ? lane : (lane & ~15);
  v4f acc[T][SL];
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int sl = 0; sl < SL; ++sl) acc[t][sl] = v4f{0.f, 0.f, 0.f, 0.f};

  auto run_group = [&](auto segc, int gi) {
    constexpr int SEG = decltype(segc)::value;
    constexpr int CB = w_chunk_bytes(SEG, FULL);
    const int gl = gi - lg.G0[SEG];
    const int nst = min(4, lg.S[SEG] - 4 * gl);
    // the lane's scale bytes of the group: byte 8 k + n for step k, slab n;
    // sw[sl] gathers the four steps' bytes of slab n0 + sl (of the next
    // super-slab's block past slab 7)
    const u4 s0 = stream_load((const u4 *)(wsc + (int64_t)gi * 2048));
    const u4 s1 = stream_load((const u4 *)(wsc + (int64_t)gi * 2048 + 16));
    u4 t0 = s0, t1 = s1;
    if (!ALIGNED) {
      t0 = stream_load((const u4 *)(wsc2 + (int64_t)gi * 2048));
      t1 = stream_load((const u4 *)(wsc2 + (int64_t)gi * 2048 + 16));
    }
    // step k's byte of slab b lies in dword 2k + b / 4
    uint32_t sw[SL];
#pragma unroll
    for (int sl = 0; sl < SL; ++sl) {
      const bool hi = !ALIGNED && n0 + sl >= kWSlabs;
      const int b = (n0 + sl) & (kWSlabs - 1);
      const u4 x0 = hi ? t0 : s0, x1 = hi ? t1 : s1;
      const uint32_t d0 = b < 4 ? x0[0] : x0[1], d1 = b < 4 ? x0[2] : x0[3];
      const uint32_t d2 = b < 4 ? x1[0] : x1[1], d3 = b < 4 ? x1[2] : x1[3];
      const int sh = 8 * (b & 3);
      sw[sl] = ((d0 >> sh) & 0xFFu) | (((d1 >> sh) & 0xFFu) << 8) | (((d2 >> sh) & 0xFFu) << 16) |
               (((d3 >> sh) & 0xFFu) << 24);
    }
    uint32_t sa[T];
#pragma unroll
    for (int t = 0; t < T; ++t)
      sa[t] = *(const uint32_t *)(g.a_exp + t * g.a_tile_sc + (int64_t)gi * 256 + 4 * alane[t]);
    const uint8_t *wseg = wsup + w_seg_base<SEG, FULL>(lg) + (int64_t)(4 * gl) * kWSlabs * CB +
                          (int64_t)n0 * CB;
    const uint8_t *aseg = g.a_mant + a_seg_base<SEG>(lg) +
                          (int64_t)(4 * gl) * kLanes * a_lane_bytes(SEG);
    // raw loads of step k (fields a segment does not use stay unread)
    struct Raw {
      u4 a0[T], a1[T];      // activation lane data (24 or 32 bytes) per tile
      u4 p[SL], h[SL];      // weight bytes of the slabs
      u2 x[SL];
      uint32_t z[SL];
    };
    auto load = [&](int k) __attribute__((always_inline)) {
      Raw r;
      const uint8_t *w0 = wseg + (int64_t)k * kWSlabs * CB;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const uint8_t *ap = aseg + t * g.a_tile + (int64_t)k * kLanes * a_lane_bytes(SEG) +
                            (int64_t)a_lane_bytes(SEG) * alane[t];
        if (SEG == 3) {
          r.a0[t] = *(const u4 *)ap;
          r.a1[t] = *(const u4 *)(ap + 16);
        } else {
          r.a0[t] = *(const u4 *)ap;
          const u2 aw = *(const u2 *)(ap + 16);
          r.a1[t] = __builtin_shufflevector(aw, aw, 0, 1, -1, -1);
        }
      }
#pragma unroll
      for (int sl = 0; sl < SL; ++sl) {
        // a slab past slab 7 lies in the next super-slab, at the same offset
        const int64_t next = (!ALIGNED && n0 + sl >= kWSlabs) ? g.w_super - (int64_t)kWSlabs * CB : 0;
        const uint8_t *w = live(sl) ? w0 + sl * CB + next : w0;
        if (SEG == 0 && !FULL) {
          r.x[sl] = stream_load((const u2 *)(w + 8 * lane));
          r.z[sl] = stream_load((const uint32_t *)(w + 512 + 4 * lane));
        } else if (SEG <= 1) {
          r.p[sl] = stream_load((const u4 *)(w + 16 * lane));
          if (SEG == 1 && FULL) r.x[sl] = stream_load((const u2 *)(w + 1024 + 8 * lane));
        } else if (SEG == 2) {
          const int jc = 16 * (grp >> 1) + line;
          r.p[sl] = stream_load((const u4 *)(w + 16 * jc));
          if (FULL) r.h[sl] = stream_load((const u4 *)(w + 512 + 16 * jc));
          else r.x[sl] = stream_load((const u2 *)(w + 512 + 8 * jc));
        } else {
          r.p[sl] = stream_load((const u4 *)(w + 32 * line + 16 * (grp & 1)));
          r.h[sl] = stream_load((const u4 *)(w + 32 * (16 + line) + 16 * (grp & 1)));
        }
      }
      return r;
    };
    auto compute = [&](auto kc, const Raw &r) __attribute__((always_inline)) {
      constexpr int k = decltype(kc)::value;
      v8i a[T];
#pragma unroll
      for (int t = 0; t < T; ++t)
        a[t] = v8i{(int)r.a0[t][0], (int)r.a0[t][1], (int)r.a0[t][2], (int)r.a0[t][3],
                   (int)r.a1[t][0], (int)r.a1[t][1], (int)r.a1[t][2], (int)r.a1[t][3]};
      if (SEG <= 1) {
        uint32_t d[SL][6];
#pragma unroll
        for (int sl = 0; sl < SL; ++sl) {
          if (SEG == 0 && !FULL) {
            const uint32_t x[3] = {r.x[sl][0], r.x[sl][1], r.z[sl]};
            unfold3(x, d[sl]);
          } else if (SEG == 1 && FULL) {
#pragma unroll
            for (int i = 0; i < 4; ++i) d[sl][i] = r.p[sl][i];
            d[sl][4] = r.x[sl][0];
            d[sl][5] = r.x[sl][1];
          } else {
            const uint32_t x[4] = {r.p[sl][0], r.p[sl][1], r.p[sl][2], r.p[sl][3]};
            unfold4(x, d[sl]);
          }
        }
        constexpr int FB = SEG == 0 ? kFmtE2M3 : kFmtE3M2;
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
          for (int sl = 0; sl < SL; ++sl)
            acc[t][sl] = mfma<kFmtE3M2, FB, k>(a[t], six(d[sl]), acc[t][sl], sa[t], sw[sl]);
      } else if (SEG == 2) {
        // the weights' high plane in every lane (scale E + 3) gives the
        // products hh and lh, their low plane (scale E) hl and ll
#pragma unroll
        for (int sl = 0; sl < SL; ++sl) {
          const uint32_t xl[4] = {r.p[sl][0], r.p[sl][1], r.p[sl][2], r.p[sl][3]};
          uint32_t L[6], H[6];
          unfold4(xl, L);
          if (FULL) {
            const uint32_t xh[4] = {r.h[sl][0], r.h[sl][1], r.h[sl][2], r.h[sl][3]};
            unfold4(xh, H);
          } else {
            const uint32_t xh[2] = {r.x[sl][0], r.x[sl][1]};
            unfold2(xh, L, H);
          }
          const uint32_t e = sw[sl];
#pragma unroll
          for (int t = 0; t < T; ++t) {
            acc[t][sl] = mfma<kFmtE3M2, kFmtE3M2, k>(a[t], six(H), acc[t][sl], sa[t], scale_plus<3>(e));
            acc[t][sl] = mfma<kFmtE3M2, kFmtE3M2, k>(a[t], six(L), acc[t][sl], sa[t], e);
          }
        }
      } else {
        // the weights' high digits in every lane (scale E + 4), then their
        // low digits (scale E)
#pragma unroll
        for (int sl = 0; sl < SL; ++sl) {
          v8i bh, bl;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const uint32_t w = i < 4 ? r.p[sl][i] : r.h[sl][i - 4];
            bh[i] = (int)hi_codes<FULL>(w);
            bl[i] = (int)lo_codes<FULL>(w);
          }
          const uint32_t e = sw[sl];
#pragma unroll
          for (int t = 0; t < T; ++t) {
            acc[t][sl] = mfma<kFmtE4M3, kFmtE4M3, k>(a[t], bh, acc[t][sl], sa[t], scale_plus<4>(e));
            acc[t][sl] = mfma<kFmtE4M3, kFmtE4M3, k>(a[t], bl, acc[t][sl], sa[t], e);
          }
        }
      }
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    if (T <= 2 && nst == 4) {
      // two steps in flight: each step's products, then the load two steps on
      const Raw r0 = load(0), r1 = load(1);
      compute(I0(), r0);
      const Raw r2 = load(2);
      compute(I1(), r1);
      const Raw r3 = load(3);
      compute(I2(), r2);
      compute(I3(), r3);
    } else {
      // one step at a time (three or four activation tiles, or a short
      // group, whose steps past its end are skipped)
      compute(I0(), load(0));
      if (nst > 1) compute(I1(), load(1));
      if (nst > 2) compute(I2(), load(2));
      if (nst > 3) compute(I3(), load(3));
    }
  };

  for (int gi = wave; gi < lg.ngroups; gi += nw) {
    if (gi < lg.G0[1]) run_group(std::integral_constant<int, 0>(), gi);
    else if (gi < lg.G0[2]) run_group(std::integral_constant<int, 1>(), gi);
    else if (gi < lg.G0[3]) run_group(std::integral_constant<int, 2>(), gi);
    else run_group(std::integral_constant<int, 3>(), gi);
  }

  // the waves' sums meet in LDS in wave order, one tile at a time
#pragma unroll
  for (int t = 0; t < T; ++t) {
    if (t > 0) __syncthreads();
#pragma unroll
    for (int sl = 0; sl < SL; ++sl) red[wave][sl][lane] = acc[t][sl];
    __syncthreads();
    for (int sl = wave; sl < SL; sl += nw) {
      if (!live(sl)) continue;
      v4f y = red[0][sl][lane];
      for (int w = 1; w < nw; ++w) y += red[w][sl][lane];
      const int64_t col = gs0 * 16 + 16 * sl + line;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * t + 4 * grp + i;
        if (row < g.M && col < g.N) g.y[row * g.ldy + col] = y[i];
      }
    }
  }
}

}  // namespace

// Waves per workgroup (one workgroup per unit of SL 16-column slabs): the
// most (up to kMaxWaves) at which every unit is resident at once, by the
// kernel's own occupancy (queried once per kernel and size; every GPU this
// runs on is the same model).
template <bool FULL, int T, int SL>
static int decode_waves(int64_t units, int cus) {
  static std::atomic<int> per_cu[kMaxWaves + 1] = {};
  for (int w = kMaxWaves; w > 2; --w) {
    int per = per_cu[w].load(std::memory_order_relaxed);
    if (per == 0) {
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, gemm_decode_kernel<FULL, T, SL>,
                                                       64 * w, 0) != hipSuccess ||
          per <= 0)
        break;
      per_cu[w].store(per, std::memory_order_relaxed);
    }
    if ((int64_t)per * cus >= units) return w;
  }
  return 2;
}

int device_cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
    return n;
  return 256;
}

hipError_t launch_gemm_decode(const GemmArgs &a, hipStream_t stream) {
  const int64_t tiles = (a.M + 15) / 16;
  if (tiles < 1 || tiles > kDecodeTiles) return hipErrorInvalidValue;
  const int cus = device_cu_count();
  // four slabs per workgroup (half the activation loads per weight byte)
  // when that still gives every CU a workgroup, else two; where the slabs
  // come to 5 to 7 per CU (M <= 16), one unit of that many per CU, since four-slab
  // units would give some CUs one unit and others two (the kernel takes as
  // long as its busiest CUs: 448 four-slab units on 256 CUs ran 26.1 us,
  // 512 ran 27.5 us)
  const bool quad = (a.N + 63) / 64 >= cus;
  const int64_t nslabs = (a.N + 15) / 16;
  const int64_t spc = (nslabs + cus - 1) / cus;
  auto go = [&](auto fc, auto tc) {
    constexpr bool FULL = decltype(fc)::value;
    constexpr int T = decltype(tc)::value;
    auto one_per_cu = [&](auto sc) {
      constexpr int SL = decltype(sc)::value;
      const int64_t units = (nslabs + SL - 1) / SL;
      const dim3 grid((unsigned)units), block((unsigned)(64 * decode_waves<FULL, T, SL>(units, cus)));
      hipLaunchKernelGGL((gemm_decode_kernel<FULL, T, SL>), grid, block, 0, stream, a);
    };
    // (one activation tile only: with more, units of 5 to 7 slabs spill)
    if (T == 1 && spc >= 5 && spc <= 7) {
      if constexpr (T == 1) {
        if (spc == 7) one_per_cu(std::integral_constant<int, 7>{});
        else if (spc == 6) one_per_cu(std::integral_constant<int, 6>{});
        else one_per_cu(std::integral_constant<int, 5>{});
      }
    } else if (quad) {
      const int64_t units = (a.N + 63) / 64;
      const dim3 grid((unsigned)units), block((unsigned)(64 * decode_waves<FULL, T, 4>(units, cus)));
      hipLaunchKernelGGL((gemm_decode_kernel<FULL, T, 4>), grid, block, 0, stream, a);
    } else {
      const int64_t units = (a.N + 31) / 32;
      const dim3 grid((unsigned)units), block((unsigned)(64 * decode_waves<FULL, T, 2>(units, cus)));
      hipLaunchKernelGGL((gemm_decode_kernel<FULL, T, 2>), grid, block, 0, stream, a);
    }
  };
  using F = std::false_type;
  using Tr = std::true_type;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  using I4 = std::integral_constant<int, 4>;
  switch ((int)tiles * 2 + (a.full ? 1 : 0)) {
    case 2: go(F(), I1()); break;
    case 3: go(Tr(), I1()); break;
    case 4: go(F(), I2()); break;
    case 5: go(Tr(), I2()); break;
    case 6: go(F(), I3()); break;
    case 7: go(Tr(), I3()); break;
    case 8: go(F(), I4()); break;
    default: go(Tr(), I4()); break;
  }
  return hipGetLastError();
}

}  // namespace mxq
