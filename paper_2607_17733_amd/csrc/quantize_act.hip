// quantize_act.hip -- online MXINT quantization of bf16 activation rows.
//
// MXSens (arXiv 2607.17733) Section 2 and Section 4.1: every 32-element
// block of the permuted row gets one shared exponent E = floor(log2 max|x|)
// + 127 and mantissas of its own width m in {4, 6, 8} (or 3, stored as 2q in
// the 4-bit layout).
//
// Work decomposition.  A workgroup owns R consecutive rows (8 for K = 4096,
// fewer for longer rows, up to 64 for short ones) and stages them in LDS with
// 16-byte loads, so the permutation becomes an LDS gather (entries outside
// [0, K) clamp to the zero padding after the row).  The workgroup first turns
// the permutation into a table of 16-bit byte offsets in LDS (rows of at most
// 32767 elements; longer rows read it from global memory per item).  A thread
// owns one (row, block) item, at most two; its segment selects a code path
// compiled for that width.  A workgroup has up to 1024 threads and fills a
// CU.  Lanes run over rows fastest, so the rows of a block write contiguous
// runs of the 32-row operand tiles (whole 128-byte lines at R = 8), and
// consecutive workgroups run on one XCD, whose L2 then completes every line
// of the tile.
//
// Arithmetic.  The block maximum is taken on the integer |bf16| patterns (two
// per register); the mantissas are computed in fp32, where every step is
// exact: x * 2^-s scales an 8-bit significand by a power of two, rint and the
// clamp act on integers below 2^8.  The packed row is assembled from the
// integers' low bytes, four elements per register.  The operand image uses the gfx950 scaled FP6/FP8 conversions (the values
// are exact in the target format, so they never round).
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef unsigned v6u __attribute__((ext_vector_type(6)));
typedef short v2s __attribute__((ext_vector_type(2)));
typedef unsigned short v2us __attribute__((ext_vector_type(2)));
typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef unsigned u2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kMaxThreads = 1024;
constexpr int kLdsBudget = 144 * 1024;  // staged rows of one workgroup per CU
constexpr int kRowPad = 8;              // zero bf16 elements after each staged row
constexpr int64_t kPermTableMaxK = 32767;  // 16-bit byte offsets into a staged row

// A block of 32 values kept as its even and odd elements (the register
// layout the FP6 conversion takes).
struct Blk {
  v16f e, o;
  __device__ float operator[](int t) const { return (t & 1) ? o[t >> 1] : e[t >> 1]; }
};

// 32 values / div as FP6 e3m2 codes, element t at bits 6t of 24 bytes (the
// conversion interleaves its two 16-element inputs).
__device__ inline v6u to_e3m2(const Blk &v, float div) {
  return __builtin_amdgcn_cvt_scalef32_2xpk16_bf6_f32(v.e, v.o, div);
}

// Elements 16h..16h+15 / div as FP8 e4m3 codes, one byte each.
__device__ inline u4 to_e4m3(const Blk &v, int h, float div) {
  u4 r;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const int t = 16 * h + 4 * d;
    v2s z = {0, 0};
    z = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(z, v[t], v[t + 1], div, false);
    z = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(z, v[t + 2], v[t + 3], div, true);
    r[d] = ((uint32_t)(uint16_t)z[1] << 16) | (uint16_t)z[0];
  }
  return r;
}

// Low bytes of the integers of elements t0, t0+step, t0+2step, t0+3step.
__device__ inline uint32_t byte_lanes(const Blk &v, int t0, int step) {
  return ((uint32_t)(int)v[t0] & 255u) | (((uint32_t)(int)v[t0 + step] & 255u) << 8) |
         (((uint32_t)(int)v[t0 + 2 * step] & 255u) << 16) |
         ((uint32_t)(int)v[t0 + 3 * step] << 24);
}

// Two's-complement nibbles of elements t0..t0+7 (element t0+t at bits 4t):
// byte j takes element t0+2j in its low and t0+2j+1 in its high nibble.
__device__ inline uint32_t nibbles8(const Blk &v, int t0) {
  const uint32_t ev = byte_lanes(v, t0, 2), od = byte_lanes(v, t0 + 1, 2);
  return (ev & 0x0F0F0F0Fu) | ((od & 0x0F0F0F0Fu) << 4);
}

// Two's-complement bytes of elements t0..t0+3.
__device__ inline uint32_t bytes4(const Blk &v, int t0) { return byte_lanes(v, t0, 1); }

// Top-bit word d of a 6-bit block (canonical packed layout): byte j holds
// the signed top two bits (bits 4-5) of elements 16d+2j, 16d+2j+1,
// 16d+8+2j, 16d+9+2j in bits 6-7, 4-5, 2-3, 0-1.
__device__ inline uint32_t top_word(const Blk &v, int d) {
  const uint32_t a = byte_lanes(v, 16 * d, 2), b = byte_lanes(v, 16 * d + 1, 2);
  const uint32_t c = byte_lanes(v, 16 * d + 8, 2), e = byte_lanes(v, 16 * d + 9, 2);
  return ((a & 0x30303030u) << 2) | (b & 0x30303030u) | ((c & 0x30303030u) >> 2) |
         ((e & 0x30303030u) >> 4);
}

// The 3-bit two's-complement codes of the 32 elements, element t at bits 3t
// of 96 bits (canonical packed row).
__device__ inline void pack3(const Blk &v, uint32_t *w) {
  w[0] = w[1] = w[2] = 0;
#pragma unroll
  for (int t = 0; t < 32; ++t) {
    const uint32_t c = (uint32_t)(int)v[t] & 7u;
    const int b = 3 * t;
    w[b >> 5] |= c << (b & 31);
    if ((b & 31) > 29) w[(b >> 5) + 1] |= c >> (32 - (b & 31));
  }
}

// Where padded block rem of segment SEG goes: its step, position in the
// step, its block of the width map, and the step's offset in a 16-row tile
// of the operand image and its scale group and byte.  The segment is a
// compile-time constant, so every per-segment quantity is a constant index
// into the width map's geometry.
struct ItemGeo {
  int s, rem, pos, b;
  bool pad;
  int step_off, group, byte;
};
template <int SEG>
__device__ inline ItemGeo item_geo_seg(const LGeo &lg, int rem) {
  ItemGeo g;
  constexpr int two = SEG < 2 ? 2 : 1;               // log2 blocks per step
  const int k = rem >> two;
  g.s = SEG;
  g.rem = rem;
  g.pos = rem & ((1 << two) - 1);
  g.pad = rem >= lg.nb[SEG];
  g.b = lg.b0[SEG] + rem;
  constexpr int sb = kLanes * a_lane_bytes(0);       // 3/4/6-bit step bytes
  int before = 0;
#pragma unroll
  for (int i = 0; i < SEG; ++i) before += lg.S[i];
  g.step_off = before * sb + k * (SEG == 3 ? kLanes * a_lane_bytes(3) : sb);
  g.group = lg.G0[SEG] + (k >> 2);
  g.byte = k & (kGroupSteps - 1);
  return g;
}
// First padded block of each segment (P[0] = 0).
struct SegStarts {
  int P[kSegs];
  __device__ explicit SegStarts(const LGeo &lg) {
    P[0] = 0;
#pragma unroll
    for (int i = 1; i < kSegs; ++i) P[i] = P[i - 1] + lg.S[i - 1] * (i - 1 < 2 ? 4 : 2);
  }
};
__device__ inline ItemGeo item_geo(const LGeo &lg, const SegStarts &ss, int bp) {
  if (bp < ss.P[1]) return item_geo_seg<0>(lg, bp);
  if (bp < ss.P[2]) return item_geo_seg<1>(lg, bp - ss.P[1]);
  if (bp < ss.P[3]) return item_geo_seg<2>(lg, bp - ss.P[2]);
  return item_geo_seg<3>(lg, bp - ss.P[3]);
}

// One (row, padded block) item: gather, quantize, write the canonical
// packed row and exponent (q.write_rows) and / or the GEMM operand image
// and its scale words (q.write_image).  sr is the staged row in LDS,
// followed by zero padding; pt is the permutation as byte offsets into a
// staged row (two 16-bit offsets per dword), or null for the identity.
template <bool RNA, int SEG>
__device__ inline void quantize_item(const QuantArgs &q, const LGeo &lg, const ItemGeo &g,
                                     const uint32_t *pt, int64_t row, const uint8_t *sr) {
  constexpr int s = SEG;
  constexpr int m = s == 0 ? 3 : s == 1 ? 4 : s == 2 ? 6 : 8;
  const int rem = g.rem, pos = g.pos, b = g.b;
  const bool pad = g.pad;

  // gather: pr[i] holds elements 2i (low half) and 2i+1 (high half)
  uint32_t pr[16];
  const int p0 = b * kBlock;
  if (pad) {
#pragma unroll
    for (int i = 0; i < 16; ++i) pr[i] = 0;
  } else if (!q.perm) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const u4 d = *(const u4 *)(sr + 2 * (p0 + 8 * u));
#pragma unroll
      for (int k = 0; k < 4; ++k) pr[4 * u + k] = d[k];
    }
  } else if (pt) {
    // the block's 32 byte offsets (entries outside [0, K) point at the zero
    // after the row)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const u4 o = *(const u4 *)(pt + 16 * b + 4 * u);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        v2us x;
        x.x = *(const uint16_t *)(sr + (o[k] & 0xFFFFu));
        x.y = *(const uint16_t *)(sr + (o[k] >> 16));
        pr[4 * u + k] = __builtin_bit_cast(uint32_t, x);
      }
    }
  } else {
    // rows too long for the table: the entries from global memory, clamped
    // to the zero after the row
    const unsigned K = (unsigned)q.K;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int4 e = *(const int4 *)(q.perm + b * kBlock + 4 * u);
      v2us x, y;
      x.x = *(const uint16_t *)(sr + 2 * min((unsigned)e.x, K));
      x.y = *(const uint16_t *)(sr + 2 * min((unsigned)e.y, K));
      y.x = *(const uint16_t *)(sr + 2 * min((unsigned)e.z, K));
      y.y = *(const uint16_t *)(sr + 2 * min((unsigned)e.w, K));
      pr[2 * u] = __builtin_bit_cast(uint32_t, x);
      pr[2 * u + 1] = __builtin_bit_cast(uint32_t, y);
    }
  }

  // block exponent from the integer maximum of |bits|, two lanes at a time
  v2us mx = {0, 0};
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const uint32_t a = pr[i] & 0x7FFF7FFFu;
    mx = __builtin_elementwise_max(mx, __builtin_bit_cast(v2us, a));
  }
  const uint32_t amax = mx.x > mx.y ? mx.x : mx.y;
  const int E = block_exponent(amax);

  // mantissas as exact integer-valued floats: rint(x * 2^(127 + m - 2 - E)),
  // clamped; a block holding Inf or NaN (E = 255) quantizes to zeros, so
  // its values are replaced by zeros first
  if (E == 255) {
#pragma unroll
    for (int i = 0; i < 16; ++i) pr[i] = 0;
  }
  Blk v;
  {
    constexpr float qmax = (float)((1 << (m - 1)) - 1);
    const float qmin = q.full_clamp ? -(qmax + 1.f) : -qmax;
    const int sh = 127 + m - 2 - E;
#pragma unroll
    for (int u = 0; u < 32; ++u) {
      const uint32_t bits = (u & 1) ? (pr[u >> 1] & 0xFFFF0000u) : (pr[u >> 1] << 16);
      float y = ldexpf(__uint_as_float(bits), sh);
      if (RNA) {
        const float tr = truncf(y);
        y = fabsf(y - tr) >= 0.5f ? tr + copysignf(1.f, y) : tr;
      } else {
        y = rintf(y);
      }
      y = __builtin_amdgcn_fmed3f(y, qmin, qmax);
      if (u & 1) v.o[u >> 1] = y; else v.e[u >> 1] = y;
    }
  }
  const uint32_t Eu = pad ? 0u : (uint32_t)E;

  if (q.write_rows && !pad) {
    q.exp[row * q.out_erb + b] = (uint8_t)E;
    // the block's offset in the packed row: 12, 16, 24 or 32 bytes per block
    const int64_t aoff = s == 0 ? 12LL * b
                       : s == 1 ? 12LL * q.n3 + 16LL * (b - q.n3)
                       : s == 2 ? 12LL * q.n3 + 16LL * (q.n4 - q.n3) + 24LL * (b - q.n4)
                                : 12LL * q.n3 + 16LL * (q.n4 - q.n3) + 24LL * q.n6 +
                                      32LL * (b - q.n4 - q.n6);
    uint8_t *p = q.mant + row * q.out_rb + aoff;
    if (m == 3) {
      uint32_t w[3];
      pack3(v, w);
      *(uint32_t *)p = w[0];
      *(uint32_t *)(p + 4) = w[1];
      *(uint32_t *)(p + 8) = w[2];
    } else if (m == 4) {
      *(u4 *)p = u4{nibbles8(v, 0), nibbles8(v, 8), nibbles8(v, 16), nibbles8(v, 24)};
    } else if (m == 6) {
      *(u2 *)p = u2{nibbles8(v, 0), nibbles8(v, 8)};
      *(u2 *)(p + 8) = u2{nibbles8(v, 16), nibbles8(v, 24)};
      *(u2 *)(p + 16) = u2{top_word(v, 0), top_word(v, 1)};
    } else {
#pragma unroll
      for (int d = 0; d < 4; ++d)
        *(u2 *)(p + 8 * d) = u2{bytes4(v, 8 * d), bytes4(v, 8 * d + 4)};
    }
  }
  if (!q.write_image) return;

  // operand image (16-row tiles) and its scale words
  const int r = (int)(row & (kATileRows - 1));
  uint8_t *stp = q.img + (row >> 4) * q.a_tile + g.step_off;
  uint8_t *scw = q.img_exp + (row >> 4) * q.a_tile_sc + g.group * 256 + g.byte;
  if (s <= 1) {
    // E3M2 codes of q (4-bit) or of 2q (3-bit)
    if (s == 0) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        v.e[i] *= 2.f;
        v.o[i] *= 2.f;
      }
    }
    const int l = 16 * pos + r;
    const v6u c = to_e3m2(v, 1.f);
    *(u2 *)(stp + 24 * l) = u2{c[0], c[1]};
    *(u2 *)(stp + 24 * l + 8) = u2{c[2], c[3]};
    *(u2 *)(stp + 24 * l + 16) = u2{c[4], c[5]};
    scw[4 * l] = (uint8_t)Eu;
  } else {
    // digits q = base h + l: the high digits first, then the low digits in
    // the same registers (h is dead once its codes are formed)
    Blk d;
    constexpr float f = s == 2 ? 0.125f : 0.0625f, base = s == 2 ? 8.f : 16.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      d.e[i] = floorf(v.e[i] * f);
      d.o[i] = floorf(v.o[i] * f);
    }
    if (s == 2) {
      // lane groups 2 pos (high plane h/2) and 2 pos + 1 (low plane l/16)
      const int lh = 16 * (2 * pos) + r, ll = lh + 16;
      const v6u ch = to_e3m2(d, 2.f);
      *(u2 *)(stp + 24 * lh) = u2{ch[0], ch[1]};
      *(u2 *)(stp + 24 * lh + 8) = u2{ch[2], ch[3]};
      *(u2 *)(stp + 24 * lh + 16) = u2{ch[4], ch[5]};
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        d.e[i] = fmaf(d.e[i], -base, v.e[i]);
        d.o[i] = fmaf(d.o[i], -base, v.o[i]);
      }
      const v6u cl = to_e3m2(d, 16.f);
      *(u2 *)(stp + 24 * ll) = u2{cl[0], cl[1]};
      *(u2 *)(stp + 24 * ll + 8) = u2{cl[2], cl[3]};
      *(u2 *)(stp + 24 * ll + 16) = u2{cl[4], cl[5]};
    } else {
      // E4M3 2h and l/8; lane group 2 plane + half holds elements
      // 16 half..16 half + 15 of the plane, at byte 16 pos
#pragma unroll
      for (int e = 0; e < 2; ++e)
        *(u4 *)(stp + 32 * (16 * e + r) + 16 * pos) = to_e4m3(d, e, 0.5f);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        d.e[i] = fmaf(d.e[i], -base, v.e[i]);
        d.o[i] = fmaf(d.o[i], -base, v.o[i]);
      }
#pragma unroll
      for (int e = 0; e < 2; ++e)
        *(u4 *)(stp + 32 * (16 * (2 + e) + r) + 16 * pos) = to_e4m3(d, e, 8.f);
    }
    scw[4 * (16 * (2 * pos) + r)] = (uint8_t)Eu;
    scw[4 * (16 * (2 * pos + 1) + r)] = (uint8_t)Eu;
  }
  // the unused scale bytes of a segment's short last group
  if (rem == 0) {
    const int S = lg.S[s], G0 = lg.G0[s];
    for (int k = S; k < (S + kGroupSteps - 1) / kGroupSteps * kGroupSteps; ++k) {
      uint8_t *z = q.img_exp + (row >> 4) * q.a_tile_sc +
                   (int64_t)(G0 + k / kGroupSteps) * 256 + k % kGroupSteps;
      for (int g = 0; g < 4; ++g) z[4 * (16 * g + r)] = 0;
    }
  }
}

// quantize_item for the item's segment (a branch that is uniform over a
// wave except where its items straddle two segments)
template <bool RNA>
__device__ inline void quantize_item_any(const QuantArgs &q, const LGeo &lg, const ItemGeo &g,
                                         const uint32_t *pt, int64_t row, const uint8_t *sr) {
  if (g.s == 0) quantize_item<RNA, 0>(q, lg, g, pt, row, sr);
  else if (g.s == 1) quantize_item<RNA, 1>(q, lg, g, pt, row, sr);
  else if (g.s == 2) quantize_item<RNA, 2>(q, lg, g, pt, row, sr);
  else quantize_item<RNA, 3>(q, lg, g, pt, row, sr);
}

__device__ inline float bf16f(uint32_t b) { return __uint_as_float(b << 16); }

// float32 -> bf16 bits, round to nearest even (gfx950 converts a pair per
// instruction; a NaN stays a NaN)
__device__ inline uint32_t to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// e^t in float32, evaluated the same way on every machine: the Cody-Waite
// reduction t = k ln2 + r (ln2 split in two so that k * LN2_HI is exact)
// and the Taylor polynomial of e^r to degree 7 (|r| <= ln2 / 2), every
// operation rounded on its own (no fused multiply-add); then 2^k exactly.
__device__ inline float exp32(float t) {
#pragma clang fp contract(off)
  constexpr float kInvLn2 = __builtin_bit_cast(float, 0x3FB8AA3Bu);
  constexpr float kLn2Hi = __builtin_bit_cast(float, 0x3F317200u);
  constexpr float kLn2Lo = __builtin_bit_cast(float, 0x35BFBE8Eu);
  t = fminf(fmaxf(t, -120.f), 120.f);
  const float k = rintf(t * kInvLn2);
  const float r = (t - k * kLn2Hi) - k * kLn2Lo;
  float p = __builtin_bit_cast(float, 0x39500D01u);                  // 1/7!
  p = p * r + __builtin_bit_cast(float, 0x3AB60B61u);                // 1/6!
  p = p * r + __builtin_bit_cast(float, 0x3C088889u);                // 1/5!
  p = p * r + __builtin_bit_cast(float, 0x3D2AAAABu);                // 1/4!
  p = p * r + __builtin_bit_cast(float, 0x3E2AAAABu);                // 1/3!
  p = p * r + 0.5f;
  p = p * r + 1.f;
  p = p * r + 1.f;
  return ldexpf(p, (int)k);
}

// bf16 bits of bf16(silu(g)) * u (float32 product, nearest-even), with
// silu(g) = g / (1 + e^-g) (the producer of the down projection's input)
__device__ inline uint32_t swiglu1(uint32_t g, uint32_t u) {
#pragma clang fp contract(off)
  const float gf = bf16f(g);
  const float s = gf != gf ? __builtin_nanf("") : gf / (1.f + exp32(-gf));
  return to_bf16(bf16f(to_bf16(s)) * bf16f(u));
}

__device__ inline u4 swiglu8(u4 g, u4 u) {
  u4 o;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    o[j] = swiglu1(g[j] & 0xFFFFu, u[j] & 0xFFFFu) | (swiglu1(g[j] >> 16, u[j] >> 16) << 16);
  return o;
}

// RMS normalisation of the R staged rows, in place (the fused producer of
// the quantizer; Appendix A.2 keeps normalisation in 16-bit floating
// point): per row, ms = sum of x^2 / K in float64 (each 32-element block
// in order, then the blocks in order), r = float32(1 / sqrt(ms + eps)),
// then y = bf16(g * bf16(x * r)) with float32 products.
__device__ void rms_normalise(const QuantArgs &q, uint8_t *smem, int R, int rowB, int t,
                              int nthr, int64_t r0) {
  const int K = (int)q.K, nbk = K / kBlock;
  double *part = (double *)(smem + R * rowB);
  float *rr = (float *)(part + R * nbk);
  for (int it = t; it < R * nbk; it += nthr) {
    const int lr = it / nbk, b = it - lr * nbk;
    const u4 *xr = (const u4 *)(smem + lr * rowB + 64 * b);
    double sum = 0.0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const u4 d = xr[u];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const double lo = (double)bf16f(d[j] & 0xFFFFu), hi = (double)bf16f(d[j] >> 16);
        sum += lo * lo;
        sum += hi * hi;
      }
    }
    part[it] = sum;
  }
  __syncthreads();
  if (t < R) {
    // the block sums in order; loaded sixteen at a time so that only the
    // additions form the dependent chain
    const double *pp = part + t * nbk;
    double acc = 0.0;
    int b = 0;
    for (; b + 16 <= nbk; b += 16) {
      double v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = pp[b + u];
#pragma unroll
      for (int u = 0; u < 16; ++u) acc += v[u];
    }
    for (; b < nbk; ++b) acc += pp[b];
    // the zero rows past the input (operand-image padding) stay zero, also
    // with eps = 0
    rr[t] = r0 + t < q.src_rows ? (float)(1.0 / sqrt(acc / (double)K + (double)q.eps)) : 0.f;
  }
  __syncthreads();
  const int cpr = K / 8;                                 // 8-element chunks per row
  for (int c = t; c < R * cpr; c += nthr) {
    const int lr = c / cpr, k0 = (c - lr * cpr) * 8;
    u4 *xp = (u4 *)(smem + lr * rowB + 2 * k0);
    const u4 d = *xp;
    const u4 gv = *(const u4 *)(q.gain + k0);
    const float r = rr[lr];
    u4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t h0 = to_bf16(bf16f(d[j] & 0xFFFFu) * r), h1 = to_bf16(bf16f(d[j] >> 16) * r);
      const uint32_t y0 = to_bf16(bf16f(gv[j] & 0xFFFFu) * bf16f(h0));
      const uint32_t y1 = to_bf16(bf16f(gv[j] >> 16) * bf16f(h1));
      o[j] = y0 | (y1 << 16);
    }
    *xp = o;
  }
  __syncthreads();
}

template <bool RNA>
__global__ __launch_bounds__(kMaxThreads) void quantize_act_kernel(QuantArgs q) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int t = threadIdx.x;
  const int nthr = blockDim.x;
  const int K = (int)q.K;
  const int rowB = 2 * (K + kRowPad);                // staged row stride (bytes)
  const int lgR = q.lg_rows;
  const int R = 1 << lgR;
  const LGeo lg(q.n3, q.n4, q.n6, q.n8);
  int nbp = 0;                                       // padded blocks per row
  for (int s = 0; s < kSegs; ++s) nbp += lg.S[s] * (s < 2 ? 4 : 2);
  // XCD-aware order: consecutive row groups (whole 32-row operand tiles)
  // stay on one XCD, so its L2 completes every line of the tile.
  int64_t w = blockIdx.x;
  const int64_t nwg = gridDim.x;
  if ((nwg & 7) == 0) w = (w & 7) * (nwg >> 3) + (w >> 3);
  const int64_t r0 = w << lgR;

  const int nit = nbp << lgR;
  const SegStarts ss(lg);

  // The permutation as byte offsets into a staged row, two per dword, in LDS
  // after the rows (and the normalisation's sums); an entry outside [0, K)
  // becomes the offset of the zero after the row.  A thread's first
  // kPermPre groups of four entries are loaded before the rows, so their
  // latency overlaps the rows' loads.
  constexpr int kPermPre = 4;
  uint32_t *pt = nullptr;
  int4 pp[kPermPre];
  auto put_perm = [&](int c, const int4 &e) {
    const unsigned k = (unsigned)K;
    const uint32_t o0 = 2u * min((unsigned)e.x, k), o1 = 2u * min((unsigned)e.y, k);
    const uint32_t o2 = 2u * min((unsigned)e.z, k), o3 = 2u * min((unsigned)e.w, k);
    *(u2 *)(pt + 2 * c) = u2{o0 | (o1 << 16), o2 | (o3 << 16)};
  };
  if (q.perm_table) {
    const int rms = q.rmsnorm ? R * (8 * (K / kBlock) + 4) : 0;
    pt = (uint32_t *)(smem + ((R * rowB + rms + 15) & ~15));
#pragma unroll
    for (int j = 0; j < kPermPre; ++j) {
      const int c = t + j * nthr;
      if (c < K / 4) pp[j] = *(const int4 *)(q.perm + 4 * c);
    }
  }

  // Stage the rows.  Each thread issues a batch of loads before it stores
  // any of them, so the batch costs one memory latency instead of one per
  // load.
  constexpr int kBatch = 8;
  if (q.vec16 && !q.swiglu && K % 512 == 0) {
    // Rows of whole 1 KB pieces go straight into LDS (direct-to-LDS loads,
    // one piece per wave instruction), so no thread waits for its data
    // before the permutation table is written.  Rows past the source's end
    // read zeros: the buffer resource ends at its last row.
    const int64_t live = q.src_rows > r0 ? q.src_rows - r0 : 0;
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(q.src + r0 * q.ld), 0, (int)min(live * q.ld * 2, (int64_t)0x7fffffff), 0x00020000);
    const int per_row = K / 512;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6), nwaves = nthr >> 6;
    for (int pc = wave; pc < R * per_row; pc += nwaves) {
      const int lr = pc / per_row, j = pc - lr * per_row;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void *)(smem + lr * rowB + j * 1024), 16,
                                               (t & 63) * 16, (int)(lr * q.ld * 2) + j * 1024, 0, 0);
    }
  } else if (q.vec16) {
    // vector v = lr * vpr + c, advanced by nthr without dividing per load
    const int vpr = K / 8, nv = R * vpr;
    const int dq = nthr / vpr, dr = nthr - dq * vpr;
    int lr0 = t / vpr, c0 = t - lr0 * vpr;
    const bool swiglu = q.swiglu != 0;
    for (int v0 = t; v0 < nv; v0 += nthr * kBatch) {
      u4 d[kBatch];
      int lrk[kBatch], ck[kBatch];
      int lr = lr0, c = c0;
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        lrk[k] = lr;
        ck[k] = c;
        if (v0 + k * nthr < nv) {
          if (r0 + lr < q.src_rows) {
            d[k] = *(const u4 *)(q.src + (r0 + lr) * q.ld + 8 * c);
            if (swiglu) d[k] = swiglu8(d[k], *(const u4 *)(q.src2 + (r0 + lr) * q.ld + 8 * c));
          } else {
            d[k] = u4{0u, 0u, 0u, 0u};
          }
        }
        c += dr;
        lr += dq;
        if (c >= vpr) {
          c -= vpr;
          ++lr;
        }
      }
      lr0 = lr;
      c0 = c;
#pragma unroll
      for (int k = 0; k < kBatch; ++k)
        if (v0 + k * nthr < nv) *(u4 *)(smem + lrk[k] * rowB + 16 * ck[k]) = d[k];
    }
  } else {
    for (int lr = 0; lr < R; ++lr) {
      const bool live = r0 + lr < q.src_rows;
      const uint16_t *src = q.src + (r0 + lr) * q.ld;
      for (int c = t; c < K; c += nthr) {
        uint32_t v = live ? src[c] : 0u;
        if (live && q.swiglu) v = swiglu1(v, q.src2[(r0 + lr) * q.ld + c]);
        *(uint16_t *)(smem + lr * rowB + 2 * c) = (uint16_t)v;
      }
    }
  }
  if (pt) {
#pragma unroll
    for (int j = 0; j < kPermPre; ++j) {
      const int c = t + j * nthr;
      if (c < K / 4) put_perm(c, pp[j]);
    }
    for (int c = t + kPermPre * nthr; c < K / 4; c += nthr)
      put_perm(c, *(const int4 *)(q.perm + 4 * c));
  }
  if (t < R) *(u4 *)(smem + t * rowB + 2 * K) = u4{0u, 0u, 0u, 0u};
  // the direct-to-LDS loads are complete before the workgroup meets
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (q.rmsnorm) rms_normalise(q, smem, R, rowB, t, nthr, r0);

  for (int it = t; it < nit; it += nthr) {
    const int lr = it & (R - 1);
    const int64_t row = r0 + lr;
    if (row < q.out_rows)
      quantize_item_any<RNA>(q, lg, item_geo(lg, ss, it >> lgR), pt, row, smem + lr * rowB);
  }
  // zero the padding of the packed and exponent rows
  if (q.write_rows && t < R) {
    const int64_t row = r0 + t;
    if (row < q.src_rows) {
      for (int64_t z = q.row_used; z < q.canon_rb; ++z) q.mant[row * q.out_rb + z] = 0;
      for (int64_t z = q.n4 + q.n6 + q.n8; z < q.canon_erb; ++z)
        q.exp[row * q.out_erb + z] = 0;
    }
  }
}

}  // namespace

int quantize_act_padded_blocks(int n3, int n4, int n6, int n8) {
  const LGeo lg(n3, n4, n6, n8);
  int nbp = 0;
  for (int s = 0; s < kSegs; ++s) nbp += lg.S[s] * (s < 2 ? 4 : 2);
  return nbp;
}

// Bytes per staged row: the row and its zero padding, plus with RMS
// normalisation its block sums and its 1/rms.
static int64_t row_lds(int64_t K, bool rmsnorm) {
  return 2 * (K + kRowPad) + (rmsnorm ? 8 * (K / kBlock) + 4 : 0);
}

// The permutation's byte-offset table (16-bit offsets, so rows of at most
// 32767 elements), with 16 bytes of alignment slack.
static int64_t perm_table_lds(int64_t K) { return 2 * K + 16; }

// Rows per workgroup: the largest power of two (at most 64) whose staged
// rows fit the LDS budget with at most two items per thread, halved while
// the rows and the permutation table exceed the LDS.  More rows per
// workgroup make longer contiguous runs in the operand tiles.
int quantize_act_rows(int64_t K, int nbp, bool perm, bool rmsnorm) {
  const int64_t per = row_lds(K, rmsnorm);
  int r = 1;
  while (r < 64 && 2 * r * per <= kLdsBudget && (int64_t)nbp * 2 * r <= 2 * kMaxThreads)
    r *= 2;
  if (perm && K <= kPermTableMaxK)
    while (r > 1 && r * per + perm_table_lds(K) > kMaxLds) r >>= 1;
  return r;
}

// Whether the permutation is gathered through the LDS table.
static bool quantize_act_table(int64_t K, int nbp, bool perm, bool rmsnorm) {
  return perm && K <= kPermTableMaxK &&
         quantize_act_rows(K, nbp, perm, rmsnorm) * row_lds(K, rmsnorm) + perm_table_lds(K) <=
             kMaxLds;
}

int64_t quantize_act_lds(int64_t K, int nbp, bool perm, bool rmsnorm) {
  return (int64_t)quantize_act_rows(K, nbp, perm, rmsnorm) * row_lds(K, rmsnorm) +
         (quantize_act_table(K, nbp, perm, rmsnorm) ? perm_table_lds(K) : 0);
}

hipError_t launch_quantize_act(const QuantArgs &args, hipStream_t stream) {
  QuantArgs a = args;
  const bool perm = a.perm != nullptr;
  const int nbp = quantize_act_padded_blocks(a.n3, a.n4, a.n6, a.n8);
  const int R = quantize_act_rows(a.K, nbp, perm, a.rmsnorm != 0);
  int lg = 0;
  while ((1 << lg) < R) ++lg;
  a.lg_rows = lg;
  a.rows_per_wg = R;
  a.stage = 0;
  a.perm_table = quantize_act_table(a.K, nbp, perm, a.rmsnorm != 0) ? 1 : 0;
  const int64_t grid = (a.out_rows + R - 1) / R;
  if (grid <= 0) return hipSuccess;
  const int64_t lds = quantize_act_lds(a.K, nbp, perm, a.rmsnorm != 0);
  if (lds > kMaxLds) return hipErrorInvalidValue;
  const int64_t items = (int64_t)nbp * R;
  const int threads = (int)(items >= kMaxThreads ? kMaxThreads : (items + 63) / 64 * 64);
  const void *fn = a.ties_away ? (const void *)quantize_act_kernel<true>
                               : (const void *)quantize_act_kernel<false>;
  (void)hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  if (a.ties_away)
    hipLaunchKernelGGL(quantize_act_kernel<true>, dim3((unsigned)grid), dim3(threads),
                       (size_t)lds, stream, a);
  else
    hipLaunchKernelGGL(quantize_act_kernel<false>, dim3((unsigned)grid), dim3(threads),
                       (size_t)lds, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
