// mxq_device.h -- device-side building blocks shared by the libmxq kernels:
// the integer MXINT quantizer (one bf16 element given its block exponent),
// packed-layout addressing, and the unpack of packed mantissas into int8
// matrix-core operands.
//
// Format (MXSens, arXiv 2607.17733, Sections 2, 4.1, 5.1): 32-element blocks
// along K, one 8-bit shared exponent E = floor(log2 max|x|) + 127 per block,
// signed mantissas of m in {4, 6, 8} bits with LSB weight 2^(E-127-(m-2)).
// (3-bit blocks are quantized with m = 3 and stored as 4-bit blocks holding 2q.)
//
// Everything is integer arithmetic on the bf16 bit pattern: no log2, no
// float scaling (2^-s overflows fp32 for small s, and bf16 subnormals would
// be flushed by float paths).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mxq {

constexpr int kBlock = 32;

// ---------------------------------------------------------------------------
// Operand layouts of the GEMMs (include/mxq.h has the byte-exact statement).
//
// Both GEMMs run V_MFMA_SCALE_F32_16X16X128_F8F6F4: 16 rows x 16 columns x
// 128 K, lane l = 16 g + r (lane group g, row / column r) holding 32 K-values
// and supplying the E8M0 scale of K-block g of its row / column.  For FP6
// the 32 values of lane group g are K 32g..32g+31; for FP8 they are K
// 16g..16g+15 (bytes 0-15) and 64+16g..64+16g+15 (bytes 16-31).
//
// The K-blocks of a width map form four segments, 3-bit, 4-bit, 6-bit and
// 8-bit blocks in that order.  A segment is walked in steps: four blocks per
// step for 3- and 4-bit blocks (K-block g = block 4s+g), two per step for 6-
// and 8-bit blocks, each split into two digit planes (K-blocks 2j and 2j+1
// hold the high and low plane of block 2s+j).  Segments are zero padded to
// whole steps; the steps of a segment form groups of four that share one
// scale word per lane (byte k = step k of the group).
//
// Digits, with each block's E as its E8M0 scale (the extra +3 / +4 of the
// weights' high planes applied by the GEMM, saturating at 255):
//   3-bit  A: E3M2 code of 2q          W: E2M3 code s|k of q/8  (k = |q|)
//   4-bit  A: E3M2 code of q           W: E3M2 code s|k of q/16
//   6-bit  A: E3M2 h/2, l/16 (q = 8h+l, h = floor(q/8))
//          W: E3M2 s|h and s|l of +-h/16 (scale +3) and +-l/16 (|q| = 8h+l)
//   8-bit  A: E4M3 2h, l/8 (q = 16h+l, h = floor(q/16))
//          W: E4M3 of +-h/512 (scale +4) and +-l/512: sign-magnitude bytes
//             (|q| = 16h+l) under the symmetric clamp, two's complement (h
//             signed, l = q mod 16) under the full clamp
// Every digit product is exact and the four products of a 6- or 8-bit block
// pair sum to qa qw 2^(sa+sw) with the scales shown.
//
// The weights' FP6 codes s|k have two zero bits per 6-bit field (one for a
// 3-bit block: s000kk has three), so they are stored "folded" at 4 (3) bits
// per element: the zero bits of one operand word hold the payload of
// another, and the kernel restores the FP6 operand with masks and shifts.
// ---------------------------------------------------------------------------
constexpr int kSegs = 4;
constexpr int kGroupSteps = 4;
constexpr int kLanes = 64;
constexpr int kWCols = 128;          // columns of a weight super-slab
constexpr int kWSlabs = 8;           // 16-column slabs per super-slab
constexpr int kATileRows = 16;

struct LGeo {
  int nb[kSegs];     // blocks of each segment
  int b0[kSegs];     // first block of the segment in the width map
  int S[kSegs];      // steps of each segment
  int st0[kSegs];    // first step of the segment
  int G0[kSegs];     // first scale group of the segment
  int nsteps, ngroups;
  __host__ __device__ LGeo(int n3, int n4, int n6, int n8) {
    nb[0] = n3; nb[1] = n4 - n3; nb[2] = n6; nb[3] = n8;
    int b = 0, st = 0, gg = 0;
    for (int s = 0; s < kSegs; ++s) {
      b0[s] = b;
      st0[s] = st;
      G0[s] = gg;
      S[s] = s < 2 ? (nb[s] + 3) / 4 : (nb[s] + 1) / 2;
      b += nb[s];
      st += S[s];
      gg += (S[s] + kGroupSteps - 1) / kGroupSteps;
    }
    nsteps = st;
    ngroups = gg;
  }
  __host__ __device__ int seg_of_step(int st) const {
    return st < st0[1] ? 0 : st < st0[2] ? 1 : st < st0[3] ? 2 : 3;
  }
  // scale group and byte of global step st
  __host__ __device__ int group_of(int st) const {
    const int s = seg_of_step(st);
    return G0[s] + (st - st0[s]) / kGroupSteps;
  }
  __host__ __device__ int byte_of(int st) const {
    const int s = seg_of_step(st);
    return (st - st0[s]) % kGroupSteps;
  }
};

// Activation operand image: 16-row tiles, each the steps in order, each step
// 64 lanes of alb bytes (lane l at l * alb).  Scales: per tile, per group, a
// dword per lane.
__host__ __device__ constexpr int a_lane_bytes(int seg) { return seg == 3 ? 32 : 24; }
__host__ __device__ inline int64_t a_step_off(const LGeo &g, int st) {
  const int s = g.seg_of_step(st);
  int64_t o = 0;
  for (int k = 0; k < s; ++k) o += (int64_t)g.S[k] * kLanes * a_lane_bytes(k);
  return o + (int64_t)(st - g.st0[s]) * kLanes * a_lane_bytes(s);
}
__host__ __device__ inline int64_t a_tile_bytes(const LGeo &g) {
  int64_t o = 0;
  for (int k = 0; k < kSegs; ++k) o += (int64_t)g.S[k] * kLanes * a_lane_bytes(k);
  return o;
}
__host__ __device__ inline int64_t a_tile_scale_bytes(const LGeo &g) {
  return (int64_t)g.ngroups * kLanes * 4;
}

// Weight super-slabs: 128 columns, each the steps in order, each step the
// chunks of its 8 slabs (chunk n at n * w_chunk_bytes).  Scales: per
// super-slab, per group, 2 KB: lane l's 32 bytes at 32 l, the byte of slab n
// for step k of the group at 8 k + n.
//   3-bit  symmetric: 64 lanes x 8 bytes (words X, Y) then 64 x 4 (word Z);
//          full: as a 4-bit chunk (|q| <= 4 fits s|kkk)
//   4-bit  symmetric: lane l's 16 folded bytes at 16 l; full: 64 x 16 then
//          64 x 8 bytes of the raw 24-byte FP6 operand
//   6-bit  per (block j, column c) of the step: the low plane (16 folded
//          bytes at 16 (16 j + c)), then the high plane (symmetric: 8 bytes
//          of 2-bit magnitudes at 512 + 8 (16 j + c), the sign taken from
//          the low plane; full: 16 folded bytes at 512 + 16 (16 j + c))
//   8-bit  per (block j, column c): 32 mantissa bytes at 32 (16 j + c)
__host__ __device__ constexpr int w_chunk_bytes(int seg, bool full) {
  return seg == 0 ? (full ? 1024 : 768)
       : seg == 1 ? (full ? 1536 : 1024)
       : seg == 2 ? (full ? 1024 : 768)
       : 1024;
}
__host__ __device__ inline int64_t w_step_off(const LGeo &g, int st, bool full) {
  const int s = g.seg_of_step(st);
  int64_t o = 0;
  for (int k = 0; k < s; ++k) o += (int64_t)g.S[k] * kWSlabs * w_chunk_bytes(k, full);
  return o + (int64_t)(st - g.st0[s]) * kWSlabs * w_chunk_bytes(s, full);
}
__host__ __device__ inline int64_t w_super_bytes(const LGeo &g, bool full) {
  int64_t o = 0;
  for (int k = 0; k < kSegs; ++k) o += (int64_t)g.S[k] * kWSlabs * w_chunk_bytes(k, full);
  return o;
}
__host__ __device__ inline int64_t w_super_scale_bytes(const LGeo &g) {
  return (int64_t)g.ngroups * kLanes * kWSlabs * 4;
}

// Segment offsets with a compile-time segment (device code indexes the
// geometry's arrays only with constants, so nothing spills to scratch).
template <int SEG>
__host__ __device__ inline int64_t a_seg_base(const LGeo &g) {
  int64_t o = 0;
#pragma unroll
  for (int k = 0; k < SEG; ++k) o += (int64_t)g.S[k] * kLanes * a_lane_bytes(k);
  return o;
}
template <int SEG, bool FULL>
__host__ __device__ inline int64_t w_seg_base(const LGeo &g) {
  int64_t o = 0;
#pragma unroll
  for (int k = 0; k < SEG; ++k) o += (int64_t)g.S[k] * kWSlabs * w_chunk_bytes(k, FULL);
  return o;
}

// Fold masks: payload bits of the FP6 operand words (element t at bits 6t of
// six words D0..D5; words 3-5 repeat the pattern of 0-2).
//   4-bit s00kkk: X = D0 | (D1 & Z0), Y = D2 | (D1 & Z2) per 16 elements
//   3-bit s000kk: X = D0 | D1 >> 1, Y = D3 | D4 >> 1,
//                 Z = D2 | D5 << 3 | D5 >> 31 per 32 elements
//   2-bit 0000hh: X = D0 | D1 | D2 per 16 elements (the sign is restored from
//                 the low plane's word at the same position)
constexpr uint32_t kF4P0 = 0xe79e79e7u, kF4Z0 = 0x18618618u;
constexpr uint32_t kF4P2 = 0x9e79e79eu, kF4Z2 = 0x61861861u;
constexpr uint32_t kF3A = 0xe38e38e3u, kF3B = 0x38e38e38u, kF3C = 0x8e38e38eu,
                   kF3C31 = 0x0e38e38eu;
constexpr uint32_t kF2Q0 = 0xc30c30c3u, kF2Q1 = 0x30c30c30u, kF2Q2 = 0x0c30c30cu;
constexpr uint32_t kSgn0 = 0x20820820u, kSgn1 = 0x08208208u, kSgn2 = 0x82082082u;

__host__ __device__ inline void fold4(const uint32_t *d, uint32_t *o) {
  o[0] = d[0] | (d[1] & kF4Z0);
  o[1] = d[2] | (d[1] & kF4Z2);
  o[2] = d[3] | (d[4] & kF4Z0);
  o[3] = d[5] | (d[4] & kF4Z2);
}
__host__ __device__ inline void unfold4(const uint32_t *x, uint32_t *d) {
  d[0] = x[0] & kF4P0;
  d[1] = (x[0] & kF4Z0) | (x[1] & kF4Z2);
  d[2] = x[1] & kF4P2;
  d[3] = x[2] & kF4P0;
  d[4] = (x[2] & kF4Z0) | (x[3] & kF4Z2);
  d[5] = x[3] & kF4P2;
}
__host__ __device__ inline void fold3(const uint32_t *d, uint32_t *o) {
  o[0] = d[0] | (d[1] >> 1);
  o[1] = d[3] | (d[4] >> 1);
  o[2] = d[2] | (d[5] << 3) | (d[5] >> 31);
}
__host__ __device__ inline void unfold3(const uint32_t *x, uint32_t *d) {
  d[0] = x[0] & kF3A;
  d[1] = (x[0] << 1) & kF3B;
  d[2] = x[2] & kF3C;
  d[3] = x[1] & kF3A;
  d[4] = (x[1] << 1) & kF3B;
  d[5] = ((x[2] >> 3) & kF3C31) | (x[2] << 31);
}
__host__ __device__ inline void fold2(const uint32_t *d, uint32_t *o) {
  o[0] = d[0] | d[1] | d[2];
  o[1] = d[3] | d[4] | d[5];
}
// high plane from its 2-bit magnitudes and the low plane's signs
__host__ __device__ inline void unfold2(const uint32_t *x, const uint32_t *lo, uint32_t *d) {
  d[0] = (x[0] & kF2Q0) | (lo[0] & kSgn0);
  d[1] = (x[0] & kF2Q1) | (lo[1] & kSgn1);
  d[2] = (x[0] & kF2Q2) | (lo[2] & kSgn2);
  d[3] = (x[1] & kF2Q0) | (lo[3] & kSgn0);
  d[4] = (x[1] & kF2Q1) | (lo[4] & kSgn1);
  d[5] = (x[1] & kF2Q2) | (lo[5] & kSgn2);
}

// 32 six-bit codes -> the six operand words (element t at bits 6t).
__host__ __device__ inline void fp6_words(const uint32_t *c, uint32_t *d) {
  for (int j = 0; j < 6; ++j) d[j] = 0;
  for (int t = 0; t < 32; ++t) {
    const int b = 6 * t, w = b >> 5, sh = b & 31;
    d[w] |= (c[t] & 63u) << sh;
    if (sh > 26) d[w + 1] |= (c[t] & 63u) >> (32 - sh);
  }
}
// and back
__host__ __device__ inline uint32_t fp6_code(const uint32_t *d, int t) {
  const int b = 6 * t, w = b >> 5, sh = b & 31;
  uint32_t v = d[w] >> sh;
  if (sh > 26) v |= d[w + 1] << (32 - sh);
  return v & 63u;
}

// Weight codes of one mantissa q of a block of width m (see above): the
// FP6 code s|k of a 3/4-bit q; the high and low plane codes of a 6-bit q
// (|q| = 8h + l); the byte of an 8-bit q.
__host__ __device__ inline uint32_t w_code34(int q) {
  return (q < 0 ? 32u : 0u) | (uint32_t)(q < 0 ? -q : q);
}
__host__ __device__ inline void w_code6(int q, uint32_t &hi, uint32_t &lo) {
  const uint32_t a = (uint32_t)(q < 0 ? -q : q), s = q < 0 ? 32u : 0u;
  hi = s | (a >> 3);
  lo = s | (a & 7u);
}
__host__ __device__ inline uint32_t w_code8(int q, bool full) {
  if (full) return (uint32_t)q & 255u;
  return (q < 0 ? 128u : 0u) | (uint32_t)(q < 0 ? -q : q);
}

// ---------------------------------------------------------------------------
// Quantizer core.  Block exponent from the integer maximum of |bits|:
// E = exponent field of the largest magnitude (0 for zero/subnormal blocks,
// which is e clamped to -127), 255 for a block holding Inf or NaN.
// ---------------------------------------------------------------------------
__device__ inline int block_exponent(uint32_t amax_bits) {
  return amax_bits >= 0x7F80u ? 255 : (int)(amax_bits >> 7);
}

// Mantissa of one element: round(x / 2^(e - (m-2))) then clamp, computed as
// a rounding right shift of the 8-bit significand by
// E - max(f, 1) + 9 - m bits (never negative for a valid block exponent).
__device__ inline int quant_elem(uint32_t bits, int E, int m, int ties_away,
                                 int full_clamp) {
  if (E == 255) return 0;
  const uint32_t f = (bits >> 7) & 0xFFu;
  const uint32_t sig = (bits & 0x7Fu) | (f ? 0x80u : 0u);
  int sh = E - (f ? (int)f : 1) + 9 - m;
  sh = sh > 10 ? 10 : sh;                 // >= 10: the result rounds to 0
  uint32_t q = sig;
  if (sh > 0) {
    const uint32_t fl = sig >> sh;
    const uint32_t rem = sig & ((1u << sh) - 1u);
    const uint32_t half = 1u << (sh - 1);
    const bool up = ties_away ? (rem >= half)
                              : (rem > half || (rem == half && (fl & 1u)));
    q = fl + (up ? 1u : 0u);
  }
  const int qmax = (1 << (m - 1)) - 1;
  int qi = (int)q;
  if (bits & 0x8000u) {
    const int lim = full_clamp ? qmax + 1 : qmax;
    qi = -(qi < lim ? qi : lim);
  } else {
    qi = qi < qmax ? qi : qmax;
  }
  return qi;
}

// ---------------------------------------------------------------------------
// Element accessors (debug / parity kernels).
// ---------------------------------------------------------------------------
__device__ inline int sext_bits(uint32_t v, int bits) {
  const int sh = 32 - bits;
  return ((int)(v << sh)) >> sh;
}

// Widths and canonical packed-row offsets of the blocks: the row holds the
// blocks in order, block b taking 4 m_b bytes (12 for a 3-bit block).
struct Segs {
  int n4, n6, n8;
  int n3;       // of the n4 blocks, the first n3 hold 3-bit mantissas
};
struct BlockInfo {
  int m;        // mantissa width
  int64_t aoff; // byte offset of the block inside a packed activation row
};
__host__ __device__ inline BlockInfo block_info(const Segs &s, int b) {
  BlockInfo r;
  if (b < s.n3) {
    r.m = 3; r.aoff = 12LL * b;
  } else if (b < s.n4) {
    r.m = 4; r.aoff = 12LL * s.n3 + 16LL * (b - s.n3);
  } else if (b < s.n4 + s.n6) {
    r.m = 6; r.aoff = 12LL * s.n3 + 16LL * (s.n4 - s.n3) + 24LL * (b - s.n4);
  } else {
    r.m = 8; r.aoff = 12LL * s.n3 + 16LL * (s.n4 - s.n3) + 24LL * s.n6 + 32LL * (b - s.n4 - s.n6);
  }
  return r;
}
__host__ __device__ inline int64_t packed_row_used(const Segs &s) {
  return 12LL * s.n3 + 16LL * (s.n4 - s.n3) + 24LL * s.n6 + 32LL * s.n8;
}

// Canonical packed activation row (layout in include/mxq.h).
__device__ inline int act_elem(const uint8_t *row, const BlockInfo &bi, int t) {
  const uint8_t *p = row + bi.aoff;
  if (bi.m == 8) return (int)(int8_t)p[t];
  if (bi.m == 3) {
    const int bit = 3 * t;
    const uint32_t v = (uint32_t)p[bit >> 3] | ((uint32_t)p[(bit >> 3) + 1 < 12 ? (bit >> 3) + 1 : 11] << 8);
    return sext_bits((v >> (bit & 7)) & 7u, 3);
  }
  const uint32_t nib = (p[t >> 1] >> (4 * (t & 1))) & 15u;
  if (bi.m == 4) return sext_bits(nib, 4);
  const int d = t >> 4, u = t & 15;
  const int j = (u & 7) >> 1;
  const int sh = (u < 8 ? 6 : 2) - 2 * (u & 1);
  const uint32_t top = (p[16 + 4 * d + j] >> sh) & 3u;
  return sext_bits(nib | (top << 4), 6);
}

// The block (block index b of the width map, segment seg, step st, position
// within the step) a weight element belongs to.
struct WLoc {
  int seg, st, pos;   // pos: lane group (3/4-bit) or block of the pair (6/8-bit)
};
__host__ __device__ inline WLoc w_loc(const LGeo &g, int b) {
  WLoc r;
  int s = 3;
  while (s > 0 && b < g.b0[s]) --s;
  const int i = b - g.b0[s];
  r.seg = s;
  r.st = g.st0[s] + (s < 2 ? i / 4 : i / 2);
  r.pos = s < 2 ? i % 4 : i % 2;
  return r;
}

// Mantissa t of block b of weight column `col` (any column of the padded
// super-slabs), read back from the weight layout.
__device__ inline int w_elem(const uint8_t *w_mant, const LGeo &g, bool full, int64_t col,
                             int b, int t) {
  const WLoc L = w_loc(g, b);
  const int n = (int)((col % kWCols) >> 4), c = (int)(col & 15);
  const uint8_t *chunk = w_mant + (col / kWCols) * w_super_bytes(g, full) +
                         w_step_off(g, L.st, full) + (int64_t)n * w_chunk_bytes(L.seg, full);
  uint32_t d[6], x[4];
  if (L.seg <= 1) {
    const int l = 16 * L.pos + c;
    if (L.seg == 0 && !full) {
      x[0] = *(const uint32_t *)(chunk + 8 * l);
      x[1] = *(const uint32_t *)(chunk + 8 * l + 4);
      x[2] = *(const uint32_t *)(chunk + 512 + 4 * l);
      unfold3(x, d);
    } else if (L.seg == 1 && full) {
      for (int k = 0; k < 4; ++k) d[k] = *(const uint32_t *)(chunk + 16 * l + 4 * k);
      for (int k = 0; k < 2; ++k) d[4 + k] = *(const uint32_t *)(chunk + 1024 + 8 * l + 4 * k);
    } else {
      for (int k = 0; k < 4; ++k) x[k] = *(const uint32_t *)(chunk + 16 * l + 4 * k);
      unfold4(x, d);
    }
    const uint32_t code = fp6_code(d, t);
    const int mag = (int)(code & 31u);
    return (code & 32u) ? -mag : mag;
  }
  const int jc = 16 * L.pos + c;
  if (L.seg == 3) {
    const uint32_t v = chunk[32 * jc + t];
    if (full) return (int)(int8_t)v;
    return (v & 128u) ? -(int)(v & 127u) : (int)(v & 127u);
  }
  uint32_t lo[6], hi[6];
  for (int k = 0; k < 4; ++k) x[k] = *(const uint32_t *)(chunk + 16 * jc + 4 * k);
  unfold4(x, lo);
  if (full) {
    for (int k = 0; k < 4; ++k) x[k] = *(const uint32_t *)(chunk + 512 + 16 * jc + 4 * k);
    unfold4(x, hi);
  } else {
    for (int k = 0; k < 2; ++k) x[k] = *(const uint32_t *)(chunk + 512 + 8 * jc + 4 * k);
    unfold2(x, lo, hi);
  }
  const uint32_t cl = fp6_code(lo, t), ch = fp6_code(hi, t);
  const int a = (int)(8 * (ch & 31u) + (cl & 31u));
  return (cl & 32u) ? -a : a;
}
// The exponent of block b of column col, from the scale words.
__device__ inline int w_exp_of(const uint8_t *w_exp, const LGeo &g, int64_t col, int b) {
  const WLoc L = w_loc(g, b);
  const int n = (int)((col % kWCols) >> 4), c = (int)(col & 15);
  const int grp = g.group_of(L.st), k = g.byte_of(L.st);
  const int lane = L.seg <= 1 ? 16 * L.pos + c : 16 * (2 * L.pos) + c;
  return w_exp[(col / kWCols) * w_super_scale_bytes(g) + (int64_t)grp * 2048 + 32 * lane + 8 * k + n];
}

}  // namespace mxq
