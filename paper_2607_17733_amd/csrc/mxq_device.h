// mxq_device.h -- device-side building blocks shared by the libmxq kernels:
// the integer MXINT quantizer (one bf16 element given its block exponent),
// packed-layout addressing, and the unpack of packed mantissas into int8
// matrix-core operands.
//
// Format (MXSens, arXiv 2607.17733, Sections 2, 4.1, 5.1): 32-element blocks
// along K, one 8-bit shared exponent E = floor(log2 max|x|) + 127 per block,
// signed mantissas of m in {4, 6, 8} bits with LSB weight 2^(E-127-(m-2)).
//
// Everything is integer arithmetic on the bf16 bit pattern: no log2, no
// float scaling (2^-s overflows fp32 for small s, and bf16 subnormals would
// be flushed by float paths).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mxq {

constexpr int kBlock = 32;

// Segment geometry of a width map grouped as n4 4-bit, n6 6-bit, n8 8-bit
// blocks (in that order along the permuted K).
struct Segs {
  int n4, n6, n8;
};

struct BlockInfo {
  int m;        // mantissa width
  int seg;      // 0, 1, 2 for 4-, 6-, 8-bit
  int idx;      // index of the block within its segment
  int nseg;     // number of blocks in the segment
  int64_t aoff; // byte offset of the block inside a packed activation row
};

__host__ __device__ inline BlockInfo block_info(const Segs &s, int b) {
  BlockInfo r;
  if (b < s.n4) {
    r.m = 4; r.seg = 0; r.idx = b; r.nseg = s.n4;
    r.aoff = 16LL * b;
  } else if (b < s.n4 + s.n6) {
    r.m = 6; r.seg = 1; r.idx = b - s.n4; r.nseg = s.n6;
    r.aoff = 16LL * s.n4 + 24LL * r.idx;
  } else {
    r.m = 8; r.seg = 2; r.idx = b - s.n4 - s.n6; r.nseg = s.n8;
    r.aoff = 16LL * s.n4 + 24LL * s.n6 + 32LL * r.idx;
  }
  return r;
}

// ---------------------------------------------------------------------------
// Packed weight layout.  Columns form slabs of 16.  Inside a slab, the
// blocks of each width segment are grouped by four ("quads"; the last one
// may hold 1-3 blocks).  A quad chunk stores, for each of the 64 matrix-core
// lanes l = kg * 16 + c (c = column in the slab, kg = which 8 elements of the
// block), the lane's bytes of every block of the quad back to back:
//   4-bit: 4 bytes per block (8 nibbles, canonical nibble order);
//   8-bit: 8 bytes per block;
//   6-bit: a nibble plane (4 bytes per lane per block) followed by a plane of
//          top-bit words (4 bytes per lane pair (kg>>1, c) per block, same
//          word format as the activation layout).
// A full slab is 16 * (16 n4 + 24 n6 + 32 n8) bytes.
// ---------------------------------------------------------------------------
__host__ __device__ inline int64_t slab_bytes(const Segs &s) {
  return 16LL * (16LL * s.n4 + 24LL * s.n6 + 32LL * s.n8);
}

__host__ __device__ inline int64_t seg_base(const Segs &s, int seg) {
  return seg == 0 ? 0 : (seg == 1 ? 256LL * s.n4 : 256LL * s.n4 + 384LL * s.n6);
}

struct WLoc {
  int64_t lo;   // offset (in the slab) of the lane's first byte for the block
  int64_t hi;   // 6-bit only: offset of the lane pair's top-bit word
};

// Location of (block, lane) inside a slab.
__host__ __device__ inline WLoc w_loc(const Segs &s, const BlockInfo &bi,
                                      int kg, int c) {
  const int g = bi.idx >> 2, r = bi.idx & 3;
  const int rg = min(4, bi.nseg - 4 * g);
  const int64_t chunk = seg_base(s, bi.seg) + 256LL * bi.m * g;
  const int lane = kg * 16 + c;
  WLoc w;
  if (bi.m == 6) {
    w.lo = chunk + (int64_t)lane * rg * 4 + r * 4;
    w.hi = chunk + 256LL * rg + (int64_t)((kg >> 1) * 16 + c) * rg * 4 + r * 4;
  } else {
    w.lo = chunk + (int64_t)lane * rg * bi.m + r * bi.m;
    w.hi = 0;
  }
  return w;
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

// Packing of 8 consecutive mantissas (one lane's group, elements 8kg..8kg+7
// of a block).
__device__ inline uint32_t pack_nibbles(const int *q) {
  uint32_t x = 0;
#pragma unroll
  for (int t = 0; t < 8; ++t) x |= ((uint32_t)q[t] & 15u) << (4 * t);
  return x;
}

// Top two bits of eight 6-bit mantissas, placed as in the top-bit word:
// for an even group (kg even) bits 6-7 / 4-5 of bytes 0-3; for an odd group
// bits 2-3 / 0-1.
__device__ inline uint32_t pack_top2(const int *q, int odd) {
  uint32_t y = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t h0 = ((uint32_t)q[2 * j] & 63u) >> 4;
    const uint32_t h1 = ((uint32_t)q[2 * j + 1] & 63u) >> 4;
    y |= ((h0 << 6) | (h1 << 4)) << (8 * j);
  }
  return odd ? (y >> 4) : y;
}

// ---------------------------------------------------------------------------
// Unpack one lane's 8 mantissas into an int8 matrix-core operand (two
// dwords).  Each width is placed at the top of the byte, so every operand
// byte equals q * 2^(8-m): the int32 product of a block then carries a factor
// 2^(2(8-m)) and the scale of any block becomes 2^(Ea + Ew - 266)
// independently of its width.  Element order inside the lane is
// [0,2,4,6,1,3,5,7] for 4/6-bit and [0..7] for 8-bit; both operands of a
// product use the same order, so the dot product is unchanged.
// ---------------------------------------------------------------------------
__device__ inline uint64_t unpack4(uint32_t x) {
  const uint32_t ev = (x << 4) & 0xF0F0F0F0u;
  const uint32_t od = x & 0xF0F0F0F0u;
  return (uint64_t)ev | ((uint64_t)od << 32);
}

// x: nibble dword; y: top-bit word already shifted so that this lane's
// elements sit in bits 6-7 (even) and 4-5 (odd) of each byte.
__device__ inline uint64_t unpack6(uint32_t x, uint32_t y) {
  const uint32_t ev = ((x << 2) & 0x3C3C3C3Cu) | (y & 0xC0C0C0C0u);
  const uint32_t od = ((x >> 2) & 0x3C3C3C3Cu) | ((y << 2) & 0xC0C0C0C0u);
  return (uint64_t)ev | ((uint64_t)od << 32);
}

// Block scale 2^(E - 133) as fp32 (exact; denormal for E < 7), NaN for the
// E8M0 NaN code.  The product of an activation and a weight scale times the
// int32 sum of the int8 operands is the block's contribution.
__device__ inline float block_scale(int E) {
  return E == 255 ? __builtin_nanf("") : ldexpf(1.0f, E - 133);
}

// Activation operand of (row, block, kg) from the canonical packed row.
__device__ inline uint64_t load_act_operand(const uint8_t *row,
                                            const BlockInfo &bi, int kg) {
  const uint8_t *p = row + bi.aoff;
  if (bi.m == 4) {
    return unpack4(*(const uint32_t *)(p + 4 * kg));
  } else if (bi.m == 6) {
    const uint32_t x = *(const uint32_t *)(p + 4 * kg);
    const uint32_t y = *(const uint32_t *)(p + 16 + 4 * (kg >> 1));
    return unpack6(x, (kg & 1) ? (y << 4) : y);
  }
  return *(const uint64_t *)(p + 8 * kg);
}

// Weight operand of (slab, block, kg, c) from the packed weight layout.
__device__ inline uint64_t load_w_operand(const uint8_t *slab, const Segs &s,
                                          const BlockInfo &bi, int kg, int c) {
  const WLoc w = w_loc(s, bi, kg, c);
  if (bi.m == 4) return unpack4(*(const uint32_t *)(slab + w.lo));
  if (bi.m == 6) {
    const uint32_t x = *(const uint32_t *)(slab + w.lo);
    const uint32_t y = *(const uint32_t *)(slab + w.hi);
    return unpack6(x, (kg & 1) ? (y << 4) : y);
  }
  const uint32_t *p = (const uint32_t *)(slab + w.lo);
  return (uint64_t)p[0] | ((uint64_t)p[1] << 32);
}

// ---------------------------------------------------------------------------
// Matrix-core operand layout for the block-scaled MFMA
// (V_MFMA_SCALE_F32_32X32X64_F8F6F4).  That instruction multiplies FP6/FP8
// elements and applies one E8M0 scale per 32-element K-block of each operand
// in hardware.  An MXINT mantissa becomes one or two exactly representable
// "digits" whose weights are folded into the element values, so the block's
// E8M0 scale byte is the MXINT shared exponent E itself (MXSens Section 2:
// value = q * 2^(E - 127 - (m - 2))):
//   m = 4: one FP6 e3m2 element q/4;
//   m = 6: h = floor(q / 8), l = q - 8h: FP6 e3m2 elements h/2 and l/16;
//   m = 8: h = floor(q / 16), l = q - 16h: FP8 e4m3 elements h/4 and l/64.
// The product of two 6-bit (8-bit) blocks is the sum of the four digit
// products, computed by four (two) instructions over the same registers.
//
// K is walked in "steps", each one K-group of the instruction per lane half
// (lanes 32h..32h+31 hold rows / columns 0..31 of a 32-wide tile):
//   4-bit: 4 blocks (two instructions, block pairs (4t, 4t+1), (4t+2, 4t+3));
//   6-bit: a block pair, 8-bit: one block.
// 4-bit blocks are padded to a multiple of 4 and 6-bit blocks to a multiple
// of 2 with zero blocks.  Lane half h (lanes 32h..32h+31) of a step holds:
//   4-bit step t: blocks 4t+h then 4t+2+h, 24 bytes each (48 bytes);
//   6-bit pair p: block 2p+h as its h-digit plane then its l-digit plane
//                 (24 bytes each);
//   8-bit block:  h digits of elements 16h..16h+15, then their l digits
//                 (32 bytes; weights repeat the h digits: 48 bytes).
// FP6 elements are packed little-endian, element e of a block at bits 6e.
// ---------------------------------------------------------------------------
struct OpGeo {
  int n4, n6, n8;
  int n4p, n6p;          // padded segment lengths
  int s4, s6, s8;        // steps per segment
  int nsteps;
  int64_t off6, off8;    // byte offsets of the 6- and 8-bit segments in a row
  __host__ __device__ OpGeo(int a, int b, int c)
      : n4(a), n6(b), n8(c), n4p((a + 3) & ~3), n6p((b + 1) & ~1), s4(n4p / 4),
        s6(n6p / 2), s8(c), nsteps(s4 + s6 + c), off6(24LL * n4p),
        off8(24LL * n4p + 48LL * n6p) {}
  __host__ __device__ int seg(int st) const { return st < s4 ? 0 : (st < s4 + s6 ? 1 : 2); }
};

// Weight operand image: 128-column tiles, each a run of per-step chunks of
// kOpChunk bytes; a chunk holds three 16-byte parts of every (half, column)
// lane and the lane's scale dword (byte 0: first scale, byte 1: second scale
// of a 4-bit step), laid out as the prefill GEMM keeps it in LDS:
//   part j at j * 4096 + h * 2048 + c * 16, scales at 12288 + h * 512 + c * 4.
constexpr int kOpCols = 128;
constexpr int kActRows = 32;
constexpr int kActStep = 3072;       // operand bytes per (32-row tile, step)
constexpr int kActScaleStep = 256;   // scale bytes per (32-row tile, step)

// Activation operand image: byte o (0..47) of lane data (row, st, h), and
// scale byte j (0, 1) of (row, st, h).
__host__ __device__ inline int64_t act_op_loc(int64_t row, int st, int nsteps, int h, int o) {
  return ((row >> 5) * nsteps + st) * (int64_t)kActStep + (o >> 4) * 1024 + h * 512 +
         (row & 31) * 16 + (o & 15);
}
__host__ __device__ inline int64_t act_sc_loc(int64_t row, int st, int nsteps, int h, int j) {
  return ((row >> 5) * nsteps + st) * (int64_t)kActScaleStep + h * 128 + (row & 31) * 4 + j;
}
__host__ __device__ inline int64_t act_op_bytes(const OpGeo &o, int64_t rows) {
  return (rows + kActRows - 1) / kActRows * o.nsteps * (int64_t)kActStep;
}
__host__ __device__ inline int64_t act_sc_bytes(const OpGeo &o, int64_t rows) {
  return (rows + kActRows - 1) / kActRows * o.nsteps * (int64_t)kActScaleStep;
}
constexpr int kOpChunk = 13312;
constexpr int kOpPart = 4096;

__host__ __device__ inline int64_t op_tile_bytes(const OpGeo &o) {
  return (int64_t)kOpChunk * o.nsteps;
}

// Location (relative to its tile) of byte `o` (0..47) of lane (h, c) of step st.
__host__ __device__ inline int64_t w_op_loc(int st, int h, int c, int o) {
  return (int64_t)kOpChunk * st + (o >> 4) * kOpPart + h * 2048 + c * 16 + (o & 15);
}
__host__ __device__ inline int64_t w_op_scale(int st, int h, int c) {
  return (int64_t)kOpChunk * st + 3 * kOpPart + h * 512 + c * 4;
}

// FP6 e3m2 code of n/16 (|n| <= 32, n exactly representable).
__host__ __device__ inline uint32_t e3m2_sixteenths(int n) {
  const uint32_t a = (uint32_t)(n < 0 ? -n : n);
  uint32_t mag = a;
  if (a >= 4) {
    const int e = 30 - __builtin_clz(a);      // floor(log2 a) - 1
    mag = ((uint32_t)e << 2) | ((a >> (e - 1)) - 4u);
  }
  return (n < 0 ? 32u : 0u) | mag;
}

// FP8 e4m3 code of n/64 (|n| <= 128, n exactly representable).
__host__ __device__ inline uint32_t e4m3_sixtyfourths(int n) {
  const uint32_t a = (uint32_t)(n < 0 ? -n : n);
  if (a == 0) return 0;
  const int e = 32 - __builtin_clz(a);        // floor(log2 a) + 1
  const uint32_t mant = ((a << 3) >> (e - 1)) - 8u;
  return (n < 0 ? 128u : 0u) | ((uint32_t)e << 3) | mant;
}

// Digits of one mantissa: d0 (the only one for m = 4) and d1.
__host__ __device__ inline void mxint_digits(int q, int m, uint32_t &d0, uint32_t &d1) {
  if (m == 4) {
    d0 = e3m2_sixteenths(4 * q);
    d1 = 0;
  } else if (m == 6) {
    const int h = q >> 3;                     // arithmetic: floor(q / 8)
    d0 = e3m2_sixteenths(8 * h);
    d1 = e3m2_sixteenths(q - 8 * h);
  } else {
    const int h = q >> 4;
    d0 = e4m3_sixtyfourths(16 * h);
    d1 = e4m3_sixtyfourths(q - 16 * h);
  }
}

}  // namespace mxq
