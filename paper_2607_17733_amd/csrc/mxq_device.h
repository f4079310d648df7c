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

// Segment geometry of a width map grouped as n4 4-bit, n6 6-bit, n8 8-bit
// blocks (in that order along the permuted K).
struct Segs {
  int n4, n6, n8;
  int n3;       // of the n4 blocks, the first n3 hold 3-bit mantissas (stored as 2q)
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
// Stream layout (decode GEMM).  Sixteen "lines" (16 weight columns = one
// slab, or the 16 activation rows of a decode batch) are stored step by step
// in the operand order of V_MFMA_SCALE_F32_16X16X128_F8F6F4, whose lane l =
// 16 g + c (c = line) holds 32 elements of K-group g and supplies the E8M0
// scale of K-block g of its line.  Steps: the 4-bit blocks four at a time
// (padded with zero blocks to a multiple of 4), the 6-bit and the 8-bit
// blocks two at a time (each padded to a multiple of 2).  The steps of each
// segment form groups of four (the last may be shorter): a 256-byte scale
// block (lane l's scale bytes of the group's steps k = 0..3 at 4 l + k),
// then each step's lane data (lane l at LB * l unless split into planes as
// noted).
//
// With the block's E as E8M0 scale, the FP8 digits of a mantissa sum to
// q * 2^-(m-2): e4m3(q/4) for a 4-bit q; two digits for 6- and 8-bit q.
// Weights keep the packed mantissas (4m bits per element) and become these
// digits in registers.  With the symmetric clamp (no -2^(m-1)) 4- and 6-bit
// mantissas are stored sign-magnitude, so a digit is one 8-entry byte lookup
// plus the sign bit: a 4-bit code is s|(|q|) (3 magnitude bits), a 6-bit code
// a nibble s|(|q| mod 8) plus the 2-bit |q| div 8 (digits h/2 and l/16 of
// |q| = 8h + l).  With the full clamp they are two's complement (q mod 16,
// and bits 4-5: digits h and l/16 of q = 16h + l).  8-bit mantissas are two's
// complement in both modes (digits h/4 and l/64 of q = 16h + l).
//   4-bit step s: lane (g, c) holds 16 bytes: elements 16(g&1)..16(g&1)+15 of
//     block 4s+(g>>1) (bytes 0-7), then the same elements of block
//     4s+2+(g>>1) (bytes 8-15), as nibble codes: the dword of elements
//     e0..e7 has byte k = code(e_k) | code(e_{k+4}) << 4.  Scale byte of lane
//     (g, c): E of block 4s+g.
//   6-bit step s: lane (g, c) holds 12 bytes for elements 16(g&1)+0..15 of
//     block 2s+(g>>1): their nibble codes (8 bytes at 8 l, same nibble
//     order) and a dword of their 2-bit codes (at 512 + 4 l: element t at
//     bits 8(t%4) + 2(t/4)).
//   8-bit step s: lane (g, c) holds 16 bytes: the same 16 elements of block
//     2s+(g>>1) as two's-complement bytes.
//   6/8-bit scale byte of lane (g, c): E of block 2s+(g&1).
// Activations (decode image, M <= 16) are stored as ready operands:
//   4-bit step s: lane (g, r) holds block 4s+g of row r as 32 FP6 e3m2
//     codes of q/4 (24 bytes: the first 16 at 16 l, the last 8 at
//     1024 + 8 l); scale byte E of block 4s+g.
//   6/8-bit step s: lane (g, r) holds elements 16(g&1)+0..15 of block
//     2s+(g>>1): the e4m3 codes of their high digits (16 bytes) then of
//     their low digits (16 bytes); scale byte E of block 2s+(g&1).
// ---------------------------------------------------------------------------
constexpr int kStreamLanes = 64;
constexpr int kStreamGroup = 4;          // steps sharing one scale block
constexpr int kScaleBlock = 256;         // 64 lanes x 4 scale bytes

struct DGeo {
  int n4, n6, n8;
  int S[3];              // steps of each segment
  int nsteps;
  __host__ __device__ DGeo(int a, int b, int c) : n4(a), n6(b), n8(c) {
    S[0] = (a + 3) / 4;
    S[1] = (b + 1) / 2;
    S[2] = (c + 1) / 2;
    nsteps = S[0] + S[1] + S[2];
  }
};

// lane-data bytes of a weight / activation step of each segment
__host__ __device__ constexpr int wd_lane_bytes(int seg) { return seg == 1 ? 12 : 16; }
__host__ __device__ constexpr int ad_lane_bytes(int seg) { return seg == 0 ? 24 : 32; }
// bytes of the 64 lanes' data of one step
__host__ __device__ constexpr int wd_step_data(int seg) { return kStreamLanes * wd_lane_bytes(seg); }
__host__ __device__ constexpr int ad_step_data(int seg) { return kStreamLanes * ad_lane_bytes(seg); }

// A segment of S steps is a run of groups of kStreamGroup steps (the last one
// may be shorter): each group is its scale block (lane l's scale byte for
// step k of the group at 4 l + k) followed by its steps' lane data.
__host__ __device__ inline int64_t seg_bytes(int S, int step_data) {
  return (int64_t)S * step_data + (int64_t)((S + kStreamGroup - 1) / kStreamGroup) * kScaleBlock;
}
__host__ __device__ inline int64_t grp_off(int g, int step_data) {
  return (int64_t)g * (kStreamGroup * step_data + kScaleBlock);
}
// byte offset of segment seg in a weight slab / the activation decode image
__host__ __device__ inline int64_t wd_seg_off(const DGeo &d, int seg) {
  int64_t o = 0;
  for (int s = 0; s < seg; ++s) o += seg_bytes(d.S[s], wd_step_data(s));
  return o;
}
__host__ __device__ inline int64_t ad_seg_off(const DGeo &d, int seg) {
  int64_t o = 0;
  for (int s = 0; s < seg; ++s) o += seg_bytes(d.S[s], ad_step_data(s));
  return o;
}
__host__ __device__ inline int64_t wd_slab_bytes(const DGeo &d) { return wd_seg_off(d, 3); }
__host__ __device__ inline int64_t ad_image_bytes(const DGeo &d) { return ad_seg_off(d, 3); }

// Where block `idx` of segment `seg` lives in the stream layout: its step
// within the segment, the lane group of each half (elements 16h..16h+15 sit
// in lane group g0 + h), the byte offset of its elements inside a 4-bit lane
// (0 or 8) and the lane groups whose scale byte is the block's exponent (one
// for 4-bit blocks, two for 6/8-bit blocks).
struct DLoc {
  int st, g0, region, sg0, sg1;
};
__host__ __device__ inline DLoc d_loc(int seg, int idx) {
  DLoc r;
  if (seg == 0) {
    r.st = idx >> 2;
    r.g0 = 2 * (idx & 1);
    r.region = 8 * ((idx >> 1) & 1);
    r.sg0 = r.sg1 = idx & 3;
  } else {
    r.st = idx >> 1;
    r.g0 = 2 * (idx & 1);
    r.region = 0;
    r.sg0 = idx & 1;
    r.sg1 = r.sg0 + 2;
  }
  return r;
}

// Step st of a segment starting at `seg`: its data and its group's scales.
__host__ __device__ inline int64_t step_data_off(int st, int step_data) {
  return grp_off(st / kStreamGroup, step_data) + kScaleBlock +
         (int64_t)(st % kStreamGroup) * step_data;
}
__host__ __device__ inline int64_t step_scale_off(int st, int step_data, int lane) {
  return grp_off(st / kStreamGroup, step_data) + 4 * lane + st % kStreamGroup;
}

// Stream codes of a mantissa: the nibble (4-bit q, or the low part of a
// 6-bit q) and the 2-bit high part of a 6-bit q; sm = sign-magnitude
// (symmetric clamp), else two's complement.
__host__ __device__ inline uint32_t stream_nibble(int q, int m, bool sm) {
  if (!sm) return (uint32_t)q & 15u;
  const uint32_t a = (uint32_t)(q < 0 ? -q : q);
  return (q < 0 ? 8u : 0u) | (m == 4 ? a : (a & 7u));
}
__host__ __device__ inline uint32_t stream_top2(int q, bool sm) {
  if (!sm) return ((uint32_t)q >> 4) & 3u;
  return (uint32_t)(q < 0 ? -q : q) >> 3;
}

// Weight stream nibble dword of eight mantissas q[0..7] of width m.
__host__ __device__ inline uint32_t stream_nibbles(const int *q, int m, bool sm) {
  uint32_t x = 0;
  for (int k = 0; k < 4; ++k)
    x |= (stream_nibble(q[k], m, sm) | (stream_nibble(q[k + 4], m, sm) << 4)) << (8 * k);
  return x;
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
// Element accessors (debug / parity kernels): mantissa t (0..31) of a block.
// ---------------------------------------------------------------------------
__device__ inline int sext_bits(uint32_t v, int bits) {
  const int sh = 32 - bits;
  return ((int)(v << sh)) >> sh;
}

// Canonical packed activation row (layout in include/mxq.h).
__device__ inline int act_elem(const uint8_t *row, const BlockInfo &bi, int t) {
  const uint8_t *p = row + bi.aoff;
  if (bi.m == 8) return (int)(int8_t)p[t];
  const uint32_t nib = (p[t >> 1] >> (4 * (t & 1))) & 15u;
  if (bi.m == 4) return sext_bits(nib, 4);
  const int d = t >> 4, u = t & 15;
  const int j = (u & 7) >> 1;
  const int sh = (u < 8 ? 6 : 2) - 2 * (u & 1);
  const uint32_t top = (p[16 + 4 * d + j] >> sh) & 3u;
  return sext_bits(nib | (top << 4), 6);
}

// Weight slab in the stream layout (see DGeo); c = column within the slab,
// sm = sign-magnitude codes (symmetric clamp).
__device__ inline int wstream_elem(const uint8_t *slab, const DGeo &dg, const BlockInfo &bi,
                                   int c, int t, bool sm) {
  const DLoc L = d_loc(bi.seg, bi.idx);
  const uint8_t *chunk = slab + wd_seg_off(dg, bi.seg) + step_data_off(L.st, wd_step_data(bi.seg));
  const int ln = 16 * (L.g0 + (t >> 4)) + c;
  const int u = t & 15;                     // element within the half
  if (bi.m == 8) return (int)(int8_t)chunk[16 * ln + u];
  const int d = u >> 3, k = u & 7;
  const uint8_t *nb = bi.m == 4 ? chunk + 16 * ln + L.region : chunk + 8 * ln;
  const uint32_t nib = (nb[4 * d + (k & 3)] >> (4 * (k >> 2))) & 15u;
  if (bi.m == 4) return sm ? ((nib & 8u) ? -(int)(nib & 7u) : (int)(nib & 7u)) : sext_bits(nib, 4);
  const uint32_t y = *(const uint32_t *)(chunk + 512 + 4 * ln);
  const uint32_t top = (y >> (8 * (k & 3) + 4 * d + 2 * (k >> 2))) & 3u;
  if (sm) {
    const int a = (int)(top * 8u + (nib & 7u));
    return (nib & 8u) ? -a : a;
  }
  return sext_bits(nib | (top << 4), 6);
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
//   part j at j * 4096 + h * 2048 + c * 16, scales at 12288 + h * 512 +
//   (c % 32) * 16 + (c / 32) * 4 (a lane's four 32-column tiles' scale
//   dwords are adjacent: one 16-byte LDS read per step).
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
  return (int64_t)kOpChunk * st + 3 * kOpPart + h * 512 + (c & 31) * 16 + (c >> 5) * 4;
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
