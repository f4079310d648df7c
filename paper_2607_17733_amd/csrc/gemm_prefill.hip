// gemm_prefill.hip -- MXINT GEMM for prefill shapes on the block-scaled
// matrix cores of gfx950.
//
// Y[i][j] = sum_b sum_k qa[i][k] qw[j][k] 2^(Ea[i][b] + Ew[j][b] - 254 - 2(m_b - 2))
// (MXSens, arXiv 2607.17733, Section 2: integer mantissas with one
// power-of-two scale per 32-element block; Section 6: mixed widths in one
// GEMM).
//
// Operands (LGeo in mxq_device.h): the activations as the quantizer's
// operand image (ready FP6/FP8 codes), the weights in the one layout both
// GEMMs read, at the MXINT size: folded FP6 codes for 3- and 4-bit blocks,
// two digit planes for 6-bit blocks, mantissa bytes for 8-bit blocks.  Both
// layouts are in the lane order of the 16x16x128 instruction; this kernel
// runs V_MFMA_SCALE_F32_32X32X64_F8F6F4, whose lane (h, x) (K half h, row /
// column x of a 32-wide tile) takes, for K-chunk c of a step, the 32 FP6
// values that lane (2c + h, x % 16) of 16-row tile / 16-column slab x / 16
// holds (for FP8 steps: block c's 16 high digits from lane (h, x % 16) and
// its 16 low digits from lane (2 + h, x % 16)), so the operands are read with
// a per-lane address and no data is moved.  Each
// lane restores its weight operand from LDS with a few masks and shifts;
// the hardware applies every block's E8M0 scale and accumulates in fp32.
// Per 32x32 tile and K-chunk (64 K-values):
//   3- and 4-bit (two blocks): one FP6 instruction;
//   6-bit (one block, its two digit planes as the K halves): two FP6
//     instructions, the weights' high plane in both halves, then the low;
//   8-bit (one block, the same way): two FP8 instructions.
// The digit products are exact; only the fp32 accumulation rounds.
//
// Tiling: 256x128 outputs per workgroup (one weight super-slab) of eight
// waves in two K groups of four, one wave of each group per SIMD.  Group g
// takes the steps s with s % 2 == g; wave (g, r) owns rows 64r..64r+63 x all
// 128 columns = 2x4 tiles of 32x32 fp32 accumulators, and the groups'
// partial sums meet in LDS at the end.
//
//   - activations go straight from the image into registers -- each row is
//     used by exactly one wave -- one iteration (two steps) ahead, in two
//     register sets, with the step's weight scale bytes;
//   - the weight chunk of each step (8 slabs, 6 to 12 KB) goes global -> LDS
//     by direct-to-LDS loads into a ring of eight step stages, three
//     iterations ahead; the four waves of a group read it per column tile,
//     one tile ahead of the products.
// One barrier per iteration; the kernel counts its own loads (vmcnt) to know
// when a stage is complete.  Workgroup ids are remapped so that each XCD owns
// a compact block of output tiles: the activation rows and weight columns it
// reads stay in its L2.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef unsigned u2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int BM = 256, BN = kWCols, NT = 512;
constexpr int kFmtE4M3 = 0, kFmtE2M3 = 2, kFmtE3M2 = 3;
constexpr int kWStages = 8;                  // weight ring: 4 iterations of 2 steps
// Reduction of the two groups: [column][row] floats, 256 rows + 4 padding.
constexpr int kRedPitch = 260;
// Loads per wave and iteration besides the weights: per 32-row tile two
// K-chunks of lane data (two loads each) and their two scale words, then
// the step's weight scale bytes (two).
constexpr int kALoads = 2 * (4 + 2) + 2;

template <int S> struct Int { static constexpr int v = S; };

template <bool FULL> struct Cfg {
  static constexpr int kPieces = FULL ? 12 : 8;           // 1 KB pieces per stage
  static constexpr int kStage = kPieces * 1024;
  static constexpr int kRing = kWStages * kStage;
  static constexpr int kWLoads = 2 * kPieces / 8;         // per wave and iteration
  static constexpr int kLds = kRing > 128 * kRedPitch * 4 ? kRing : 128 * kRedPitch * 4;
};
static_assert(Cfg<true>::kLds <= 160 * 1024, "LDS");

template <int FA, int FB>
__device__ inline v16f mma(const v8i &a, const v8i &b, v16f c, uint32_t sa, uint32_t sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, FA, FB, 0, (int)sa, 0, (int)sb);
}

template <int N>
__device__ inline void wait_loads_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(N) : "memory");
}
template <int N>
__device__ inline void wait_loads() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ inline void barrier() { asm volatile("s_barrier" ::: "memory"); }

// 4x4 transpose within each quad of lanes: lane j of a quad holds v[i] = the
// element of row i, column j; afterwards it holds row j, columns 0..3.
template <int CTRL>
__device__ inline float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF,
                                                             0xF, false));
}
__device__ inline v4f quad_transpose(v4f a, int j) {
  // swap the off-diagonal 2x2 blocks with lane j ^ 2, then within them with j ^ 1
  const bool b1 = j & 2, b0 = j & 1;
  constexpr int kSwap2 = 0x4E, kSwap1 = 0xB1;   // quad_perm [2,3,0,1] and [1,0,3,2]
  const float u0 = dpp<kSwap2>(b1 ? a[0] : a[2]);
  const float u1 = dpp<kSwap2>(b1 ? a[1] : a[3]);
  v4f x;
  x[0] = b1 ? u0 : a[0];
  x[1] = b1 ? u1 : a[1];
  x[2] = b1 ? a[2] : u0;
  x[3] = b1 ? a[3] : u1;
  const float w0 = dpp<kSwap1>(b0 ? x[0] : x[1]);
  const float w1 = dpp<kSwap1>(b0 ? x[2] : x[3]);
  v4f y;
  y[0] = b0 ? w0 : x[0];
  y[1] = b0 ? x[1] : w0;
  y[2] = b0 ? w1 : x[2];
  y[3] = b0 ? x[3] : w1;
  return y;
}

// The lane id as a value the compiler cannot hoist: lane-dependent offsets
// are recomputed where they are used (a few VALU operations) instead of
// being kept live, one register each, across the whole kernel.
__device__ inline int fresh_lane() {
  int x = (int)__lane_id();
  asm volatile("" : "+v"(x));
  return x;
}

__device__ inline v8i six(const uint32_t *d) {
  const u4 lo = u4{d[0], d[1], d[2], d[3]};
  const u4 hi = u4{d[4], d[5], d[5], d[5]};
  return (v8i)__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, -1, -1);
}

// E8M0 scale byte e + N, saturating at 255 (NaN).
template <int N>
__device__ inline uint32_t sat_plus(uint32_t e) {
  const uint32_t v = e + N;
  return v < 255u ? v : 255u;
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

template <bool FULL>
__global__ __launch_bounds__(NT, 1) void gemm_prefill_kernel(GemmArgs g, int mtiles, int ntiles,
                                                             int gm, int gn) {
  using C = Cfg<FULL>;
  __shared__ __attribute__((aligned(16))) u4 lds[C::kLds / 16];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);      // wave-uniform
  const int l32 = lane & 31, lh = lane >> 5, l16 = lane & 15, hx = l32 >> 4;
  const int kg = wave >> 2, wr = wave & 3;                      // K group, row block
  int mt, nt;
  {
    // XCD x (workgroups pid % 8 == x) owns a block of (mtiles / gm) x
    // (ntiles / gn) tiles, walked row by row.
    const int pid = blockIdx.x;
    if (gm > 0) {
      const int x = pid & 7, loc = pid >> 3;
      const int bm = mtiles / gm, bn = ntiles / gn;
      mt = (x / gn) * bm + loc / bn;
      nt = (x % gn) * bn + loc % bn;
    } else {
      mt = pid / ntiles;
      nt = pid - mt * ntiles;
    }
  }
  const int64_t row0 = (int64_t)mt * BM, col0 = (int64_t)nt * BN;
  const LGeo lg(g.n3, g.n4, g.n6, g.n8);
  const int nsteps = lg.nsteps;
  char *const ring = (char *)lds;

  // This wave's rows: two 32-row tiles = four 16-row image tiles (tiles
  // past the last one read the last tile; those rows are never stored).  The
  // activation resources start at the wave's first 16-row tile (64-bit
  // arithmetic), so the 32-bit buffer offsets stay below 4 image tiles; the
  // host rejects shapes where 16 tiles pass INT32_MAX.
  const int64_t last = (g.M - 1) / kATileRows;
  const int64_t ta = min(row0 / kATileRows + 4 * wr, last);
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.a_mant + ta * g.a_tile), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.a_exp + ta * g.a_tile_sc), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.w_mant + (int64_t)nt * g.w_super), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rws = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.w_exp + (int64_t)nt * g.w_super_sc), 0, 0x7fffffff, 0x00020000);
  const int v16 = lane * 16;
  // The lane (lh, x) of the 32-wide tile reads, for K-chunk c, what lane
  // 16 (2 c + lh) + x % 16 of 16-row tile / slab x / 16 holds; the lane of a
  // 32-row tile tm is in image tile 2 tm + x / 16.

  v16f acc[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[a][n] = v16f{};

  // Activation registers of one step: per 32-row tile and K-chunk the lane
  // data (24 bytes for FP6 steps, 32 for FP8 steps) and the scale word; the
  // step's weight scale bytes for each K-chunk (slab n at byte n).  The two
  // shapes are kept apart so that the FP6 segments hold 24-byte sets only:
  // FP8 sets are first loaded by the last FP6 iteration (or the prologue)
  // right before the FP8 segment.
  struct A6 {
    u4 p[2][2];
    u2 q[2][2];
    uint32_t sc[2][2];
    u2 ws[2];
  };
  struct A8 {
    u4 p[2][2], r[2][2];
    uint32_t sc[2][2];
    u2 ws[2];
  };
  A6 xa6[2];
  A8 xa8[2];

  // Offsets of step st in the images, its scale group and its byte.
  auto seg_of = [&](int st) __attribute__((always_inline)) {
    return st < lg.st0[1] ? 0 : st < lg.st0[2] ? 1 : st < lg.st0[3] ? 2 : 3;
  };
  auto seg_start = [&](int sg) __attribute__((always_inline)) {
    return sg == 0 ? 0 : sg == 1 ? lg.st0[1] : sg == 2 ? lg.st0[2] : lg.st0[3];
  };
  auto a_off = [&](int st) __attribute__((always_inline)) {
    const int sg = seg_of(st);
    int o = 0;
    if (sg > 0) o += lg.S[0] * kLanes * 24;
    if (sg > 1) o += lg.S[1] * kLanes * 24;
    if (sg > 2) o += lg.S[2] * kLanes * 24;
    return o + (st - seg_start(sg)) * kLanes * (sg == 3 ? 32 : 24);
  };
  auto w_off = [&](int st, int &pieces) __attribute__((always_inline)) {
    const int sg = seg_of(st);
    int o = 0;
    if (sg > 0) o += lg.S[0] * kWSlabs * w_chunk_bytes(0, FULL);
    if (sg > 1) o += lg.S[1] * kWSlabs * w_chunk_bytes(1, FULL);
    if (sg > 2) o += lg.S[2] * kWSlabs * w_chunk_bytes(2, FULL);
    const int cb = sg == 0 ? w_chunk_bytes(0, FULL) : sg == 1 ? w_chunk_bytes(1, FULL)
                 : sg == 2 ? w_chunk_bytes(2, FULL) : w_chunk_bytes(3, FULL);
    pieces = cb * kWSlabs / 1024;
    return o + (st - seg_start(sg)) * kWSlabs * cb;
  };
  auto s_grp = [&](int st) __attribute__((always_inline)) {
    const int sg = seg_of(st);
    const int g0 = sg == 0 ? 0 : sg == 1 ? lg.G0[1] : sg == 2 ? lg.G0[2] : lg.G0[3];
    return g0 + (st - seg_start(sg)) / kGroupSteps;
  };
  auto s_byte = [&](int st) __attribute__((always_inline)) {
    return (st - seg_start(seg_of(st))) % kGroupSteps;
  };

  // Weight loads of iteration it (steps 2 it, 2 it + 1) into their stages:
  // pieces n = 0 .. 2 kPieces - 1 of 1 KB (a step's pieces past its chunk
  // bytes repeat its last piece); wave w issues n = w + 8 j.
  auto issue_w = [&](int it) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < C::kWLoads; ++j) {
      const int n = wave + 8 * j;
      const int st = min(2 * it + n / C::kPieces, nsteps - 1);
      int have;
      const int wo = w_off(st, have);
      const int kb = min(n % C::kPieces, have - 1);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rw, (lds_void *)(ring + (st % kWStages) * C::kStage + kb * 1024), 16, v16,
          wo + kb * 1024, 0, 0);
    }
  };
  // Activation loads of the wave's step in iteration it, row tile tm, into
  // register set S of shape WIDE (and, with tm = 1, the step's weight scale
  // bytes): six loads per row tile and two for the scales, whatever the shape.
  auto issue_a_half = [&](auto set_tag, auto wide_tag, int it, int tm) __attribute__((always_inline)) {
    constexpr int S = decltype(set_tag)::v;
    constexpr bool WIDE = decltype(wide_tag)::v;
    const int st = min(2 * it + kg, nsteps - 1);
    const int so = __builtin_amdgcn_readfirstlane(a_off(st));
    constexpr int lb = WIDE ? 32 : 24;
    const int sgrp = s_grp(st);
    const int fl = fresh_lane();
    const int fk0 = (fl & 15) + 16 * (fl >> 5), fk1 = fk0 + 32;
    const int vtile = (int)(min(ta + 2 * tm + ((fl >> 4) & 1), last) - ta);
    uint32_t *sc = WIDE ? xa8[S].sc[tm] : xa6[S].sc[tm];
    u2 *ws = WIDE ? xa8[S].ws : xa6[S].ws;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int vt = vtile * (int)g.a_tile;
      if (WIDE) {
        // chunk c = block c of the step: the high digits of the lane's 16
        // elements (lane group lh, bytes 16 c) as K-block 0, their low
        // digits (lane group 2 + lh) as K-block 1
        xa8[S].p[tm][c] = __builtin_bit_cast(
            u4, __builtin_amdgcn_raw_buffer_load_b128(ra, vt + 32 * fk0 + 16 * c, so, 0));
        xa8[S].r[tm][c] = __builtin_bit_cast(
            u4, __builtin_amdgcn_raw_buffer_load_b128(ra, vt + 32 * fk1 + 16 * c, so, 0));
      } else {
        const int vo = vt + lb * (c ? fk1 : fk0);
        const u4 d0 = __builtin_bit_cast(u4, __builtin_amdgcn_raw_buffer_load_b128(ra, vo, so, 0));
        xa6[S].p[tm][c] = d0;
        xa6[S].q[tm][c] =
            __builtin_bit_cast(u2, __builtin_amdgcn_raw_buffer_load_b64(ra, vo + 16, so, 0));
      }
      sc[c] = __builtin_amdgcn_raw_buffer_load_b32(
          rs, vtile * (int)g.a_tile_sc + 4 * (c ? fk1 : fk0),
          __builtin_amdgcn_readfirstlane(sgrp * 256), 0);
    }
    if (tm == 1) {
      const int sb = __builtin_amdgcn_readfirstlane(sgrp * 2048 + 8 * s_byte(st));
#pragma unroll
      for (int c = 0; c < 2; ++c)
        ws[c] = __builtin_bit_cast(
            u2, __builtin_amdgcn_raw_buffer_load_b64(rws, 32 * (c ? fk1 : fk0), sb, 0));
    }
  };

  // Weight operand of column tile tn, K-chunk c: the raw bytes of the lane
  // (two chunks in flight), restored to FP6 / FP8 codes at use.
  struct WRaw {
    u4 p, h;
    u2 q;
    uint32_t z;
  };
  WRaw w[2];
  auto read_w = [&](auto seg, const char *stage, int o, int tn, int c) __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v;
    constexpr int CB = w_chunk_bytes(SEG, FULL);
    const int fl = fresh_lane(), f16 = fl & 15, fh = fl >> 5;
    const char *ch = stage + (2 * tn + ((fl >> 4) & 1)) * CB;
    const int lk = f16 + 16 * (2 * c + fh);
    WRaw &r = w[o];
    if (SEG == 0 && !FULL) {
      r.q = *(const u2 *)(ch + 8 * lk);
      r.z = *(const uint32_t *)(ch + 512 + 4 * lk);
    } else if (SEG <= 1) {
      r.p = *(const u4 *)(ch + 16 * lk);
      if (SEG == 1 && FULL) r.q = *(const u2 *)(ch + 1024 + 8 * lk);
    } else if (SEG == 2) {
      const int jc = 16 * c + f16;
      r.p = *(const u4 *)(ch + 16 * jc);
      if (FULL) {
        r.h = *(const u4 *)(ch + 512 + 16 * jc);
      } else {
        r.q = *(const u2 *)(ch + 512 + 8 * jc);
      }
    } else {
      r.p = *(const u4 *)(ch + 32 * (16 * c + f16) + 16 * fh);
    }
  };

  // Iteration it: the products of this wave's step s = 2 it + kg from
  // register set S, column tile by column tile, each tile's weight operand
  // read one tile ahead.  Each iteration issues a bundle of loads, the
  // activations of it + 1 (into the other register set, around tiles 0 and
  // 1) and then the weights of it + 3 (at tile 2).  Between tiles 1 and 2
  // the workgroup meets at a barrier.  Before it each wave waits for its own
  // weight loads of iteration it + 1 (issued before the bundle of it - 1,
  // the weights of it + 2 and the activations of it + 1); after it the
  // stages of it + 1 are complete, so tile 0 of the next step is read during
  // tile 3, and every wave is past iteration it - 1, whose stages the
  // weights of it + 3 then overwrite.
  auto iteration = [&](auto seg, auto set_tag, auto nw_tag, int it, bool mul)
                       __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v, S = decltype(set_tag)::v;
    auto hook = [&](int tn) __attribute__((always_inline)) {
      if (tn == 0) issue_a_half(Int<1 - S>{}, nw_tag, it + 1, 0);
      else if (tn == 1) issue_a_half(Int<1 - S>{}, nw_tag, it + 1, 1);
      else if (tn == 2) issue_w(it + 3);
    };
    auto meet = [&]() __attribute__((always_inline)) {
      wait_loads<2 * kALoads + C::kWLoads>();
      barrier();
    };
    if (!mul) {
      hook(0);
      hook(1);
      meet();
      hook(2);
      return;
    }
    const int s = 2 * it + kg;
    const char *W = ring + (s % kWStages) * C::kStage;
    const int kb = s_byte(s);
    const uint32_t(&xsc)[2][2] = SEG == 3 ? xa8[S].sc : xa6[S].sc;
    const u2(&xws)[2] = SEG == 3 ? xa8[S].ws : xa6[S].ws;
    // activation scales of the step
    uint32_t sa[2][2];
#pragma unroll
    for (int tm = 0; tm < 2; ++tm)
#pragma unroll
      for (int c = 0; c < 2; ++c) sa[tm][c] = (xsc[tm][c] >> (8 * kb)) & 0xFFu;
#pragma unroll
    for (int tc = 0; tc < 8; ++tc) {
      const int tn = tc >> 1, c = tc & 1, o = tc & 1;
      if (tc == 4) meet();
      if (tc < 7) {
        read_w(seg, W, o ^ 1, (tc + 1) >> 1, (tc + 1) & 1);
      } else {
        // chunk 0 of tile 0 of the wave's next step (its stage is complete
        // after the barrier of this iteration)
        const int s2 = s + 2;
        if (s2 < nsteps && seg_of(s2) == SEG) read_w(seg, ring + (s2 % kWStages) * C::kStage, 0, 0, 0);
      }
      if (c == 0) hook(tn);
      const int n = 2 * tn + hx;             // the lane's slab
      const uint32_t e = (xws[c][n >> 2] >> (8 * (n & 3))) & 0xFFu;
      const WRaw &r = w[o];
      v8i av[2];
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) {
        if (SEG == 3) {
          av[tm] = (v8i)__builtin_shufflevector(xa8[S].p[tm][c], xa8[S].r[tm][c], 0, 1, 2, 3, 4, 5,
                                                6, 7);
        } else {
          const u4 q4 = u4{xa6[S].q[tm][c][0], xa6[S].q[tm][c][1], 0u, 0u};
          av[tm] = (v8i)__builtin_shufflevector(xa6[S].p[tm][c], q4, 0, 1, 2, 3, 4, 5, -1, -1);
        }
      }
      if (SEG <= 1) {
        uint32_t d[6];
        if (SEG == 0 && !FULL) {
          const uint32_t f[3] = {r.q[0], r.q[1], r.z};
          unfold3(f, d);
        } else if (SEG == 1 && FULL) {
          d[0] = r.p[0]; d[1] = r.p[1]; d[2] = r.p[2]; d[3] = r.p[3]; d[4] = r.q[0]; d[5] = r.q[1];
        } else {
          const uint32_t f[4] = {r.p[0], r.p[1], r.p[2], r.p[3]};
          unfold4(f, d);
        }
        constexpr int FB = SEG == 0 ? kFmtE2M3 : kFmtE3M2;
        const v8i b = six(d);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
          acc[tm][tn] = mma<kFmtE3M2, FB>(av[tm], b, acc[tm][tn], sa[tm][c], e);
      } else if (SEG == 2) {
        // the block's digit planes are the K halves of both operands: the
        // weights' high plane in both halves (scale E + 3) gives hh and lh,
        // their low plane (scale E) hl and ll
        const uint32_t fl[4] = {r.p[0], r.p[1], r.p[2], r.p[3]};
        uint32_t L[6], H[6];
        unfold4(fl, L);
        if (FULL) {
          const uint32_t fh[4] = {r.h[0], r.h[1], r.h[2], r.h[3]};
          unfold4(fh, H);
        } else {
          const uint32_t fh[2] = {r.q[0], r.q[1]};
          unfold2(fh, L, H);
        }
        const v8i bh = six(H);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
          acc[tm][tn] = mma<kFmtE3M2, kFmtE3M2>(av[tm], bh, acc[tm][tn], sa[tm][c], sat_plus<3>(e));
        const v8i bl = six(L);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
          acc[tm][tn] = mma<kFmtE3M2, kFmtE3M2>(av[tm], bl, acc[tm][tn], sa[tm][c], e);
      } else {
        // the weights' high digits in both K halves (scale E + 4), then
        // their low digits (scale E)
        v8i bh;
#pragma unroll
        for (int k = 0; k < 4; ++k) bh[k] = bh[4 + k] = (int)hi_codes<FULL>(r.p[k]);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
          acc[tm][tn] = mma<kFmtE4M3, kFmtE4M3>(av[tm], bh, acc[tm][tn], sa[tm][c], sat_plus<4>(e));
        v8i bl;
#pragma unroll
        for (int k = 0; k < 4; ++k) bl[k] = bl[4 + k] = (int)lo_codes<FULL>(r.p[k]);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
          acc[tm][tn] = mma<kFmtE4M3, kFmtE4M3>(av[tm], bl, acc[tm][tn], sa[tm][c], e);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Group g's steps 2 it + g of segment [b, e) are the iterations
  // [(b - g + 1) / 2, (e - g + 1) / 2).
  auto bound = [&](int e) { return (e - kg + 1) >> 1; };
  const int i1 = bound(lg.st0[1]), i2 = bound(lg.st0[2]), i3 = bound(lg.st0[3]),
            i4 = bound(nsteps);
  // Iterations [ib, ie) of one segment (register set = it % 2), prefetching
  // the activations of the same shape.  The first iteration of a segment
  // reads its own first weight chunk (the previous segment's last iteration
  // reads it only when the segment does not change).
  auto run = [&](auto seg, int ib, int ie) __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v;
    using NW = Int<SEG == 3>;
    int it = ib;
    if (it < ie) {
      const int s = 2 * it + kg;
      read_w(seg, ring + (s % kWStages) * C::kStage, 0, 0, 0);
    }
    if (it < ie && (it & 1)) iteration(seg, Int<1>{}, NW{}, it++, true);
    for (; it + 2 <= ie; it += 2) {
      iteration(seg, Int<0>{}, NW{}, it, true);
      iteration(seg, Int<1>{}, NW{}, it + 1, true);
    }
    if (it < ie) iteration(seg, Int<0>{}, NW{}, it, true);
  };
  // The last FP6 iteration, it = i3 - 1, which prefetches the first FP8 set.
  auto last_fp6 = [&](auto seg) __attribute__((always_inline)) {
    const int it = i3 - 1;
    const int s = 2 * it + kg;
    read_w(seg, ring + (s % kWStages) * C::kStage, 0, 0, 0);
    if (it & 1) iteration(seg, Int<1>{}, Int<1>{}, it, true);
    else iteration(seg, Int<0>{}, Int<1>{}, it, true);
  };

  // Prologue: weights of iterations 0 and 1, then the bundle of iteration -1
  // (activations of 0, weights of 2), and the wait for the stages of
  // iteration 0 (issued before the weights of 1, the activations of 0 and
  // the weights of 2).
  issue_w(0);
  issue_w(1);
  __builtin_amdgcn_sched_barrier(0);
  if (i3 == 0) {
    // every step of this wave is FP8
    issue_a_half(Int<0>{}, Int<1>{}, 0, 0);
    issue_a_half(Int<0>{}, Int<1>{}, 0, 1);
    __builtin_amdgcn_sched_barrier(0);
    issue_w(2);
    __builtin_amdgcn_sched_barrier(0);
    wait_loads<C::kWLoads + kALoads + C::kWLoads>();
    barrier();
  } else {
    issue_a_half(Int<0>{}, Int<0>{}, 0, 0);
    issue_a_half(Int<0>{}, Int<0>{}, 0, 1);
    __builtin_amdgcn_sched_barrier(0);
    issue_w(2);
    __builtin_amdgcn_sched_barrier(0);
    wait_loads<C::kWLoads + kALoads + C::kWLoads>();
    barrier();
    // the FP6 segments but their last iteration, then that one
    const int j = i3 - 1;
    run(Int<0>{}, 0, min(i1, j));
    run(Int<1>{}, min(i1, j), min(i2, j));
    run(Int<2>{}, min(i2, j), j);
    const int sg = seg_of(2 * j + kg);
    if (sg == 0) last_fp6(Int<0>{});
    else if (sg == 1) last_fp6(Int<1>{});
    else last_fp6(Int<2>{});
  }
  run(Int<3>{}, i3, i4);
  // Group 1 has one iteration less when nsteps is odd; it still meets the
  // barrier of group 0's last iteration.
  const int niter = (nsteps + 1) >> 1;
  if (i4 < niter) {
    if (i4 & 1) iteration(Int<3>{}, Int<1>{}, Int<1>{}, i4, false);
    else iteration(Int<3>{}, Int<0>{}, Int<1>{}, i4, false);
  }
  wait_loads_lds<0>();
  barrier();                                 // every wave is done with the ring

  // Reduction: group 1 leaves its sums in LDS as [column][row] (four rows of
  // a lane's tile are one 16-byte write), group 0 adds them, transposes each
  // quad of lanes to row pieces of four columns, and stores 16 bytes a lane.
  float *red = (float *)ring;
  if (kg == 1) {
#pragma unroll
    for (int tm = 0; tm < 2; ++tm)
#pragma unroll
      for (int tn = 0; tn < 4; ++tn)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int rr = wr * 64 + tm * 32 + 8 * q + 4 * lh, cc = tn * 32 + l32;
          *(v4f *)&red[cc * kRedPitch + rr] =
              v4f{acc[tm][tn][4 * q], acc[tm][tn][4 * q + 1], acc[tm][tn][4 * q + 2],
                  acc[tm][tn][4 * q + 3]};
        }
  }
  barrier();
  if (kg == 0) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    const bool vec = (g.ldy & 3) == 0 && ((uintptr_t)g.y & 15) == 0 && col0 + BN <= g.N;
    const int j = l32 & 3;
#pragma unroll
    for (int tm = 0; tm < 2; ++tm)
#pragma unroll
      for (int tn = 0; tn < 4; ++tn)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int rr = wr * 64 + tm * 32 + 8 * q + 4 * lh, cc = tn * 32 + l32;
          const v4f o = *(const v4f *)&red[cc * kRedPitch + rr];
          v4f s = v4f{acc[tm][tn][4 * q] + o[0], acc[tm][tn][4 * q + 1] + o[1],
                      acc[tm][tn][4 * q + 2] + o[2], acc[tm][tn][4 * q + 3] + o[3]};
          // lane (quad k, j) now: row rr + j, columns (cc & ~3) .. + 3
          s = quad_transpose(s, j);
          const int64_t row = row0 + rr + j, col = col0 + (cc & ~3);
          if (row >= g.M) continue;
          float *dst = g.y + row * g.ldy + col;
          if (vec) {
            __builtin_nontemporal_store(s, (v4f *)dst);
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c)
              if (col + c < g.N) dst[c] = s[c];
          }
        }
  }
}

}  // namespace

hipError_t launch_gemm_prefill(const GemmArgs &a, hipStream_t stream) {
  const int mtiles = (int)((a.M + BM - 1) / BM), ntiles = (int)((a.N + BN - 1) / BN);
  // Split the tile grid into 8 blocks (one per XCD) along rows x columns,
  // minimising the bytes each XCD reads: an activation tile (256 rows) weighs
  // about twice a weight tile (128 columns).
  int gm = 0, gn = 0, best = 0;
  for (int m = 1; m <= 8; m *= 2) {
    const int n = 8 / m;
    if (mtiles % m || ntiles % n) continue;
    const int cost = 2 * (mtiles / m) + ntiles / n;
    if (gm == 0 || cost < best) gm = m, gn = n, best = cost;
  }
  if (a.full)
    hipLaunchKernelGGL(gemm_prefill_kernel<true>, dim3((unsigned)(mtiles * ntiles)), dim3(NT), 0,
                       stream, a, mtiles, ntiles, gm, gn);
  else
    hipLaunchKernelGGL(gemm_prefill_kernel<false>, dim3((unsigned)(mtiles * ntiles)), dim3(NT), 0,
                       stream, a, mtiles, ntiles, gm, gn);
  return hipGetLastError();
}

}  // namespace mxq
