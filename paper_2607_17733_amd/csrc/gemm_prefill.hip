// gemm_prefill.hip -- MXINT GEMM for prefill shapes on the block-scaled
// matrix cores of gfx950.
//
// Y[i][j] = sum_b sum_k qa[i][k] qw[j][k] 2^(Ea[i][b] + Ew[j][b] - 254 - 2(m_b - 2))
// (MXSens, arXiv 2607.17733, Section 2: integer mantissas with one
// power-of-two scale per 32-element block; Section 6: mixed widths in one
// GEMM).
//
// Both operands arrive as matrix-core operand images (OpGeo in mxq_device.h):
// every MXINT mantissa is one or two exactly representable FP6/FP8 digits and
// every block's E8M0 scale byte is its shared exponent, so
// V_MFMA_SCALE_F32_32X32X64_F8F6F4 applies the block scales itself and
// accumulates straight into fp32.  Per K step:
//   4-bit (4 blocks): two FP6 instructions (block pairs), scale bytes 0 / 1;
//   6-bit (2 blocks): four FP6 instructions, the digit products hh, ll, hl, lh;
//   8-bit (1 block):  two FP8 instructions, [h|l].[h|l] and [h|l].[l|h].
// The digit products are exact; only the fp32 accumulation rounds.
//
// Tiling: 256x128 outputs per workgroup of eight waves, two per SIMD; wave
// (r, c) owns rows 64r..64r+63 x columns 64c..64c+63 = 2x2 tiles of 32x32
// fp32 accumulators and runs every K step.
//
// Data path: each step's operands -- the eight 32-row activation blocks,
// their scale blocks and the weight chunk, already in the layout the lanes
// read -- are copied global -> LDS by the buffer unit's direct-to-LDS loads
// (no registers), five 1 KB loads per wave and step, into a ring of four LDS
// stages.  Loads run four steps ahead of the products and the operands of a
// step are read from LDS into registers one step ahead, so neither latency
// meets a matrix instruction.  A step waits for the wave's loads of the next
// stage and its reads of the current one, meets the other waves at a
// barrier (after which the next stage is complete and the current one is
// free), then spreads the loads of step + 4 into the freed stage and the
// reads of step + 1 between its products.  Two waves per SIMD keep the
// matrix core busy while one of them waits at the barrier.
// Workgroup ids are remapped so that each XCD owns a compact block of output
// tiles: the activation rows and weight columns it reads stay in its L2.
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

constexpr int BM = 256, BN = kOpCols, NT = 512;
constexpr int kFmtFp8 = 0, kFmtFp6 = 3;      // e4m3, e3m2
constexpr int kStages = 4;                   // LDS ring; loads run kStages - 1 steps ahead
// One stage: the eight activation tile blocks (3 KB each), their 256-byte
// scale blocks, then the 13 KB weight chunk.
constexpr int kStA = 0;
constexpr int kStAScale = kStA + 8 * kActStep;              // 24576
constexpr int kStW = kStAScale + 8 * kActScaleStep;         // 26624
constexpr int kStage = kStW + kOpChunk;                     // 39936
static_assert(kStage % 16 == 0 && kStages * kStage <= 160 * 1024, "LDS ring");
// A step's 39 loads of 1 KB (24 activation, 2 activation scale, 13 weight),
// plus one repeat of the last, as five per wave.
constexpr int kDmaPerStep = 5;

template <int S> struct Int { static constexpr int v = S; };

// A lane's 48 bytes of one step, as three 16-byte pieces (one LDS read
// each).  FP6 operands are bytes 0-23 and 24-47 and FP8 operands 0-31 and
// 16-47, so the middle piece is split or shared; the register copies that
// needs are cheaper than more, narrower LDS reads, which cost the same per
// instruction.
struct Lane48 {
  u4 p[3];
};
__device__ inline v8i fp6_lo(const Lane48 &x) {
  return (v8i)__builtin_shufflevector(x.p[0], x.p[1], 0, 1, 2, 3, 4, 5, -1, -1);
}
__device__ inline v8i fp6_hi(const Lane48 &x) {
  return (v8i)__builtin_shufflevector(x.p[1], x.p[2], 2, 3, 4, 5, 6, 7, -1, -1);
}
__device__ inline v8i fp8_lo(const Lane48 &x) {
  return (v8i)__builtin_shufflevector(x.p[0], x.p[1], 0, 1, 2, 3, 4, 5, 6, 7);
}
__device__ inline v8i fp8_hi(const Lane48 &x) {
  return (v8i)__builtin_shufflevector(x.p[1], x.p[2], 0, 1, 2, 3, 4, 5, 6, 7);
}

template <int FA, int SA, int SB>
__device__ inline v16f mma(const v8i &a, const v8i &b, v16f c, int sa, int sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, FA, FA, SA, sa, SB, sb);
}

// The LDS ring's synchronisation is explicit: the compiler neither knows
// which direct-to-LDS load fills which stage nor may move LDS reads across
// these points.
template <int N>
__device__ inline void wait_loads() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// ... and also until this wave's LDS reads have completed.
template <int N>
__device__ inline void wait_loads_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(N) : "memory");
}
__device__ inline void barrier() { asm volatile("s_barrier" ::: "memory"); }

__global__ __launch_bounds__(NT, 1) void gemm_prefill_kernel(GemmArgs g, int mtiles, int ntiles,
                                                             int gm, int gn) {
  __shared__ __attribute__((aligned(16))) u4 lds[kStages * kStage / 16];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);      // wave-uniform
  const int l32 = lane & 31, lh = lane >> 5;
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
  const OpGeo og(g.n4, g.n6, g.n8);
  const int nsteps = og.nsteps;

  // Wave (r, c): row block r (two 32-row tiles), column half c.
  const int wr = wave >> 1, wc = wave & 1;
  // The workgroup's eight 32-row tiles of the activation operand image
  // (tiles past the last one load the last tile; those rows are never
  // stored).
  const int last = (int)((g.M - 1) / kActRows);
  const int tile0 = (int)(row0 / kActRows);
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.a_mant + g.a_op), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.a_exp + g.a_sc), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.w_mant + g.w_op + (int64_t)nt * g.w_tile), 0, 0x7fffffff, 0x00020000);
  const int v16 = lane * 16;
  char *const ring = (char *)lds;
  auto tile_of = [&](int t) { return min(tile0 + t, last); };
  // Scale gathers: lane l reads bytes (l % 16) * 16 .. +15 of the scale block
  // of tile 4 h + l / 16 (h = 0, 1), whose step st block starts at
  // (tile * nsteps + st) * 256; the per-lane part of that offset is fixed.
  int vsc[2];
#pragma unroll
  for (int h = 0; h < 2; ++h)
    vsc[h] = tile_of(4 * h + (lane >> 4)) * nsteps * kActScaleStep + (lane & 15) * 16;

  // The step's loads are numbered 0..39: 0..23 activation tile n / 3,
  // kilobyte n % 3; 24, 25 the scale blocks of tiles 4 (n - 24) .. +3;
  // 26..38 weight kilobyte n - 26 (the last one the scale dwords); 39 repeats
  // 38.  Wave w issues loads w + 8 j, j = 0..4; their descriptors are fixed
  // but for the step offset (soff + st * sstep).
  struct Load {
    __amdgpu_buffer_rsrc_t rsrc;
    int lds, voff, soff, sstep;
  } ld[kDmaPerStep];
#pragma unroll
  for (int j = 0; j < kDmaPerStep; ++j) {
    const int n = wave + 8 * j;
    if (n < 24) {
      const int t = n / 3, kb = n % 3;
      ld[j] = {ra, kStA + t * kActStep + kb * 1024, v16, tile_of(t) * nsteps * kActStep + kb * 1024,
               kActStep};
    } else if (n < 26) {
      const int h = n - 24;
      ld[j] = {rs, kStAScale + 4 * h * kActScaleStep, vsc[h], 0, kActScaleStep};
    } else {
      const int kb = min(n - 26, 12);
      ld[j] = {rw, kStW + kb * 1024, v16, kb * 1024, kOpChunk};
    }
  }
  // This wave's load j (0..4) of step st into stage q.
  auto issue = [&](int st, int q, int j) __attribute__((always_inline)) {
    st = min(st, nsteps - 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ld[j].rsrc, (lds_void *)(ring + q * kStage + ld[j].lds),
                                             16, ld[j].voff, ld[j].soff + st * ld[j].sstep, 0, 0);
  };

  v16f acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int n = 0; n < 2; ++n) acc[a][n] = v16f{};

  // All operands of one step in registers: the wave's two activation tiles
  // and the four weight column tiles.
  struct Ops {
    Lane48 x[2], w[2];
    uint32_t sa[2], sw[2];
  } ops[2];

  // Read the operands of step st (stage st % 4) into ops[O]: the activation
  // tiles, and weight column tile tn.
  auto read_x = [&](auto o_tag, int st) __attribute__((always_inline)) {
    constexpr int O = decltype(o_tag)::v;
    const char *stage = ring + (st & 3) * kStage;
    Ops &d = ops[O];
#pragma unroll
    for (int tm = 0; tm < 2; ++tm) {
      const u4 *blk = (const u4 *)(stage + kStA + (wr * 2 + tm) * kActStep);   // 64 lanes
#pragma unroll
      for (int j = 0; j < 3; ++j) d.x[tm].p[j] = blk[j * 64 + lane];
      d.sa[tm] = ((const uint32_t *)(stage + kStAScale))[(wr * 2 + tm) * 64 + lane];
    }
  };
  auto read_w = [&](auto o_tag, int st, int tn) __attribute__((always_inline)) {
    constexpr int O = decltype(o_tag)::v;
    const char *W = ring + (st & 3) * kStage + kStW;                  // 256 lanes
    Ops &d = ops[O];
    const int L = lh * 128 + wc * 64 + tn * 32 + l32;
#pragma unroll
    for (int j = 0; j < 3; ++j) d.w[tn].p[j] = ((const u4 *)W)[j * 256 + L];
    d.sw[tn] = ((const uint32_t *)(W + 3 * kOpPart))[L];
  };
  // The products of column tile tn (both row tiles) of one step from ops[O].
  auto mul_tile = [&](auto seg, auto o_tag, int tn) __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v, O = decltype(o_tag)::v;
    constexpr int NK = SEG == 1 ? 4 : 2;
    const Ops &d = ops[O];
#pragma unroll
    for (int k = 0; k < NK; ++k)
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) {
        v16f &c = acc[tm][tn];
        const Lane48 &x = d.x[tm], &w = d.w[tn];
        const int as = (int)d.sa[tm], ws = (int)d.sw[tn];
        if (SEG == 0) {          // block pairs (4s', 4s'+1), (4s'+2, 4s'+3): scale bytes 0, 1
          if (k == 0) c = mma<kFmtFp6, 0, 0>(fp6_lo(x), fp6_lo(w), c, as, ws);
          else c = mma<kFmtFp6, 1, 1>(fp6_hi(x), fp6_hi(w), c, as, ws);
        } else if (SEG == 1) {   // digit products hh, ll, hl, lh
          const v8i av = (k == 0 || k == 2) ? fp6_lo(x) : fp6_hi(x);
          const v8i wv = (k == 0 || k == 3) ? fp6_lo(w) : fp6_hi(w);
          c = mma<kFmtFp6, 0, 0>(av, wv, c, as, ws);
        } else {                 // [h|l].[h|l], [h|l].[l|h]
          c = mma<kFmtFp8, 0, 0>(fp8_lo(x), k == 0 ? fp8_lo(w) : fp8_hi(w), c, as, ws);
        }
      }
  };

  // Step s multiplies from ops[O] (read during step s - 1).  Before that, the
  // wave waits until its loads of stage s + 1 have landed and its reads of
  // stage s (into ops[O]) have completed; after the barrier every wave is in
  // that state, so stage s + 1 is complete and stage s is free.  Then, between
  // the products, it issues the loads of step s + 4 into stage s % 4 and reads
  // the operands of step s + 1 into ops[1 - O].
  auto step = [&](auto seg, auto o_tag, int s) __attribute__((always_inline)) {
    constexpr int O = decltype(o_tag)::v;
    constexpr Int<1 - O> nx{};
    const int sn = min(s + 1, nsteps - 1);
    wait_loads_lds<2 * kDmaPerStep>();
    barrier();
    // Chunks in a fixed order (the scheduler may interleave within a chunk
    // only): the products of column tile 0 with three of the loads of step
    // s + 4 and the activation reads of step s + 1, then those of column tile
    // 1 with the other two loads and the weight reads.
    issue(s + 4, s & 3, 0);
    issue(s + 4, s & 3, 1);
    issue(s + 4, s & 3, 2);
    read_x(nx, sn);
    mul_tile(seg, o_tag, 0);
    __builtin_amdgcn_sched_barrier(0);
    issue(s + 4, s & 3, 3);
    issue(s + 4, s & 3, 4);
    read_w(nx, sn, 0);
    read_w(nx, sn, 1);
    mul_tile(seg, o_tag, 1);
  };
  // The steps [b, e) of one segment, in pairs so that the operand sets
  // alternate statically; after the last step the next step's operands are
  // in ops[0].
  auto run = [&](auto seg, int b, int e) __attribute__((always_inline)) {
    int s = b;
    for (; s + 2 <= e; s += 2) {
      step(seg, Int<0>{}, s);
      step(seg, Int<1>{}, s + 1);
    }
    if (s < e) {
      step(seg, Int<0>{}, s);
      ops[0] = ops[1];
    }
  };

  // Prologue: the loads of steps 0..3, then the operands of step 0.
#pragma unroll
  for (int st = 0; st < 4; ++st)
#pragma unroll
    for (int j = 0; j < kDmaPerStep; ++j) issue(st, st, j);
  wait_loads_lds<3 * kDmaPerStep>();
  barrier();
  read_x(Int<0>{}, 0);
#pragma unroll
  for (int tn = 0; tn < 2; ++tn) read_w(Int<0>{}, 0, tn);

  const int e4 = og.s4, e6 = og.s4 + og.s6;
  run(Int<0>{}, 0, e4);
  run(Int<1>{}, e4, e6);
  run(Int<2>{}, e6, nsteps);
  // The last steps' loads (of clamped steps) must land before the workgroup
  // releases its LDS.
  wait_loads<0>();

  // Epilogue through LDS: each wave writes its 64 x 64 tile row-major (row
  // pitch 72 floats: the two row groups one instruction writes fall in
  // disjoint banks) and reads it back as 16-byte row pieces, so the stores
  // are 16 bytes per lane -- a quarter of the store instructions, which the
  // address unit issues at a fixed rate per instruction.
  constexpr int kPitch = 72;
  static_assert(8 * 64 * kPitch * 4 <= kStages * kStage, "epilogue tile");
  barrier();                                 // every wave is done with the ring
  float *tile = (float *)ring + wave * 64 * kPitch;
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int tn = 0; tn < 2; ++tn)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        tile[(tm * 32 + 8 * (r >> 2) + 4 * lh + (r & 3)) * kPitch + tn * 32 + l32] = acc[tm][tn][r];
  // only this wave reads its tile back
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  const int q = lane & 15, rq = lane >> 4;   // 4 columns 4q.., row 4 i + rq
  const int64_t jc = col0 + wc * 64 + 4 * q;
  // 16-byte stores when the wave's 64 columns are all inside Y and aligned
  const bool vec = (g.ldy & 3) == 0 && ((uintptr_t)g.y & 15) == 0 &&
                   col0 + wc * 64 + 64 <= g.N;
  if (vec) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int rr = 4 * i + rq;
      const int64_t row = row0 + wr * 64 + rr;
      const v4f v = *(const v4f *)&tile[rr * kPitch + 4 * q];
      if (row < g.M) __builtin_nontemporal_store(v, (v4f *)(g.y + row * g.ldy + jc));
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int rr = 4 * i + rq;
      const int64_t row = row0 + wr * 64 + rr;
      if (row >= g.M) continue;
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (jc + c < g.N) g.y[row * g.ldy + jc + c] = tile[rr * kPitch + 4 * q + c];
    }
  }
}

}  // namespace

hipError_t launch_gemm_prefill(const GemmArgs &a, hipStream_t stream) {
  const int mtiles = (int)((a.M + BM - 1) / BM), ntiles = (int)((a.N + BN - 1) / BN);
  // Split the tile grid into 8 blocks (one per XCD) along rows x columns,
  // minimising the bytes each XCD reads: an activation tile (256 rows) weighs
  // twice a weight tile (128 columns).
  int gm = 0, gn = 0, best = 0;
  for (int m = 1; m <= 8; m *= 2) {
    const int n = 8 / m;
    if (mtiles % m || ntiles % n) continue;
    const int cost = 2 * (mtiles / m) + ntiles / n;
    if (gm == 0 || cost < best) gm = m, gn = n, best = cost;
  }
  hipLaunchKernelGGL(gemm_prefill_kernel, dim3((unsigned)(mtiles * ntiles)), dim3(NT), 0,
                     stream, a, mtiles, ntiles, gm, gn);
  return hipGetLastError();
}

}  // namespace mxq
