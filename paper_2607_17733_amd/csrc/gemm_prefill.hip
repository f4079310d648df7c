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
// Tiling: 256x128 outputs per workgroup of eight waves in two K groups.
// Group g (waves 4g..4g+3) takes the steps s with s % 2 == g; within a group
// wave r computes rows 64r..64r+63 x all 128 columns = 2x4 tiles of 32x32
// with fp32 accumulators.  Two waves per SIMD (one of each group) keep the
// matrix core busy while the other waits on memory or LDS; at the end the
// groups' partial sums meet in LDS (fixed order: even steps + odd steps).
//   - A: each lane loads its rows' 48-byte step data straight from the
//     activation operand image (32-row tiles: every load of the wave reads
//     one contiguous kilobyte) into registers, one own step ahead.
//   - W: each group loads its next step's 13 KB chunk of the weight operand
//     image (already in the LDS layout) into registers, stores it to LDS one
//     iteration later (double buffer per group), and its lanes read it with
//     16-byte reads.
// Workgroup ids are remapped so that each XCD works on a contiguous range of
// column tiles: its share of the weights stays in its L2.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef unsigned u12 __attribute__((ext_vector_type(12)));   // one lane's 48 bytes

constexpr int BM = 256, BN = kOpCols, NT = 512;
constexpr int kChunkVec = kOpChunk / 16;     // 16-byte pieces per chunk (832)
constexpr int kFmtFp8 = 0, kFmtFp6 = 3;      // e4m3, e3m2
constexpr int kSmemVec = BM * BN * 4 / 16;   // 128 KB: the end reduction (W buffers alias it)

template <int S> struct Seg { static constexpr int v = S; };

__device__ inline u12 cat3(u4 a, u4 b, u4 c) {
  return __builtin_shufflevector(__builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7),
                                 __builtin_shufflevector(c, c, 0, 1, 2, 3, -1, -1, -1, -1),
                                 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11);
}
// Operand registers of one instruction out of a lane's 48 bytes:
// bytes 0-23 / 24-47 (FP6), 0-31 / 16-47 (FP8).
__device__ inline v8i fp6_lo(u12 x) { return (v8i)__builtin_shufflevector(x, x, 0, 1, 2, 3, 4, 5, -1, -1); }
__device__ inline v8i fp6_hi(u12 x) { return (v8i)__builtin_shufflevector(x, x, 6, 7, 8, 9, 10, 11, -1, -1); }
__device__ inline v8i fp8_lo(u12 x) { return (v8i)__builtin_shufflevector(x, x, 0, 1, 2, 3, 4, 5, 6, 7); }
__device__ inline v8i fp8_hi(u12 x) { return (v8i)__builtin_shufflevector(x, x, 4, 5, 6, 7, 8, 9, 10, 11); }

template <int FA, int SA, int SB>
__device__ inline v16f mma(const v8i &a, const v8i &b, v16f c, int sa, int sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, FA, FA, SA, sa, SB, sb);
}

__global__ __launch_bounds__(NT, 1) void gemm_prefill_kernel(GemmArgs g, int mtiles,
                                                             int ntiles) {
  __shared__ __attribute__((aligned(16))) u4 smem[kSmemVec];
  // W chunks during the K loop: [buffer][group][chunk]
  u4 (*Wl)[2][kChunkVec] = (u4 (*)[2][kChunkVec])smem;

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);     // wave-uniform
  const int kg = wave >> 2, rw = wave & 3, tg = t & 255;   // K group, row block, thread in group
  const int l32 = lane & 31, lh = lane >> 5;
  int mt, nt;
  {
    const int pid = blockIdx.x;
    if ((ntiles & 7) == 0) {               // XCD x: column tiles [x*nx, (x+1)*nx)
      const int nx = ntiles >> 3, x = pid & 7, loc = pid >> 3;
      nt = x * nx + loc % nx;
      mt = loc / nx;
    } else {
      mt = pid / ntiles;
      nt = pid - mt * ntiles;
    }
  }
  const int64_t row0 = (int64_t)mt * BM, col0 = (int64_t)nt * BN;
  const OpGeo og(g.n4, g.n6, g.n8);
  const int nsteps = og.nsteps;
  const int niter = (nsteps + 1) >> 1;     // iterations; group 1's last may be empty

  // This wave's two 32-row tiles of the activation operand image (tiles past
  // the last one read the last tile; those rows are never stored).  Lane
  // (h, r) reads its 16-byte pieces at part * 1024 + h * 512 + r * 16.
  const int64_t last = (g.M - 1) / kActRows;
  const int64_t ta = min((row0 + rw * 64) / kActRows, last);
  const int64_t tb = min((row0 + rw * 64) / kActRows + 1, last);
  const uint8_t *aop0 = g.a_mant + g.a_op + ta * nsteps * kActStep + lh * 512 + l32 * 16;
  const uint8_t *aop1 = g.a_mant + g.a_op + tb * nsteps * kActStep + lh * 512 + l32 * 16;
  const uint8_t *asc0 = g.a_exp + g.a_sc + ta * nsteps * kActScaleStep + lh * 128 + l32 * 4;
  const uint8_t *asc1 = g.a_exp + g.a_sc + tb * nsteps * kActScaleStep + lh * 128 + l32 * 4;
  const uint8_t *wtile = g.w_mant + g.w_op + (int64_t)nt * g.w_tile;

  v16f acc[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[a][n] = v16f{};

  // Per wave: W staging (one chunk piece set), A lane data and scales in a
  // ring of two, indexed by the iteration's position relative to the start
  // of the current segment.
  u4 ws[4];
  u12 xa[2][2];
  uint32_t xs[2][2];

  // The group's own step of iteration i (clamped: past the end it refetches
  // the last step, which is not multiplied).
  auto own = [&](int i) __attribute__((always_inline)) { return min(2 * i + kg, nsteps - 1); };
  auto load_w = [&](int st) __attribute__((always_inline)) {
    const u4 *src = (const u4 *)(wtile + (int64_t)st * kOpChunk);
#pragma unroll
    for (int j = 0; j < 3; ++j) ws[j] = src[j * 256 + tg];
    if (tg < 64) ws[3] = src[768 + tg];
  };
  auto store_w = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 3; ++j) Wl[buf][kg][j * 256 + tg] = ws[j];
    if (tg < 64) Wl[buf][kg][768 + tg] = ws[3];
  };
  auto load_a = [&](int st, u12 (&x)[2], uint32_t (&s)[2]) __attribute__((always_inline)) {
    const u4 *p0 = (const u4 *)(aop0 + (int64_t)st * kActStep);
    const u4 *p1 = (const u4 *)(aop1 + (int64_t)st * kActStep);
    x[0] = cat3(p0[0], p0[64], p0[128]);
    x[1] = cat3(p1[0], p1[64], p1[128]);
    s[0] = *(const uint32_t *)(asc0 + (int64_t)st * kActScaleStep);
    s[1] = *(const uint32_t *)(asc1 + (int64_t)st * kActScaleStep);
  };
  // One column tile of the step's instructions (both row tiles).
  auto mul_tile = [&](auto seg, const u12 (&x)[2], const uint32_t (&s)[2], u12 w, int sw,
                      int tn) __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v;
    constexpr int NK = SEG == 1 ? 4 : 2;
#pragma unroll
    for (int k = 0; k < NK; ++k)
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) {
        const int sa = (int)s[tm];
        v16f &c = acc[tm][tn];
        if (SEG == 0) {          // block pairs (4s', 4s'+1), (4s'+2, 4s'+3): scale bytes 0, 1
          if (k == 0) c = mma<kFmtFp6, 0, 0>(fp6_lo(x[tm]), fp6_lo(w), c, sa, sw);
          else c = mma<kFmtFp6, 1, 1>(fp6_hi(x[tm]), fp6_hi(w), c, sa, sw);
        } else if (SEG == 1) {   // digit products hh, ll, hl, lh
          const v8i av = (k == 0 || k == 2) ? fp6_lo(x[tm]) : fp6_hi(x[tm]);
          const v8i wv = (k == 0 || k == 3) ? fp6_lo(w) : fp6_hi(w);
          c = mma<kFmtFp6, 0, 0>(av, wv, c, sa, sw);
        } else {                 // [h|l].[h|l], [h|l].[l|h]
          c = mma<kFmtFp8, 0, 0>(fp8_lo(x[tm]), k == 0 ? fp8_lo(w) : fp8_hi(w), c, sa, sw);
        }
      }
  };
  auto compute = [&](auto seg, const u12 (&x)[2], const uint32_t (&s)[2], int buf)
      __attribute__((always_inline)) {
    const u4 *W = Wl[buf][kg];
    const uint32_t *scl = (const uint32_t *)&W[768];
#pragma unroll
    for (int tn = 0; tn < 4; ++tn) {
      const int c = tn * 32 + l32;
      const u12 w = cat3(W[lh * 128 + c], W[256 + lh * 128 + c], W[512 + lh * 128 + c]);
      mul_tile(seg, x, s, w, (int)scl[lh * 128 + c], tn);
      // one column tile's operands live at a time (the other wave on the
      // SIMD covers the LDS latency)
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Iteration i: the group's chunk of step own(i) is in Wl[i & 1][kg] and
  // its A data in xc; stage the chunk of own(i+1) into Wl[(i+1) & 1][kg],
  // fetch the chunk of own(i+2) and the A data of own(i+1); multiply own(i)
  // unless it lies past the last step.  Group 0 fetches first and group 1
  // multiplies first, so that after each barrier one group streams memory
  // while the other keeps the matrix cores busy.
  auto iteration = [&](auto seg, int i, const u12 (&xc)[2], const uint32_t (&sc)[2],
                       u12 (&xn)[2], uint32_t (&sn)[2]) __attribute__((always_inline)) {
    __syncthreads();
    const bool mul = 2 * i + kg < nsteps;
    if (kg == 1 && mul) compute(seg, xc, sc, i & 1);
    store_w((i + 1) & 1);
    load_w(own(i + 2));
    load_a(own(i + 1), xn, sn);
    if (kg == 0 && mul) compute(seg, xc, sc, i & 1);
  };
  // Iterations [ib, ie) whose own steps lie in one segment; ring slots
  // relative to ib.
  auto run = [&](auto seg, int ib, int ie) __attribute__((always_inline)) {
    for (int i = ib; i < ie; i += 2) {
      iteration(seg, i, xa[0], xs[0], xa[1], xs[1]);
      if (i + 1 < ie) iteration(seg, i + 1, xa[1], xs[1], xa[0], xs[0]);
    }
  };
  // After n iterations the next iteration's A data sits in slot n % 2.
  auto realign = [&](int n) __attribute__((always_inline)) {
    if (n & 1) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const u12 tx = xa[0][j];
        xa[0][j] = xa[1][j];
        xa[1][j] = tx;
        const uint32_t tsc = xs[0][j];
        xs[0][j] = xs[1][j];
        xs[1][j] = tsc;
      }
    }
  };

  // Prologue: the group's chunk of own(0) in LDS, own(1)'s in the staging
  // registers, A of own(0).
  load_w(own(0));
  load_a(own(0), xa[0], xs[0]);
  store_w(0);
  load_w(own(1));

  // Iteration ranges of the group's own steps per segment: own step 2i+kg
  // is in segment 0 while 2i+kg < e4, and so on.
  const int e4 = og.s4, e6 = og.s4 + og.s6;
  const int i4 = (e4 - kg + 1) / 2, i6 = max(i4, (e6 - kg + 1) / 2);
  run(Seg<0>{}, 0, i4);
  realign(i4);
  run(Seg<1>{}, i4, i6);
  realign(i6 - i4);
  run(Seg<2>{}, i6, niter);

  // Sum the two groups: group g finishes row tile tm = g of its row block;
  // each wave hands its other row tile to the partner wave through LDS.
  __syncthreads();
  float *red = (float *)smem;              // [row block][tm][tn][r][lane]
  auto finish = [&](auto mine_tag) __attribute__((always_inline)) {
    constexpr int MINE = decltype(mine_tag)::v, OTHER = 1 - MINE;
#pragma unroll
    for (int tn = 0; tn < 4; ++tn)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        red[(((rw * 2 + OTHER) * 4 + tn) * 16 + r) * 64 + lane] = acc[OTHER][tn][r];
    __syncthreads();
#pragma unroll
    for (int tn = 0; tn < 4; ++tn) {
      const int64_t j = col0 + tn * 32 + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float v = acc[MINE][tn][r] + red[(((rw * 2 + MINE) * 4 + tn) * 16 + r) * 64 + lane];
        const int64_t i = row0 + rw * 64 + MINE * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (i < g.M && j < g.N) g.y[i * g.ldy + j] = v;
      }
    }
  };
  if (kg == 0) finish(Seg<0>{});
  else finish(Seg<1>{});
}

}  // namespace

hipError_t launch_gemm_prefill(const GemmArgs &a, hipStream_t stream) {
  const int mtiles = (int)((a.M + BM - 1) / BM), ntiles = (int)((a.N + BN - 1) / BN);
  hipLaunchKernelGGL(gemm_prefill_kernel, dim3((unsigned)(mtiles * ntiles)), dim3(NT), 0,
                     stream, a, mtiles, ntiles);
  return hipGetLastError();
}

}  // namespace mxq
