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
// Tiling: 256x128 outputs per workgroup of four waves (one per SIMD), each
// wave 64 rows x 128 columns = 2x4 tiles of 32x32 with fp32 accumulators.
//   - A: each lane loads its rows' 48-byte step data straight from the
//     activation operand image (32-row tiles: every load of the wave reads
//     one contiguous kilobyte) into registers, two steps ahead.
//   - W: the step's 13 KB chunk of the weight operand image (already in the
//     LDS layout) is loaded to registers three steps ahead, stored to LDS one
//     step ahead (double buffer), and read by the lanes with 16-byte reads.
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

constexpr int BM = 256, BN = kOpCols, NT = 256;
constexpr int kChunkVec = kOpChunk / 16;     // 16-byte pieces per chunk (832)
constexpr int kFmtFp8 = 0, kFmtFp6 = 3;      // e4m3, e3m2

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
  __shared__ __attribute__((aligned(16))) u4 Wl[2][kChunkVec];

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
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

  // This wave's two 32-row tiles of the activation operand image (tiles past
  // the last one read the last tile; those rows are never stored).  Lane
  // (h, r) reads its 16-byte pieces at part * 1024 + h * 512 + r * 16.
  const int64_t last = (g.M - 1) / kActRows;
  const int64_t ta = min((row0 + wave * 64) / kActRows, last);
  const int64_t tb = min((row0 + wave * 64) / kActRows + 1, last);
  const uint8_t *aop0 = g.a_mant + g.a_op + ta * nsteps * kActStep + lh * 512 + l32 * 16;
  const uint8_t *aop1 = g.a_mant + g.a_op + tb * nsteps * kActStep + lh * 512 + l32 * 16;
  const uint8_t *asc0 = g.a_exp + g.a_sc + ta * nsteps * kActScaleStep + lh * 64 + l32 * 2;
  const uint8_t *asc1 = g.a_exp + g.a_sc + tb * nsteps * kActScaleStep + lh * 64 + l32 * 2;
  const uint8_t *wtile = g.w_mant + g.w_op + (int64_t)nt * g.w_tile;

  v16f acc[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[a][n] = v16f{};

  // Register rings, indexed by the step's position relative to the start of
  // the current segment: W staging (2 slots), A lane data and scales (3).
  u4 ws[2][4];
  u12 xa[3][2];
  uint32_t xs[3][2];

  auto load_w = [&](int st, u4 (&w)[4]) __attribute__((always_inline)) {
    const u4 *src = (const u4 *)(wtile + (int64_t)st * kOpChunk);
#pragma unroll
    for (int j = 0; j < 3; ++j) w[j] = src[j * 256 + t];
    if (t < 64) w[3] = src[768 + t];
  };
  auto store_w = [&](const u4 (&w)[4], int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 3; ++j) Wl[buf][j * 256 + t] = w[j];
    if (t < 64) Wl[buf][768 + t] = w[3];
  };
  // A lane data (48 bytes: three contiguous kilobytes per wave) and scales.
  auto load_a = [&](int st, u12 (&x)[2], uint32_t (&s)[2]) __attribute__((always_inline)) {
    const u4 *p0 = (const u4 *)(aop0 + (int64_t)st * kActStep);
    const u4 *p1 = (const u4 *)(aop1 + (int64_t)st * kActStep);
    x[0] = cat3(p0[0], p0[64], p0[128]);
    x[1] = cat3(p1[0], p1[64], p1[128]);
    s[0] = *(const uint16_t *)(asc0 + (int64_t)st * kActScaleStep);
    s[1] = *(const uint16_t *)(asc1 + (int64_t)st * kActScaleStep);
  };
  auto compute = [&](auto seg, const u12 (&x)[2], const uint32_t (&s)[2], int buf)
      __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v;
    const uint32_t *scl = (const uint32_t *)&Wl[buf][768];
#pragma unroll
    for (int tn = 0; tn < 4; ++tn) {
      const int c = tn * 32 + l32;
      const u12 w = cat3(Wl[buf][lh * 128 + c], Wl[buf][256 + lh * 128 + c],
                         Wl[buf][512 + lh * 128 + c]);
      const int sw = (int)scl[lh * 128 + c];
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) {
        const int sa = (int)s[tm];
        if (SEG == 0) {            // two block pairs, scale bytes 0 and 1
          acc[tm][tn] = mma<kFmtFp6, 0, 0>(fp6_lo(x[tm]), fp6_lo(w), acc[tm][tn], sa, sw);
          acc[tm][tn] = mma<kFmtFp6, 1, 1>(fp6_hi(x[tm]), fp6_hi(w), acc[tm][tn], sa, sw);
        } else if (SEG == 1) {     // digit products hh, ll, hl, lh
          acc[tm][tn] = mma<kFmtFp6, 0, 0>(fp6_lo(x[tm]), fp6_lo(w), acc[tm][tn], sa, sw);
          acc[tm][tn] = mma<kFmtFp6, 0, 0>(fp6_hi(x[tm]), fp6_hi(w), acc[tm][tn], sa, sw);
          acc[tm][tn] = mma<kFmtFp6, 0, 0>(fp6_lo(x[tm]), fp6_hi(w), acc[tm][tn], sa, sw);
          acc[tm][tn] = mma<kFmtFp6, 0, 0>(fp6_hi(x[tm]), fp6_lo(w), acc[tm][tn], sa, sw);
        } else {                   // [h|l].[h|l] and [h|l].[l|h]
          acc[tm][tn] = mma<kFmtFp8, 0, 0>(fp8_lo(x[tm]), fp8_lo(w), acc[tm][tn], sa, sw);
          acc[tm][tn] = mma<kFmtFp8, 0, 0>(fp8_lo(x[tm]), fp8_hi(w), acc[tm][tn], sa, sw);
        }
      }
    }
  };

  // Step st: W chunk st in Wl[st&1]; stage st+1 into the other buffer and
  // fetch st+3; fetch A of st+2; multiply step st.
  auto iteration = [&](auto seg, int st, u4 (&wst)[4], const u12 (&xc)[2],
                       const uint32_t (&sc)[2], u12 (&xn)[2], uint32_t (&sn)[2])
      __attribute__((always_inline)) {
    __syncthreads();
    // Unconditional (clamped) so that every path issues the same memory
    // operations: past the end they refetch the last step, which is unused.
    store_w(wst, (st + 1) & 1);
    load_w(min(st + 3, nsteps - 1), wst);
    load_a(min(st + 2, nsteps - 1), xn, sn);
    // keep the prefetches here: the compiler may not sink them to their uses
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    compute(seg, xc, sc, st & 1);
  };
  // Steps [begin, end) of one segment, six per trip so that the ring slots
  // are compile-time registers (relative to begin).  Every iteration issues
  // the same memory operations whatever the branches, which keeps the
  // compiler's memory-counter waits tight.
  auto run = [&](auto seg, int begin, int end) __attribute__((always_inline)) {
    for (int st = begin; st < end; st += 6) {
      iteration(seg, st, ws[1], xa[0], xs[0], xa[2], xs[2]);
      if (st + 1 < end) iteration(seg, st + 1, ws[0], xa[1], xs[1], xa[0], xs[0]);
      if (st + 2 < end) iteration(seg, st + 2, ws[1], xa[2], xs[2], xa[1], xs[1]);
      if (st + 3 < end) iteration(seg, st + 3, ws[0], xa[0], xs[0], xa[2], xs[2]);
      if (st + 4 < end) iteration(seg, st + 4, ws[1], xa[1], xs[1], xa[0], xs[0]);
      if (st + 5 < end) iteration(seg, st + 5, ws[0], xa[2], xs[2], xa[1], xs[1]);
    }
  };
  // After a segment of n steps, step st sits in slot (st - begin) % 3 (A) and
  // (st - begin) % 2 (W); the next segment numbers it st - end: rotate.
  auto realign = [&](int n) __attribute__((always_inline)) {
    const int ra3 = n % 3;
    if (ra3 == 1) {                        // new slot k <- old slot (k + 1) % 3
      const u12 t0 = xa[0][0], t1 = xa[0][1];
      const uint32_t s0 = xs[0][0], s1 = xs[0][1];
      xa[0][0] = xa[1][0]; xa[0][1] = xa[1][1]; xs[0][0] = xs[1][0]; xs[0][1] = xs[1][1];
      xa[1][0] = xa[2][0]; xa[1][1] = xa[2][1]; xs[1][0] = xs[2][0]; xs[1][1] = xs[2][1];
      xa[2][0] = t0; xa[2][1] = t1; xs[2][0] = s0; xs[2][1] = s1;
    } else if (ra3 == 2) {                 // new slot k <- old slot (k + 2) % 3
      const u12 t0 = xa[2][0], t1 = xa[2][1];
      const uint32_t s0 = xs[2][0], s1 = xs[2][1];
      xa[2][0] = xa[1][0]; xa[2][1] = xa[1][1]; xs[2][0] = xs[1][0]; xs[2][1] = xs[1][1];
      xa[1][0] = xa[0][0]; xa[1][1] = xa[0][1]; xs[1][0] = xs[0][0]; xs[1][1] = xs[0][1];
      xa[0][0] = t0; xa[0][1] = t1; xs[0][0] = s0; xs[0][1] = s1;
    }
    if (n & 1) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const u4 tw = ws[0][j];
        ws[0][j] = ws[1][j];
        ws[1][j] = tw;
      }
    }
  };

  // Prologue: W chunks of steps 0, 1, 2 in flight, step 0 in LDS; A of 0, 1.
  load_w(0, ws[0]);
  if (nsteps > 1) load_w(1, ws[1]);
  load_a(0, xa[0], xs[0]);
  if (nsteps > 1) load_a(1, xa[1], xs[1]);
  store_w(ws[0], 0);
  if (nsteps > 2) load_w(2, ws[0]);

  const int e4 = og.s4, e6 = og.s4 + og.s6;
  run(Seg<0>{}, 0, e4);
  realign(e4);
  run(Seg<1>{}, e4, e6);
  realign(e6 - e4);
  run(Seg<2>{}, e6, nsteps);

#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int tn = 0; tn < 4; ++tn) {
      const int64_t j = col0 + tn * 32 + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t i = row0 + wave * 64 + tm * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (i < g.M && j < g.N) g.y[i * g.ldy + j] = acc[tm][tn][r];
      }
    }
}

}  // namespace

hipError_t launch_gemm_prefill(const GemmArgs &a, hipStream_t stream) {
  const int mtiles = (int)((a.M + BM - 1) / BM), ntiles = (int)((a.N + BN - 1) / BN);
  hipLaunchKernelGGL(gemm_prefill_kernel, dim3((unsigned)(mtiles * ntiles)), dim3(NT), 0,
                     stream, a, mtiles, ntiles);
  return hipGetLastError();
}

}  // namespace mxq
