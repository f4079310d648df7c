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
// Tiling: 256x128 outputs per workgroup of eight waves in two K groups of
// four, one wave of each group per SIMD.  Group g takes the steps s with
// s % 2 == g; wave (g, r) owns rows 64r..64r+63 x all 128 columns = 2x4 tiles
// of 32x32 fp32 accumulators, and the groups' partial sums meet in LDS at the
// end.
//
// Data path, chosen by what gfx950 charges (measured): an LDS read costs the
// same per instruction whatever its width, direct-to-LDS loads and LDS reads
// serialise, and load instructions issue at a fixed rate per wave.  So:
//   - activations go straight from the row-tiled operand image into
//     registers -- each 32-row block is used by exactly one wave -- one
//     iteration (two steps) ahead, in two register sets;
//   - the weight chunk of each step (13 KB, already in the LDS layout) goes
//     global -> LDS by direct-to-LDS loads into a ring of eight step stages,
//     three iterations ahead; the four waves of a group read it per column
//     tile, one tile ahead of the products.
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
typedef __attribute__((address_space(3))) void lds_void;

constexpr int BM = 256, BN = kOpCols, NT = 512;
constexpr int kFmtFp8 = 0, kFmtFp6 = 3;      // e4m3, e3m2
constexpr int kWStages = 8;                  // weight ring: 4 iterations of 2 steps
constexpr int kRing = kWStages * kOpChunk;   // 106496 bytes
// Reduction of the two groups: [column][row] floats, 256 rows + 4 padding.
constexpr int kRedPitch = 260;
static_assert(kRing <= 160 * 1024 && 128 * kRedPitch * 4 <= 160 * 1024, "LDS");
// Loads per wave and iteration: 4 direct-to-LDS weight loads (the two steps'
// 26 kilobytes and 6 repeats, over 8 waves), then 8 activation loads (two
// 32-row tiles: three 16-byte parts and the scale dword each).
constexpr int kWLoads = 4, kALoads = 8;
// The fewest activation loads a bundle holds: 8-bit steps leave the third
// part unread, so the compiler drops its load.
constexpr int kMinALoads = 6;

template <int S> struct Int { static constexpr int v = S; };

// A lane's 48 bytes of one step, as three 16-byte pieces.  FP6 operands are
// bytes 0-23 and 24-47 and FP8 operands 0-31 and 16-47, so the middle piece
// is split or shared through register copies.
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

// The ring's synchronisation is explicit: the compiler does not know which
// direct-to-LDS load fills which stage, and may not move LDS accesses across
// these points.
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

__global__ __launch_bounds__(NT, 1) void gemm_prefill_kernel(GemmArgs g, int mtiles, int ntiles,
                                                             int gm, int gn) {
  __shared__ __attribute__((aligned(16))) u4 lds[(128 * kRedPitch * 4 > kRing ? 128 * kRedPitch * 4
                                                                               : kRing) / 16];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);      // wave-uniform
  const int l32 = lane & 31, lh = lane >> 5;
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
  const OpGeo og(g.n4, g.n6, g.n8);
  const int nsteps = og.nsteps;
  char *const ring = (char *)lds;

  // This wave's two 32-row tiles (tiles past the last one load the last tile;
  // those rows are never stored).
  // The activation resources start at tile ta (64-bit arithmetic), so the
  // 32-bit buffer offsets stay below 2 * nsteps * kActStep; the host rejects
  // shapes where that exceeds INT32_MAX.
  const int64_t last = (g.M - 1) / kActRows;
  const int64_t ta = min(row0 / kActRows + 2 * wr, last);
  const int dtb = (int)(min(ta + 1, last) - ta);          // 0 or 1: tile tb = ta + dtb
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.a_mant + g.a_op + ta * nsteps * (int64_t)kActStep), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.a_exp + g.a_sc + ta * nsteps * (int64_t)kActScaleStep), 0, 0x7fffffff,
      0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.w_mant + g.w_op + (int64_t)nt * g.w_tile), 0, 0x7fffffff, 0x00020000);
  const int v16 = lane * 16, v4 = lane * 4;

  v16f acc[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[a][n] = v16f{};

  Lane48 xa[2][2];          // activation lane data: register set, row tile
  uint32_t xs[2][2];        // activation scale dwords

  // Weight loads of iteration it (steps 2 it, 2 it + 1) into their stages:
  // kilobytes n = 0..25 (13 per step), 26..31 repeat the last; wave w issues
  // n = w + 8 j.
  auto issue_w = [&](int it) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < kWLoads; ++j) {
      const int n = min(wave + 8 * j, 25);
      const int st = min(2 * it + n / 13, nsteps - 1), kb = n % 13;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rw, (lds_void *)(ring + (st % kWStages) * kOpChunk + kb * 1024), 16, v16,
          st * kOpChunk + kb * 1024, 0, 0);
    }
  };
  // Activation loads of the wave's step in iteration it, row tile tm, into
  // register set S.
  auto issue_a_half = [&](auto set_tag, int it, int tm) __attribute__((always_inline)) {
    constexpr int S = decltype(set_tag)::v;
    const int st = min(2 * it + kg, nsteps - 1);
    const int blk = (tm == 0 ? 0 : dtb) * nsteps + st;
#pragma unroll
    for (int j = 0; j < 3; ++j)
      xa[S][tm].p[j] = __builtin_bit_cast(
          u4, __builtin_amdgcn_raw_buffer_load_b128(ra, v16, blk * kActStep + j * 1024, 0));
    xs[S][tm] = __builtin_amdgcn_raw_buffer_load_b32(rs, v4, blk * kActScaleStep, 0);
  };

  // Weight operands: two column tiles in flight (w), and the scale dwords of
  // the four column tiles of the current step (one 16-byte read).
  Lane48 w[2];
  u4 swc;
  auto read_w = [&](const char *base, int o, int tn) __attribute__((always_inline)) {
    const int L = lh * 128 + tn * 32 + l32;
#pragma unroll
    for (int j = 0; j < 3; ++j) w[o].p[j] = ((const u4 *)base)[j * 256 + L];
  };
  auto read_sw = [&](const char *base) __attribute__((always_inline)) {
    return ((const u4 *)(base + 3 * kOpPart))[lh * 32 + l32];
  };

  // Iteration it: the products of this wave's step s = 2 it + kg from
  // register set S, column tile by column tile, each tile's weight operand
  // read one tile ahead.  Its first tile and the step's scales were read at
  // the end of the previous iteration, so the products start at once.
  //
  // Each iteration issues a bundle of loads, the activations of it + 1 (into
  // the other register set, around tiles 0 and 1) and then the weights of
  // it + 3 (at tile 2), spread over the products so that the matrix core
  // keeps running while they queue.  Between tiles 1 and 2 the workgroup
  // meets at a barrier.  Before it each wave waits for its own weight loads
  // of iteration it + 1 (at least 16 loads have been issued since them:
  // the bundle of it - 1 and the activations of it + 1); after it the stages
  // of it + 1 are complete, so tile 0 of the next step is read during tile 3,
  // and every wave is past iteration it - 1, whose stages the weights of
  // it + 3 then overwrite.
  auto iteration = [&](auto seg, auto set_tag, int it, bool mul) __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v, S = decltype(set_tag)::v;
    constexpr int NK = SEG == 1 ? 4 : 2;
    auto hook = [&](int tn) __attribute__((always_inline)) {
      if (tn == 0) issue_a_half(Int<1 - S>{}, it + 1, 0);
      else if (tn == 1) issue_a_half(Int<1 - S>{}, it + 1, 1);
      else if (tn == 2) issue_w(it + 3);
    };
    auto meet = [&]() __attribute__((always_inline)) {
      wait_loads<kMinALoads + kWLoads + kMinALoads>();
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
    const char *W = ring + (s % kWStages) * kOpChunk;            // 256 lanes
    const char *Wn = ring + ((s + 2) % kWStages) * kOpChunk;     // the next step
    const u4 sw = swc;
#pragma unroll
    for (int tn = 0; tn < 4; ++tn) {
      const int o = tn & 1;
      if (tn == 2) meet();
      if (tn < 3) {
        read_w(W, o ^ 1, tn + 1);
      } else {
        read_w(Wn, o ^ 1, 0);
        swc = read_sw(Wn);
      }
      hook(tn);
#pragma unroll
      for (int k = 0; k < NK; ++k)
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
          v16f &c = acc[tm][tn];
          const Lane48 &x = xa[S][tm];
          const int as = (int)xs[S][tm], ws = (int)sw[tn];
          if (SEG == 0) {          // block pairs (4s', 4s'+1), (4s'+2, 4s'+3): scale bytes 0, 1
            if (k == 0) c = mma<kFmtFp6, 0, 0>(fp6_lo(x), fp6_lo(w[o]), c, as, ws);
            else c = mma<kFmtFp6, 1, 1>(fp6_hi(x), fp6_hi(w[o]), c, as, ws);
          } else if (SEG == 1) {   // digit products hh, ll, hl, lh
            const v8i av = (k == 0 || k == 2) ? fp6_lo(x) : fp6_hi(x);
            const v8i wv = (k == 0 || k == 3) ? fp6_lo(w[o]) : fp6_hi(w[o]);
            c = mma<kFmtFp6, 0, 0>(av, wv, c, as, ws);
          } else {                 // [h|l].[h|l], [h|l].[l|h]
            c = mma<kFmtFp8, 0, 0>(fp8_lo(x), k == 0 ? fp8_lo(w[o]) : fp8_hi(w[o]), c, as, ws);
          }
        }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Iterations [ib, ie) of one segment; register set = it % 2.
  auto run = [&](auto seg, int ib, int ie) __attribute__((always_inline)) {
    int it = ib;
    if (it < ie && (it & 1)) iteration(seg, Int<1>{}, it++, true);
    for (; it + 2 <= ie; it += 2) {
      iteration(seg, Int<0>{}, it, true);
      iteration(seg, Int<1>{}, it + 1, true);
    }
    if (it < ie) iteration(seg, Int<0>{}, it, true);
  };

  // Prologue: weights of iterations 0 and 1, then the bundle of iteration -1
  // (activations of 0, weights of 2).
  issue_w(0);
  issue_w(1);
  __builtin_amdgcn_sched_barrier(0);
  issue_a_half(Int<0>{}, 0, 0);
  issue_a_half(Int<0>{}, 0, 1);
  __builtin_amdgcn_sched_barrier(0);
  issue_w(2);
  __builtin_amdgcn_sched_barrier(0);
  // the stages of iteration 0 (at least 14 loads since the weights of 0)
  wait_loads<kWLoads + kMinALoads + kWLoads>();
  barrier();
  read_w(ring + kg * kOpChunk, 0, 0);
  swc = read_sw(ring + kg * kOpChunk);

  // Group g's steps 2 it + g of segment [b, e) are the iterations
  // [(b - g + 1) / 2, (e - g + 1) / 2).
  const int e4 = og.s4, e6 = og.s4 + og.s6;
  const int i4 = (e4 - kg + 1) >> 1, i6 = (e6 - kg + 1) >> 1, i8 = (nsteps - kg + 1) >> 1;
  run(Int<0>{}, 0, i4);
  run(Int<1>{}, i4, i6);
  run(Int<2>{}, i6, i8);
  // Group 1 has one iteration less when nsteps is odd; it still meets the
  // barrier of group 0's last iteration.
  const int niter = (nsteps + 1) >> 1;
  if (i8 < niter) {
    if (i8 & 1) iteration(Int<2>{}, Int<1>{}, i8, false);
    else iteration(Int<2>{}, Int<0>{}, i8, false);
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
