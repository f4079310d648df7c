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
// a per-lane address and no data is moved.  Each lane restores its weight
// operand from LDS with a few masks and shifts; the hardware applies every
// block's E8M0 scale and accumulates in fp32.  Per 32x32 tile and K-chunk
// (64 K-values):
//   3- and 4-bit (two blocks): one FP6 instruction;
//   6-bit (one block, its two digit planes as the K halves): two FP6
//     instructions, the weights' high plane in both halves, then the low;
//   8-bit (one block, the same way): two FP8 instructions.
// The digit products are exact; only the fp32 accumulation rounds.
//
// Tiling: 256x128 outputs per workgroup (one weight super-slab) of four
// waves, one per SIMD, so that each wave has the whole register file: wave
// w owns rows 64w..64w+63 x all 128 columns = 2x4 tiles of 32x32 fp32
// accumulators, and walks every step.  Grids of fewer such workgroups than
// the device has CUs take 128x128 tiles instead (wave w: rows 32w..32w+31,
// 1x4 tiles; two workgroups per CU fit): twice the workgroups, each wave
// half the products per step.
//   - activations go straight from the image into registers -- each row is
//     used by exactly one wave -- one step ahead, in two register sets, two
//     loads in each of the step's first four positions;
//   - the scale words (activation and weight) are loaded once per group of
//     four steps, a group ahead, over three positions;
//   - the weight chunk of each step (8 slabs, 6 to 12 KB) goes global -> LDS
//     by direct-to-LDS loads into a ring of eight step stages, four steps
//     ahead (a wave's share over two positions); the four waves read it per
//     column tile and K-chunk, two
//     (tile, chunk) positions ahead of the products, and restore each
//     operand among the previous position's products (a few VALU
//     instructions after each) into alternating registers.
// A step has no branch, so the compiler keeps this order.  One barrier per
// step; the kernel counts its own loads (vmcnt) to know when a stage is
// complete.  Workgroup ids are remapped so that each XCD owns
// a compact block of output tiles: the activation rows and weight columns it
// reads stay in its L2.
#include "mxq_device.h"
#include "mxq_internal.h"

#include <type_traits>

namespace mxq {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef unsigned u2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int BN = kWCols, NT = 256, kWaves = NT / 64;
constexpr int kFmtE4M3 = 0, kFmtE2M3 = 2, kFmtE3M2 = 3;
constexpr int kWStages = 8;                  // weight ring: one stage per step (a power of two)
constexpr int kWAhead = 4;                   // weight stages loaded ahead
constexpr int kASets = 2;                    // activation register sets (one ahead)
// Activation loads per wave and step: per 32-row tile (TM of them) and
// K-chunk the lane data (two loads).
template <int TM> constexpr int kALoads = 2 * 2 * TM;
// Loads per wave and scale group: the activation scale word per 32-row tile
// and K-chunk, then the group's weight scale bytes (two 16-byte pieces per
// K-chunk).
template <int TM> constexpr int kGLoads = 2 * TM + 2 * 2;

template <int S> struct Int { static constexpr int v = S; };

template <bool FULL> struct Cfg {
  static constexpr int kPieces = FULL ? 12 : 8;           // 1 KB pieces per stage
  static constexpr int kStage = kPieces * 1024;
  static constexpr int kRing = kWStages * kStage;
  static constexpr int kWLoads = kPieces / kWaves;        // per wave and step
};
static_assert(Cfg<true>::kRing <= 160 * 1024, "LDS");
static_assert((kWStages & (kWStages - 1)) == 0, "stage index by mask");
static_assert(Cfg<true>::kPieces % kWaves == 0 && Cfg<false>::kPieces % kWaves == 0, "pieces");

// The scale operands are dwords whose byte OA (activations) / OB (weights)
// holds the E8M0 scale.
template <int FA, int FB, int OA, int OB>
__device__ inline v16f mma(const v8i &a, const v8i &b, v16f c, uint32_t sa, uint32_t sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, FA, FB, OA, (int)sa, OB, (int)sb);
}

// The ring's synchronisation is explicit: the compiler does not know which
// direct-to-LDS load fills which stage, and may not move LDS accesses across
// these points.
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

// The six dwords of an FP6 operand as the instruction's eight-dword operand
// (the last two are not read for FP6 and stay undefined: no write).
__device__ inline v8i six(const uint32_t *d) {
  const u4 a = u4{d[0], d[1], d[2], d[3]};
  const u2 b = u2{d[4], d[5]};
  const u4 b4 = __builtin_shufflevector(b, b, 0, 1, -1, -1);
  return (v8i)__builtin_shufflevector(a, b4, 0, 1, 2, 3, 4, 5, 6, 7);
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

// TM: 32-row tiles per wave (2: 256-row workgroup tiles, one workgroup per
// CU; 1: 128-row tiles, two per CU).
template <bool FULL, int TM>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(3 - TM, 3 - TM)))
void gemm_prefill_kernel(GemmArgs g, int mtiles, int ntiles, int gm, int gn) {
  constexpr int BM = 128 * TM;
  using C = Cfg<FULL>;
  __shared__ __attribute__((aligned(16))) u4 lds[C::kRing / 16];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);      // wave-uniform
  const int l32 = lane & 31, lh = lane >> 5, l16 = lane & 15, hx = l32 >> 4;
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

  // This wave's rows: TM 32-row tiles = 2 TM 16-row image tiles (tiles
  // past the last one read the last tile; those rows are never stored).  The
  // activation resources start at the wave's first 16-row tile (64-bit
  // arithmetic), so the 32-bit buffer offsets stay below 4 image tiles; the
  // host rejects shapes where 16 tiles pass INT32_MAX.
  const int64_t last = (g.M - 1) / kATileRows;
  const int64_t ta = min(row0 / kATileRows + 2 * TM * wave, last);
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.a_mant + ta * g.a_tile), 0,
      (int)min((last + 1 - ta) * g.a_tile, (int64_t)0x7fffffff), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.a_exp + ta * g.a_tile_sc), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.w_mant + (int64_t)nt * g.w_super), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rws = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(g.w_exp + (int64_t)nt * g.w_super_sc), 0, 0x7fffffff, 0x00020000);
  // The lane (lh, x) of a 32-wide tile reads, for K-chunk c, lane
  // lk(c) = 16 (2 c + lh) + x % 16 of 16-row image tile (or slab) 2 tm + x / 16.
  const int lk0 = 16 * lh + l16, lk1 = lk0 + 32;
  int vt[TM];                                 // the lane's image tile of row tile tm
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) vt[tm] = (int)(min(ta + 2 * tm + hx, last) - ta);

  v16f acc[TM][4];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[a][n] = v16f{};

  // Activation registers of one step: per 32-row tile and K-chunk the lane
  // data (24 bytes of FP6 codes or 32 of FP8 codes) and the scale word; the
  // step's weight scale bytes for each K-chunk (slab n at byte n).
  struct ASet {
    v8i d[TM][2];
  };
  ASet xa[kASets];
  // Scale words of a group of four steps: per 32-row tile and K-chunk the
  // activation scale dword (byte k for step k), per K-chunk the lane's 32
  // weight scale bytes (slab n's byte of step k at 8 k + n).  Set 0 serves
  // the current group; set 1 receives the next group's.
  struct GScale {
    uint32_t sc[TM][2];
    u4 ws[2][2];
  };
  GScale gsc[2];

  // Offsets of step st in the images, in branch-free scalar arithmetic (a
  // segment's steps before st are clamp(st - st0, 0, S)).  Scale groups are
  // counted as the segments walk them (a segment's steps start a group).
  constexpr int CB0 = w_chunk_bytes(0, FULL), CB1 = w_chunk_bytes(1, FULL),
                CB2 = w_chunk_bytes(2, FULL), CB3 = w_chunk_bytes(3, FULL);
  auto dseg = [&](int st, int k) __attribute__((always_inline)) {
    return min(max(st - lg.st0[k], 0), lg.S[k]);
  };
  auto a_off = [&](int st) __attribute__((always_inline)) {
    // 24-byte lanes before the 8-bit segment, 32-byte lanes in it
    return kLanes * (24 * min(st, lg.st0[3]) + 32 * max(st - lg.st0[3], 0));
  };
  auto w_off = [&](int st) __attribute__((always_inline)) {
    return kWSlabs * (CB0 * dseg(st, 0) + CB1 * dseg(st, 1) + CB2 * dseg(st, 2) +
                      CB3 * max(st - lg.st0[3], 0));
  };
  auto w_pieces = [&](int st) __attribute__((always_inline)) {
    int cb = CB0;
    cb = st >= lg.st0[1] ? CB1 : cb;
    cb = st >= lg.st0[2] ? CB2 : cb;
    cb = st >= lg.st0[3] ? CB3 : cb;
    return cb * kWSlabs / 1024;
  };

  // Weight loads of step st (clamped to the last) into its stage: pieces
  // n = 0 .. kPieces - 1 of 1 KB (pieces past the step's chunk bytes repeat
  // its last piece); wave w issues n = w + 4 j for j in [j0, j1).
  auto issue_w = [&](int st, int j0, int j1) __attribute__((always_inline)) {
    st = min(st, nsteps - 1);
    const int wo = w_off(st), np = w_pieces(st);
    char *stage = ring + (st & (kWStages - 1)) * C::kStage;
#pragma unroll
    for (int j = j0; j < j1; ++j) {
      const int kb = min(wave + kWaves * j, np - 1);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_void *)(stage + kb * 1024), 16, lane * 16,
                                               wo + kb * 1024, 0, 0);
    }
  };
  // Activation loads of step st (clamped to the last) into register set S,
  // part = the (32-row tile, K-chunk) pair: tile part % TM, chunk part / TM.
  // A wave that issues its loads in bursts stalls on them; spread over the
  // positions, they are accepted while the products run.
  auto issue_a = [&](auto set_tag, int st, int part) __attribute__((always_inline)) {
    constexpr int S = decltype(set_tag)::v;
    st = min(st, nsteps - 1);
    const int so = a_off(st);
    const bool wide = st >= lg.st0[3];
    const int tm = part % TM, c = part / TM;
    const int lk = c ? lk1 : lk0;
    const int vb = vt[tm] * (int)g.a_tile;
    const int olo = wide ? 32 * lk0 + 16 * c : 24 * lk;
    const int ohi = wide ? 32 * lk1 + 16 * c : 24 * lk + 16;
    const u4 lo = __builtin_bit_cast(u4, __builtin_amdgcn_raw_buffer_load_b128(ra, vb + olo, so, 0));
    const u4 hi = __builtin_bit_cast(u4, __builtin_amdgcn_raw_buffer_load_b128(ra, vb + ohi, so, 0));
    xa[S].d[tm][c] = (v8i)__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  // Scale loads of group grp (clamped to the last) into set G: part 0 the
  // activation scale dwords, part 1 + c the weight scale bytes of K-chunk c.
  auto issue_g = [&](auto gset_tag, int grp, int part) __attribute__((always_inline)) {
    constexpr int G = decltype(gset_tag)::v;
    grp = min(grp, lg.ngroups - 1);
    if (part == 0) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int c = 0; c < 2; ++c)
          gsc[G].sc[tm][c] = __builtin_amdgcn_raw_buffer_load_b32(
              rs, vt[tm] * (int)g.a_tile_sc + 4 * (c ? lk1 : lk0), grp * 256, 0);
    } else {
      const int c = part - 1;
#pragma unroll
      for (int h = 0; h < 2; ++h)
        gsc[G].ws[c][h] = __builtin_bit_cast(
            u4, __builtin_amdgcn_raw_buffer_load_b128(rws, 32 * (c ? lk1 : lk0) + 16 * h,
                                                      grp * 2048, 0));
    }
  };

  // Weight operand of column tile tn, K-chunk c (position p = 2 tn + c of
  // a step): the lane's raw bytes, read from LDS two positions ahead into
  // one of four slots, and its FP6 / FP8 codes, restored one position ahead
  // into one of two operand registers, so that a restore never writes the
  // registers the products in flight read.
  struct WRaw {
    u4 p, h;
    u2 q;
    uint32_t z;
  };
  struct WOp {
    v8i b0, b1;                   // 3/4-bit: b0; 6/8-bit: high plane b0, low plane b1
  };
  WRaw w[4];
  WOp bo[2];
  auto read_w = [&](auto seg, const char *stage, int o, int p) __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v;
    constexpr int CB = w_chunk_bytes(SEG, FULL);
    const int tn = p >> 1, c = p & 1;
    const char *ch = stage + (2 * tn + hx) * CB;
    const int lk = c ? lk1 : lk0;
    WRaw &r = w[o];
    if (SEG == 0 && !FULL) {
      r.q = *(const u2 *)(ch + 8 * lk);
      r.z = *(const uint32_t *)(ch + 512 + 4 * lk);
    } else if (SEG <= 1) {
      r.p = *(const u4 *)(ch + 16 * lk);
      if (SEG == 1 && FULL) r.q = *(const u2 *)(ch + 1024 + 8 * lk);
    } else if (SEG == 2) {
      const int jc = 16 * c + l16;
      r.p = *(const u4 *)(ch + 16 * jc);
      if (FULL) r.h = *(const u4 *)(ch + 512 + 16 * jc);
      else r.q = *(const u2 *)(ch + 512 + 8 * jc);
    } else {
      r.p = *(const u4 *)(ch + 32 * (16 * c + l16) + 16 * lh);
    }
  };
  auto restore = [&](auto seg, int o, int ob) __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v;
    const WRaw &r = w[o];
    WOp &B = bo[ob];
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
      B.b0 = six(d);
    } else if (SEG == 2) {
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
      B.b0 = six(H);
      B.b1 = six(L);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        B.b0[k] = B.b0[4 + k] = (int)hi_codes<FULL>(r.p[k]);
        B.b1[k] = B.b1[4 + k] = (int)lo_codes<FULL>(r.p[k]);
      }
    }
  };
  // The products of position p with operand register ob, first or second
  // half: 3/4-bit: row tile 0 | 1; 6-bit: the weights' high plane in both K
  // halves (scale E + 3) for both row tiles | their low plane (scale E);
  // 8-bit: the high digits (scale E + 4) | the low digits.
  // The activation scale of step k is byte k of the group's scale dword;
  // the weight scale of slab n = 2 tn + hx is byte 8 k + n of the lane's 32
  // bytes, i.e. byte 2 (tn & 1) of dword 2 k + (tn >> 1) once the lane's
  // dwords are shifted right by 8 hx (done when a group's scales become
  // current).  3- and 4-bit products select both bytes with the
  // instruction's operand selects; 6- and 8-bit products add 3 or 4 to the
  // weight scale first.
  auto products = [&](auto seg, auto k_tag, const ASet &x, int p, int ob, int half)
                      __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v, K = decltype(k_tag)::v;
    const int tn = p >> 1, c = p & 1;
    const uint32_t wd = gsc[0].ws[c][K >> 1][2 * (K & 1) + (tn >> 1)];
    const WOp &B = bo[ob];
    if (SEG <= 1) {
      constexpr int FB = SEG == 0 ? kFmtE2M3 : kFmtE3M2;
      const int tm = half;
      if (tm >= TM) return;
      acc[tm][tn] = (tn & 1)
          ? mma<kFmtE3M2, FB, K, 2>(x.d[tm][c], B.b0, acc[tm][tn], gsc[0].sc[tm][c], wd)
          : mma<kFmtE3M2, FB, K, 0>(x.d[tm][c], B.b0, acc[tm][tn], gsc[0].sc[tm][c], wd);
    } else {
      const uint32_t e = (wd >> (16 * (tn & 1))) & 0xFFu;
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        if (SEG == 2)
          acc[tm][tn] = half == 0
              ? mma<kFmtE3M2, kFmtE3M2, K, 0>(x.d[tm][c], B.b0, acc[tm][tn], gsc[0].sc[tm][c],
                                              sat_plus<3>(e))
              : mma<kFmtE3M2, kFmtE3M2, K, 0>(x.d[tm][c], B.b1, acc[tm][tn], gsc[0].sc[tm][c], e);
        else
          acc[tm][tn] = half == 0
              ? mma<kFmtE4M3, kFmtE4M3, K, 0>(x.d[tm][c], B.b0, acc[tm][tn], gsc[0].sc[tm][c],
                                              sat_plus<4>(e))
              : mma<kFmtE4M3, kFmtE4M3, K, 0>(x.d[tm][c], B.b1, acc[tm][tn], gsc[0].sc[tm][c], e);
      }
    }
  };
  // The next group's scales become current (the weight dwords shifted).
  auto next_group = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int c = 0; c < 2; ++c) gsc[0].sc[tm][c] = gsc[1].sc[tm][c];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 4; ++i) gsc[0].ws[c][h][i] = gsc[1].ws[c][h][i] >> (8 * hx);
  };

  // Step s (register set S = s % 2): the products position by position.  At
  // position p the step reads the raw operand of p + 2 (positions 8 and 9
  // are the next step's first two, read after the barrier), issues the
  // first half of p's products, restores the operand of p + 1, then issues
  // the second half.  Positions 0 to 3 issue the activation loads of step
  // s + 1, one (tile, chunk) pair each; between positions 3 and 4 the
  // workgroup meets at a barrier, then positions 4 and 6 issue the weight
  // loads of step s + 4 (and positions 4 to 6 of a group's first step the
  // next group's scale loads).  Before the barrier each wave waits for its
  // own weight loads of step s + 1: since them it has issued the activations
  // of s - 1, s and s + 1 and the weights of s + 2 and s + 3, perhaps with
  // scale loads between them, so leaving at most two activation and two
  // weight bundles in flight waits for them (and for the activations of
  // s - 1, already consumed; this also holds in the first steps, after the
  // prologue).  After the barrier the stage of s + 1 is complete, and every
  // wave is past step s - 1, whose stage ((s + 4) % 8 = (s - 4) % 8 is older
  // still) the weight loads of s + 4 may then overwrite.
  auto step = [&](auto seg, auto set_tag, auto k_tag, int s, int grp) __attribute__((always_inline)) {
    constexpr int SEG = decltype(seg)::v, S = decltype(set_tag)::v, K = decltype(k_tag)::v;
    const char *W = ring + (s & (kWStages - 1)) * C::kStage;
    const char *Wn = ring + ((s + 1) & (kWStages - 1)) * C::kStage;
    const ASet &x = xa[S];
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      if (p == 4) {
        wait_loads<2 * kALoads<TM> + 2 * C::kWLoads>();
        barrier();
        issue_w(s + kWAhead, 0, 1);
      }
      if (p == 6) issue_w(s + kWAhead, 1, C::kWLoads);
      // positions 8 and 9: the next step's (unused when that step starts a
      // new segment, whose loop reads them again)
      if (p + 2 < 8) read_w(seg, W, (p + 2) & 3, p + 2);
      else read_w(seg, Wn, (p + 2) & 3, p - 6);
      if (p < 2 * TM) issue_a(Int<(S + 1) % kASets>{}, s + 1, p);
      if (p >= 4 && p < 7 && K == 0) issue_g(Int<1>{}, grp + 1, p - 4);
      __builtin_amdgcn_sched_barrier(0);
      // the products interleaved with the next operand's restore: a wave
      // hides a few VALU instructions behind each of its matrix-core
      // products, not a long run of them
      products(seg, k_tag, x, p, p & 1, 0);
      restore(seg, (p + 1) & 3, (p + 1) & 1);
      products(seg, k_tag, x, p, p & 1, 1);
      if (SEG <= 1) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 16, 0);
      } else {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 24, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Steps [sb, se) of one segment: pairs of steps (register sets 0 and 1)
  // in a loop with one exit, then a last odd step.  `cur` is the set that
  // holds the next step's activations; a segment that starts with them in
  // set 1 first copies them to set 0 (at most three times per kernel).  The
  // first step reads its own first two raw operands and restores the first.
  int cur = 0, grpc = 0;
  auto run = [&](auto seg, int sb, int se) __attribute__((always_inline)) {
    if (sb >= se) return;
    if (cur) xa[0] = xa[1];
    const char *W0 = ring + (sb & (kWStages - 1)) * C::kStage;
    read_w(seg, W0, 0, 0);
    read_w(seg, W0, 1, 1);
    restore(seg, 0, 0);
    // groups of four steps (a segment starts a group): the first step of a
    // group loads the next group's scales, which then replace the current
    int s = sb;
    for (; s + 4 <= se; s += 4) {
      const int grp = grpc++;
      step(seg, Int<0>{}, Int<0>{}, s, grp);
      step(seg, Int<1>{}, Int<1>{}, s + 1, grp);
      step(seg, Int<0>{}, Int<2>{}, s + 2, grp);
      step(seg, Int<1>{}, Int<3>{}, s + 3, grp);
      next_group();
    }
    const int n = se - s;
    cur = n & 1;
    if (n > 0) {
      const int grp = grpc++;
      step(seg, Int<0>{}, Int<0>{}, s, grp);
      if (n > 1) step(seg, Int<1>{}, Int<1>{}, s + 1, grp);
      if (n > 2) step(seg, Int<0>{}, Int<2>{}, s + 2, grp);
      next_group();
    }
  };

  // Prologue: the weights of steps 0 and 1, the activations of step 0, the
  // weights of steps 2 and 3, and the wait for the stage of step 0.
  issue_w(0, 0, C::kWLoads);
  issue_w(1, 0, C::kWLoads);
  for (int pp = 0; pp < 2 * TM; ++pp) issue_a(Int<0>{}, 0, pp);
  for (int pp = 0; pp < 3; ++pp) issue_g(Int<1>{}, 0, pp);
  issue_w(2, 0, C::kWLoads);
  issue_w(3, 0, C::kWLoads);
  __builtin_amdgcn_sched_barrier(0);
  wait_loads<3 * C::kWLoads + kALoads<TM> + kGLoads<TM>>();
  barrier();
  next_group();

  run(Int<0>{}, 0, lg.st0[1]);
  run(Int<1>{}, lg.st0[1], lg.st0[2]);
  run(Int<2>{}, lg.st0[2], lg.st0[3]);
  run(Int<3>{}, lg.st0[3], nsteps);
  // no direct-to-LDS load may outlive the workgroup
  wait_loads<0>();

  // Epilogue: each quad of lanes transposes its 4x4 pieces (rows of a lane,
  // columns of the quad) so that a lane stores four consecutive columns.
  const bool vec = (g.ldy & 3) == 0 && ((uintptr_t)g.y & 15) == 0 && col0 + BN <= g.N;
  const int j = l32 & 3;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < 4; ++tn)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int rr = wave * 32 * TM + tm * 32 + 8 * q + 4 * lh, cc = tn * 32 + l32;
        v4f s = v4f{acc[tm][tn][4 * q], acc[tm][tn][4 * q + 1], acc[tm][tn][4 * q + 2],
                    acc[tm][tn][4 * q + 3]};
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

}  // namespace

hipError_t launch_gemm_prefill(const GemmArgs &a, hipStream_t stream) {
  auto go = [&](auto fc, auto tc) {
    constexpr bool FULL = decltype(fc)::value;
    constexpr int TM = decltype(tc)::value;
    constexpr int BM = 128 * TM;
    const int mtiles = (int)((a.M + BM - 1) / BM), ntiles = (int)((a.N + BN - 1) / BN);
    // Split the tile grid into 8 blocks (one per XCD) along rows x columns,
    // minimising the bytes each XCD reads: an activation tile weighs about
    // TM times a weight tile.
    int gm = 0, gn = 0, best = 0;
    for (int m = 1; m <= 8; m *= 2) {
      const int n = 8 / m;
      if (mtiles % m || ntiles % n) continue;
      const int cost = TM * (mtiles / m) + ntiles / n;
      if (gm == 0 || cost < best) gm = m, gn = n, best = cost;
    }
    hipLaunchKernelGGL((gemm_prefill_kernel<FULL, TM>), dim3((unsigned)(mtiles * ntiles)), dim3(NT),
                       0, stream, a, mtiles, ntiles, gm, gn);
  };
  // 128-row tiles when 256-row tiles would leave CUs without a workgroup
  // (measured at K = N = 4096: 29-33 us against 37-41 us for M = 65 to
  // 1024; 256-row tiles are faster from one workgroup per CU up).  The
  // full clamp's 12 KB weight stages fit one workgroup per CU only.
  const int64_t wg256 = ((a.M + 255) / 256) * ((a.N + BN - 1) / BN);
  if (a.full) go(std::true_type{}, std::integral_constant<int, 2>{});
  else if (wg256 < device_cu_count()) go(std::false_type{}, std::integral_constant<int, 1>{});
  else go(std::false_type{}, std::integral_constant<int, 2>{});
  return hipGetLastError();
}

}  // namespace mxq
