// attn.hip -- decode attention over an MXINT KV cache.
//
// MXSens (arXiv 2607.17733), Appendix A.2: the KV cache is quantized to
// MXINT (32-element blocks along the head dimension, 4 to 8 bits each) and
// attention reads it.  One new token per sequence attends to the T cached
// tokens of its sequence: per query head h (KV head h / G, G = Hq / Hkv),
// s_t = (q_h . K_t) * scale, p = softmax(s), o_h = sum_t p_t V_t, with K_t
// and V_t dequantized block by block, value = q * 2^(E - 127 - (m - 2)).
//
// The caches are the activation quantizer's packed rows (row (b * T + t) *
// Hkv + h, D = 128 values in four blocks) and exponent rows.  The token range
// of a (sequence, KV head) is split over workgroups so that a small batch
// still fills the GPU; the four waves of a workgroup take chunks of 32 tokens
// in turn, staging the chunk's K and V rows in LDS.
//
// Both products run on the bf16 matrix cores (16x16x32, float32
// accumulation).  A dequantized value q * 2^k with |q| <= 128 is exact in
// bf16, and so is a bf16 query element, so every product is exact:
//   scores  S[token][head] = sum over the four blocks of K_blk . Q_blk^T,
//           the block scale applied to K's digits before the conversion;
//   values  O[head][d] += P . V, where the float32 probabilities are split
//           into three bf16 terms whose sum is the float32 value, so the
//           weights are those of a float32 softmax.
// A lane of the score product's output holds one head and four tokens of
// each 16-token half, the online softmax state (running maximum and sum) is
// one value per head, and the same lane supplies that head's probabilities
// to the value product, its eight tokens being the product's reduction slots
// (the V operand takes its tokens in the same slots).  Waves, then splits, are
// merged in a fixed order, so results do not depend on timing.  Each width mix
// of the four blocks is its own instance, so block offsets and widths are
// compile-time constants.
#include <mutex>

#include "mxq_internal.h"

namespace mxq {

// Per-split partial results of the allocation-free entry point: one array
// per GPU, resident until the process ends.  In host code `scratch` names a
// host-side stand-in, not device memory; its device address comes from
// hipGetSymbolAddress, once per device, with that device current.
static __device__ __align__(256) float scratch[kAttnStaticWorkBytes / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float *g_scratch_ptr[kMaxDevices] = {};

}  // namespace

hipError_t attn_static_scratch(float **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = (float *)p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

namespace {

typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef unsigned u2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr int kD = 128;
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxG = 16;
constexpr int kChunk = 32;         // tokens per wave step: the value product's reduction

// The four blocks of a cache row (head dimension 128): N3 3-bit, N4 4-bit,
// N6 6-bit and N8 8-bit blocks, in that order.
template <int N3, int N4, int N6, int N8>
struct Geo {
  static constexpr int width(int b) {
    return b < N3 ? 3 : b < N3 + N4 ? 4 : b < N3 + N4 + N6 ? 6 : 8;
  }
  static constexpr int off(int b) { return b == 0 ? 0 : off(b - 1) + 4 * width(b - 1); }
  static constexpr int kRow = (off(4) + 15) / 16 * 16;
  static constexpr int kVec = kRow / 16;                  // 16-byte pieces per row
  // LDS row stride of 8k + 4 dwords: 16 lanes' 16-byte accesses hit distinct banks
  static constexpr int kLds = (kRow + 31) / 32 * 32 + 16;
  static constexpr int kPieces = kChunk * kVec;
};

__device__ inline int sext(uint32_t v, int bits) { return (int)(v << (32 - bits)) >> (32 - bits); }

// 2^(E - 127 - (M - 2)) for block blk of an exponent dword (four blocks)
template <int M>
__device__ inline float block_scale(uint32_t ex, int blk) {
  const int E = (int)((ex >> (8 * blk)) & 255u);
  return __builtin_amdgcn_ldexpf(1.f, E - 127 - (M - 2));
}

// Mantissas 8g .. 8g+7 of the block at p (a K row in LDS).
template <int M>
__device__ inline void mants8(const uint8_t *p, int g, int (&q)[8]) {
  if (M == 3) {
    // elements 8g..8g+7: bits 24g..24g+23 of the block, bytes 3g..3g+2
    const uint32_t w = (uint32_t)p[3 * g] | ((uint32_t)p[3 * g + 1] << 8) |
                       ((uint32_t)p[3 * g + 2] << 16);
#pragma unroll
    for (int j = 0; j < 8; ++j) q[j] = sext((w >> (3 * j)) & 7u, 3);
  } else if (M == 8) {
    const u2 w = *(const u2 *)(p + 8 * g);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      q[j] = sext(w.x >> (8 * j), 8);
      q[4 + j] = sext(w.y >> (8 * j), 8);
    }
  } else {
    const uint32_t w = *(const uint32_t *)(p + 4 * g);
    uint32_t tw = 0;
    if (M == 6) tw = *(const uint32_t *)(p + 16 + 4 * (g >> 1));
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t nib = (w >> (4 * j)) & 15u;
      if (M == 4) {
        q[j] = sext(nib, 4);
      } else {
        const int sh = ((g & 1) ? 2 : 6) - 2 * (j & 1);
        q[j] = sext(nib | (((tw >> (8 * (j >> 1) + sh)) & 3u) << 4), 6);
      }
    }
  }
}

// Mantissa e of the block at p (a V row in LDS), e varying by lane.
template <int M>
__device__ inline int mant1(const uint8_t *p, int e) {
  if (M == 8) return (int)(int8_t)p[e];
  if (M == 3) {
    // bits 3e..3e+2; the byte after the block is read for e = 31 but its
    // bits are shifted out (the row in LDS continues past the block)
    const int bit = 3 * e;
    const uint32_t v = (uint32_t)p[bit >> 3] | ((uint32_t)p[(bit >> 3) + 1] << 8);
    return sext((v >> (bit & 7)) & 7u, 3);
  }
  if (M == 4) return __builtin_amdgcn_sbfe((int)p[e >> 1], 4 * (e & 1), 4);
  const uint32_t nib = __builtin_amdgcn_ubfe((uint32_t)p[e >> 1], 4 * (e & 1), 4);
  const int u = e & 15;
  const int sh = (u < 8 ? 6 : 2) - 2 * (u & 1);
  const int top = __builtin_amdgcn_sbfe((int)p[16 + 4 * (e >> 4) + ((u & 7) >> 1)], sh, 2);
  return top * 16 + (int)nib;
}

__device__ inline bf8 to_bf8(const float (&x)[8]) {
  bf8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = (__bf16)x[j];      // exact: at most 8 significant bits
  return r;
}

// S tile += K rows (token n of the tile, this lane's 8 elements of block BLK) . Q_BLK
template <class Gm, int BLK>
__device__ inline f4 score_block(const uint8_t *kr, uint32_t ex, int g, bf8 qop, f4 acc) {
  constexpr int M = Gm::width(BLK);
  int q[8];
  mants8<M>(kr + Gm::off(BLK), g, q);
  const float sc = block_scale<M>(ex, BLK);
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = (float)q[j] * sc;
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(to_bf8(x), qop, acc, 0, 0, 0);
}

// O tile DT (d = 16 DT + n) += P . V over the chunk's 32 tokens
template <class Gm, int DT>
__device__ inline f4 value_tile(const uint8_t *const (&vr)[8], const uint32_t (&vx)[8], int n,
                                bf8 p1, bf8 p2, bf8 p3, f4 acc) {
  constexpr int BLK = DT >> 1, M = Gm::width(BLK);
  const int e = 16 * (DT & 1) + n;
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
    x[j] = (float)mant1<M>(vr[j] + Gm::off(BLK), e) * block_scale<M>(vx[j], BLK);
  const bf8 v = to_bf8(x);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(p1, v, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(p2, v, acc, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(p3, v, acc, 0, 0, 0);
}

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int N3, int N4, int N6, int N8>
__global__ __launch_bounds__(kThreads, 2) void attn_decode_kernel(AttnArgs a) {
  using Gm = Geo<N3, N4, N6, N8>;
  constexpr int kStage = 2 * kChunk * Gm::kLds;           // a wave's K rows, then V rows
  constexpr int kMerge = kWaves * kMaxG * kD * 4;
  constexpr int kPool = kWaves * kStage > kMerge ? kWaves * kStage : kMerge;
  __shared__ __attribute__((aligned(16))) uint8_t pool[kPool];
  __shared__ uint32_t xs[kWaves][2][kChunk];               // exponent dwords of K, V rows
  __shared__ float mm[kWaves][kMaxG], ml[kWaves][kMaxG];
  const int t = threadIdx.x, lane = t & 63, g = lane >> 4, n = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int G = a.G;
  const float ninf = -__builtin_inff();
  uint8_t *ks = pool + wave * kStage;
  uint8_t *vs = ks + kChunk * Gm::kLds;

  // the score product's Q operand: head n of the group, elements 32 blk + 8 g ..
  bf8 qop[4];
#pragma unroll
  for (int blk = 0; blk < 4; ++blk) {
    u4 x = {0u, 0u, 0u, 0u};
    if (n < G)
      x = *(const u4 *)(a.q + ((int64_t)b * a.Hq + (int64_t)kvh * G + n) * kD + 32 * blk + 8 * g);
    qop[blk] = __builtin_bit_cast(bf8, x);
  }

  const int64_t t0 = (int64_t)split * a.tokens_per_split;
  const int64_t t1 = t0 + a.tokens_per_split < a.T ? t0 + a.tokens_per_split : a.T;
  const int64_t seq0 = (int64_t)b * a.T;
  float run_m = ninf, run_l = 0.f;                         // head n
  f4 o[8];                                                 // heads 4g + r, d = 16 dt + n
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = (f4){0.f, 0.f, 0.f, 0.f};

  // A chunk's rows travel global -> registers -> LDS; the next chunk's loads
  // are issued before the current chunk is computed.  Rows past the end are
  // the chunk's last token (weight 0).
  constexpr int kPer = (Gm::kPieces + 63) / 64;
  u4 pk[kPer], pv[kPer];
  uint32_t px = 0;
  auto fetch = [&](int64_t c) {
    const int m = (int)(t1 - c < kChunk ? t1 - c : kChunk);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int pc = i * 64 + lane;
      if (pc < Gm::kPieces) {
        const int r = pc / Gm::kVec, cc = pc % Gm::kVec;
        const int64_t row = (seq0 + c + (r < m ? r : m - 1)) * a.Hkv + kvh;
        pk[i] = *(const u4 *)(a.k_mant + row * Gm::kRow + 16 * cc);
        pv[i] = *(const u4 *)(a.v_mant + row * Gm::kRow + 16 * cc);
      }
    }
    const int r = lane & 31;
    const int64_t row = (seq0 + c + (r < m ? r : m - 1)) * a.Hkv + kvh;
    px = *(const uint32_t *)((lane < 32 ? a.k_exp : a.v_exp) + row * a.exp_bytes);
  };
  if (t0 + kChunk * wave < t1) fetch(t0 + kChunk * wave);

  for (int64_t c0 = t0 + kChunk * wave; c0 < t1; c0 += kChunk * kWaves) {
    const int nt = (int)(t1 - c0 < kChunk ? t1 - c0 : kChunk);
    wave_sync();                                           // the previous chunk is consumed
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int pc = i * 64 + lane;
      if (pc < Gm::kPieces) {
        const int r = pc / Gm::kVec, cc = pc % Gm::kVec;
        *(u4 *)(ks + r * Gm::kLds + 16 * cc) = pk[i];
        *(u4 *)(vs + r * Gm::kLds + 16 * cc) = pv[i];
      }
    }
    xs[wave][lane >> 5][lane & 31] = px;
    wave_sync();
    if (c0 + kChunk * kWaves < t1) fetch(c0 + kChunk * kWaves);

    // scores: tokens 16 mt + 4 g + r of head n
    f4 sacc[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const uint8_t *kr = ks + (16 * mt + n) * Gm::kLds;
      const uint32_t ex = xs[wave][0][16 * mt + n];
      f4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = score_block<Gm, 0>(kr, ex, g, qop[0], acc);
      acc = score_block<Gm, 1>(kr, ex, g, qop[1], acc);
      acc = score_block<Gm, 2>(kr, ex, g, qop[2], acc);
      acc = score_block<Gm, 3>(kr, ex, g, qop[3], acc);
      sacc[mt] = acc * a.scale;
    }
    // online softmax; slot j of this lane is token tok(j)
    float p[8];
    float cm = ninf;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int tok = 16 * (j >> 2) + 4 * g + (j & 3);
      p[j] = tok < nt ? sacc[j >> 2][j & 3] : ninf;
      cm = fmaxf(cm, p[j]);
    }
    cm = fmaxf(cm, __shfl_xor(cm, 16));
    cm = fmaxf(cm, __shfl_xor(cm, 32));
    const float nm = fmaxf(run_m, cm);
    const float alpha = expf(run_m - nm);                  // 0 while nothing was seen
    float ls = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      p[j] = expf(p[j] - nm);
      ls += p[j];
    }
    ls += __shfl_xor(ls, 16);
    ls += __shfl_xor(ls, 32);
    run_l = run_l * alpha + ls;
    run_m = nm;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float ah = __shfl(alpha, 4 * g + r);           // head 4g + r lives in lane 4g + r
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) o[dt][r] *= ah;
    }
    // the probabilities as three bf16 terms summing to the float32 value
    float x1[8], x2[8], x3[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      x1[j] = (float)(__bf16)p[j];
      const float r1 = p[j] - x1[j];
      x2[j] = (float)(__bf16)r1;
      x3[j] = r1 - x2[j];
    }
    const bf8 p1 = to_bf8(x1), p2 = to_bf8(x2), p3 = to_bf8(x3);
    // values: the V operand takes token tok(j) in slot j
    const uint8_t *vr[8];
    uint32_t vx[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int tok = 16 * (j >> 2) + 4 * g + (j & 3);
      vr[j] = vs + tok * Gm::kLds;
      vx[j] = xs[wave][1][tok];
    }
    o[0] = value_tile<Gm, 0>(vr, vx, n, p1, p2, p3, o[0]);
    o[1] = value_tile<Gm, 1>(vr, vx, n, p1, p2, p3, o[1]);
    o[2] = value_tile<Gm, 2>(vr, vx, n, p1, p2, p3, o[2]);
    o[3] = value_tile<Gm, 3>(vr, vx, n, p1, p2, p3, o[3]);
    o[4] = value_tile<Gm, 4>(vr, vx, n, p1, p2, p3, o[4]);
    o[5] = value_tile<Gm, 5>(vr, vx, n, p1, p2, p3, o[5]);
    o[6] = value_tile<Gm, 6>(vr, vx, n, p1, p2, p3, o[6]);
    o[7] = value_tile<Gm, 7>(vr, vx, n, p1, p2, p3, o[7]);
  }

  // merge the waves in order (the staging area now holds their outputs)
  __syncthreads();
  float *mo = (float *)pool;                               // [kWaves][kMaxG][kD]
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (4 * g + r < G) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) mo[(wave * kMaxG + 4 * g + r) * kD + 16 * dt + n] = o[dt][r];
    }
  }
  if (g == 0 && n < G) {
    mm[wave][n] = run_m;
    ml[wave][n] = run_l;
  }
  __syncthreads();
  float *part = a.work + (((int64_t)b * a.Hkv + kvh) * a.splits + split) * G * (kD + 2);
  for (int i = t; i < G * kD; i += kThreads) {
    const int h = i / kD, d = i - h * kD;
    float M = ninf;
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, mm[w][h]);
    float L = 0.f, O = 0.f;
    for (int w = 0; w < kWaves; ++w) {
      if (mm[w][h] == ninf) continue;                      // a wave that had no chunk
      const float f = expf(mm[w][h] - M);
      L += ml[w][h] * f;
      O += mo[(w * kMaxG + h) * kD + d] * f;
    }
    part[h * (kD + 2) + 2 + d] = O;
    if (d == 0) {
      part[h * (kD + 2)] = M;
      part[h * (kD + 2) + 1] = L;
    }
  }
}

// o[b][h] = the splits' partials merged in a fixed order.  The splits'
// maxima and sums are gathered in parallel, their weights kept in LDS; four
// thread groups take every fourth split (each issuing its loads together),
// and their sums are added in group order.
constexpr int kCombGroups = 4;

__global__ __launch_bounds__(kD * kCombGroups) void attn_combine_kernel(AttnArgs a) {
  __shared__ float wf[kAttnMaxSplits], wl[kAttnMaxSplits], red[kCombGroups * 2];
  __shared__ float po[kCombGroups][kD], pl[kCombGroups];
  const int t = threadIdx.x, d = t % kD, grp = t / kD, h = blockIdx.x, b = blockIdx.y;
  const int G = a.G, kvh = h / G, g = h - kvh * G, S = a.splits;
  const float *base = a.work + (((int64_t)b * a.Hkv + kvh) * S * G + g) * (kD + 2);
  const int64_t stride = (int64_t)G * (kD + 2);
  float M = -__builtin_inff();
  for (int s = t; s < S; s += kD * kCombGroups) {
    wf[s] = base[s * stride];
    wl[s] = base[s * stride + 1];
    M = fmaxf(M, wf[s]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
  if ((t & 63) == 0) red[t >> 6] = M;
  __syncthreads();
  M = red[0];
  for (int w = 1; w < kCombGroups * 2; ++w) M = fmaxf(M, red[w]);
  for (int s = t; s < S; s += kD * kCombGroups) {
    const float f = expf(wf[s] - M);
    wf[s] = f;
    wl[s] *= f;
  }
  __syncthreads();
  float L = 0.f, O = 0.f;
#pragma unroll 16
  for (int s = grp; s < S; s += kCombGroups) {
    L += wl[s];
    O += base[s * stride + 2 + d] * wf[s];
  }
  po[grp][d] = O;
  if (d == 0) pl[grp] = L;
  __syncthreads();
  if (grp == 0) {
    float Ls = 0.f, Os = 0.f;
    for (int k = 0; k < kCombGroups; ++k) {
      Ls += pl[k];
      Os += po[k][d];
    }
    a.o[((int64_t)b * a.Hq + h) * kD + d] = Os / Ls;
  }
}

template <int N3, int N4, int N6, int N8>
void launch_t(const AttnArgs &a, hipStream_t s) {
  hipLaunchKernelGGL((attn_decode_kernel<N3, N4, N6, N8>),
                     dim3((unsigned)a.splits, (unsigned)a.Hkv, (unsigned)a.B), dim3(kThreads), 0,
                     s, a);
}

// The kernel for a row's width mix, code = 125 n3 + 25 n4 + 5 n6 + n8 (the
// 35 mixes of four blocks).
template <int C>
bool dispatch(int code, const AttnArgs &a, hipStream_t s) {
  constexpr int n3 = C / 125, n4 = C / 25 % 5, n6 = C / 5 % 5, n8 = C % 5;
  if constexpr (n3 + n4 + n6 + n8 == 4) {
    if (code == C) {
      launch_t<n3, n4, n6, n8>(a, s);
      return true;
    }
  }
  if constexpr (C > 0) {
    return dispatch<C - 1>(code, a, s);
  } else {
    return false;
  }
}

}  // namespace

int64_t attn_tokens_per_split(int64_t B, int64_t Hkv, int64_t T) {
  // about 512 workgroups, whole multiples of 64 tokens
  const int64_t chunks = (T + 63) / 64;
  int64_t s = (512 + B * Hkv - 1) / (B * Hkv);
  if (s > chunks) s = chunks;
  if (s < 1) s = 1;
  return (chunks + s - 1) / s * 64;
}

hipError_t launch_attn_decode(const AttnArgs &a, hipStream_t s) {
  const int n3 = a.n3, n4 = a.n4 - a.n3;
  if (n3 < 0 || n4 < 0 || n3 + n4 + a.n6 + a.n8 != 4) return hipErrorInvalidValue;
  if (!dispatch<500>(125 * n3 + 25 * n4 + 5 * a.n6 + a.n8, a, s)) return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_combine_kernel, dim3((unsigned)a.Hq, (unsigned)a.B), dim3(kD * kCombGroups),
                     0, s, a);
  return hipGetLastError();
}

}  // namespace mxq
