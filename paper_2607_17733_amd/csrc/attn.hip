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
// Hkv + h, D = 128 values in four blocks) and exponent rows.  The token
// range of a (sequence, KV head) is split over workgroups so that a small
// batch still fills the GPU.  A workgroup's four waves take chunks of 64
// tokens in turn and keep, per query head of the group, a running maximum,
// sum and output (online softmax, float32):
//   scores  lanes over tokens; each lane reads its token's K row and forms
//           the G dot products against the scaled queries in LDS, block by
//           block (the block's integer dot product, then its scale);
//   values  the chunk's V rows staged in LDS; lane (parity, e) takes
//           element e of every block for the tokens of its parity.
// Waves, then splits, are merged in a fixed order, so results do not depend
// on timing.  Each width mix of the four blocks is its own instance, so
// block offsets and widths are compile-time constants.
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxG = 16;

template <int N4, int N6, int N8>
struct Geo {
  static constexpr int width(int b) { return b < N4 ? 4 : b < N4 + N6 ? 6 : 8; }
  static constexpr int off(int b) {
    return b < N4 ? 16 * b : b < N4 + N6 ? 16 * N4 + 24 * (b - N4)
                                         : 16 * N4 + 24 * N6 + 32 * (b - N4 - N6);
  }
  static constexpr int kRow = (16 * N4 + 24 * N6 + 32 * N8 + 15) / 16 * 16;
  static constexpr int kVec = kRow / 16;
  // LDS row stride of 8k + 4 dwords: 16 lanes' 16-byte reads hit distinct banks
  static constexpr int kLds = (kRow + 31) / 32 * 32 + 16;
};

__device__ inline int sext(uint32_t v, int bits) { return (int)(v << (32 - bits)) >> (32 - bits); }

// Mantissa t of a packed block whose dwords start at w (t a constant after
// unrolling): 4-bit nibbles, 6-bit nibbles plus signed top bits, 8-bit bytes.
template <int M>
__device__ inline int elem(const uint32_t *w, int t) {
  if (M == 8) return sext(w[t >> 2] >> (8 * (t & 3)), 8);
  const uint32_t nib = (w[t >> 3] >> (4 * (t & 7))) & 15u;
  if (M == 4) return sext(nib, 4);
  const int d = t >> 4, u = t & 15, j = (u & 7) >> 1;
  const int sh = (u < 8 ? 6 : 2) - 2 * (u & 1);
  const uint32_t top = (w[4 + d] >> (8 * j + sh)) & 3u;
  return sext(nib | (top << 4), 6);
}

// The same from a row in LDS, t varying by lane.
template <int M>
__device__ inline int elem_lds(const uint8_t *p, int t) {
  if (M == 8) return (int)(int8_t)p[t];
  const uint32_t nib = (p[t >> 1] >> (4 * (t & 1))) & 15u;
  if (M == 4) return sext(nib, 4);
  const int d = t >> 4, u = t & 15, j = (u & 7) >> 1;
  const int sh = (u < 8 ? 6 : 2) - 2 * (u & 1);
  const uint32_t top = (p[16 + 4 * d + j] >> sh) & 3u;
  return sext(nib | (top << 4), 6);
}

template <int M>
__device__ inline float block_scale(uint32_t e_bytes, int blk) {
  const int E = (int)((e_bytes >> (8 * blk)) & 255u);
  return __builtin_amdgcn_ldexpf(1.f, E - 127 - (M - 2));
}

// s[g] += scale_blk * sum_e q_e * qs[32 blk + e][g]
template <class Gm, int BLK>
__device__ inline void score_block(const uint32_t *kw, uint32_t ke, float (&s)[kMaxG], int G,
                                   const float (*qs)[kMaxG]) {
  constexpr int M = Gm::width(BLK);
  float qv[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) qv[e] = (float)elem<M>(kw + Gm::off(BLK) / 4, e);
  const float sc = block_scale<M>(ke, BLK);
#pragma unroll
  for (int gg = 0; gg < kMaxG / 4; ++gg) {
    if (4 * gg < G) {
      f4 part = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int e = 0; e < 32; ++e) part += *(const f4 *)&qs[32 * BLK + e][4 * gg] * qv[e];
#pragma unroll
      for (int k = 0; k < 4; ++k) s[4 * gg + k] += part[k] * sc;
    }
  }
}

// acc[g][BLK] += p[g] * V[row][32 BLK + e]
template <class Gm, int BLK>
__device__ inline void value_block(const uint8_t *vr, uint32_t ve, int e, const float (&p)[kMaxG],
                                   float (&acc)[kMaxG][4], int G) {
  constexpr int M = Gm::width(BLK);
  const float v = (float)elem_lds<M>(vr + Gm::off(BLK), e) * block_scale<M>(ve, BLK);
#pragma unroll
  for (int g = 0; g < kMaxG; ++g)
    if (g < G) acc[g][BLK] += p[g] * v;
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int N4, int N6, int N8>
__global__ __launch_bounds__(kThreads) void attn_decode_kernel(AttnArgs a) {
  using Gm = Geo<N4, N6, N8>;
  // ps and vs during the token loop, then mo for the merge of the waves
  constexpr int kPs = kWaves * 64 * kMaxG * 4, kVs = kWaves * 64 * Gm::kLds;
  static_assert(kPs + kVs >= kWaves * kMaxG * kD * 4, "merge area");
  __shared__ __attribute__((aligned(16))) float qs[kD][kMaxG];
  __shared__ __attribute__((aligned(16))) uint8_t pool[kPs + kVs];
  __shared__ uint32_t vx[kWaves][64];
  __shared__ float mm[kWaves][kMaxG], ml[kWaves][kMaxG];
  float (*ps)[64][kMaxG] = (float (*)[64][kMaxG])pool;
  uint8_t (*vs)[64 * Gm::kLds] = (uint8_t (*)[64 * Gm::kLds])(pool + kPs);
  float (*mo)[kMaxG][kD] = (float (*)[kMaxG][kD])pool;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int G = a.G;
  const float ninf = -__builtin_inff();

  for (int i = t; i < kD * kMaxG; i += kThreads) {
    const int d = i / kMaxG, g = i % kMaxG;
    float v = 0.f;
    if (g < G) {
      const uint16_t qb = a.q[((int64_t)b * a.Hq + (int64_t)kvh * G + g) * kD + d];
      v = __uint_as_float((uint32_t)qb << 16) * a.scale;
    }
    qs[d][g] = v;
  }
  __syncthreads();

  const int64_t t0 = (int64_t)split * a.tokens_per_split;
  const int64_t t1 = t0 + a.tokens_per_split < a.T ? t0 + a.tokens_per_split : a.T;
  float run_m[kMaxG], run_l[kMaxG], acc[kMaxG][4];
#pragma unroll
  for (int g = 0; g < kMaxG; ++g) {
    run_m[g] = ninf;
    run_l[g] = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[g][k] = 0.f;
  }
  const int tp = lane >> 5, e = lane & 31;
  const int64_t seq_row0 = (int64_t)b * a.T;

  for (int64_t c0 = t0 + 64 * wave; c0 < t1; c0 += 64 * kWaves) {
    const int nt = (int)(t1 - c0 < 64 ? t1 - c0 : 64);
    // this lane's token (past the end: the chunk's last token, probability 0)
    const int64_t row = (seq_row0 + c0 + (lane < nt ? lane : nt - 1)) * a.Hkv + kvh;
    uint32_t kw[Gm::kVec * 4];
    const u4 *kp = (const u4 *)(a.k_mant + row * Gm::kRow);
#pragma unroll
    for (int i = 0; i < Gm::kVec; ++i) {
      const u4 x = kp[i];
      kw[4 * i] = x.x;
      kw[4 * i + 1] = x.y;
      kw[4 * i + 2] = x.z;
      kw[4 * i + 3] = x.w;
    }
    const uint32_t ke = *(const uint32_t *)(a.k_exp + row * a.exp_bytes);
    // the chunk's V rows, 16-byte pieces in row order
#pragma unroll
    for (int i = 0; i < Gm::kVec; ++i) {
      const int pc = i * 64 + lane, r = pc / Gm::kVec, c = pc % Gm::kVec;
      const int64_t vrow = (seq_row0 + c0 + (r < nt ? r : nt - 1)) * a.Hkv + kvh;
      *(u4 *)&vs[wave][r * Gm::kLds + 16 * c] = *(const u4 *)(a.v_mant + vrow * Gm::kRow + 16 * c);
    }
    vx[wave][lane] = *(const uint32_t *)(a.v_exp + row * a.exp_bytes);

    float s[kMaxG];
#pragma unroll
    for (int g = 0; g < kMaxG; ++g) s[g] = 0.f;
    score_block<Gm, 0>(kw, ke, s, G, qs);
    score_block<Gm, 1>(kw, ke, s, G, qs);
    score_block<Gm, 2>(kw, ke, s, G, qs);
    score_block<Gm, 3>(kw, ke, s, G, qs);

    const bool live = lane < nt;
#pragma unroll
    for (int g = 0; g < kMaxG; ++g) {
      float p = 0.f;
      if (g < G) {
        const float nm = fmaxf(run_m[g], wave_max(live ? s[g] : ninf));
        const float alpha = expf(run_m[g] - nm);   // 0 while nothing was seen
        p = live ? expf(s[g] - nm) : 0.f;
        run_l[g] = run_l[g] * alpha + wave_sum(p);
        run_m[g] = nm;
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[g][k] *= alpha;
      }
      ps[wave][lane][g] = p;
    }
    wave_sync();

    for (int j = 0; j < nt; j += 2) {
      const int r = j + tp;          // past nt: probability 0, a valid staged row
      const uint8_t *vr = &vs[wave][r * Gm::kLds];
      const uint32_t ve = vx[wave][r];
      float p[kMaxG];
#pragma unroll
      for (int gg = 0; gg < kMaxG / 4; ++gg) {
        f4 x = {0.f, 0.f, 0.f, 0.f};
        if (4 * gg < G) x = *(const f4 *)&ps[wave][r][4 * gg];
        p[4 * gg] = x.x;
        p[4 * gg + 1] = x.y;
        p[4 * gg + 2] = x.z;
        p[4 * gg + 3] = x.w;
      }
      value_block<Gm, 0>(vr, ve, e, p, acc, G);
      value_block<Gm, 1>(vr, ve, e, p, acc, G);
      value_block<Gm, 2>(vr, ve, e, p, acc, G);
      value_block<Gm, 3>(vr, ve, e, p, acc, G);
    }
    wave_sync();
  }

  // the two token parities, then the waves in order
  __syncthreads();
#pragma unroll
  for (int g = 0; g < kMaxG; ++g) {
    if (g < G) {
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[g][k] += __shfl_xor(acc[g][k], 32);
      if (lane == 0) {
        mm[wave][g] = run_m[g];
        ml[wave][g] = run_l[g];
      }
      if (tp == 0) {
#pragma unroll
        for (int k = 0; k < 4; ++k) mo[wave][g][32 * k + e] = acc[g][k];
      }
    }
  }
  __syncthreads();
  float *part = a.work + (((int64_t)b * a.Hkv + kvh) * a.splits + split) * G * (kD + 2);
  for (int i = t; i < G * kD; i += kThreads) {
    const int g = i / kD, d = i - g * kD;
    float M = ninf;
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, mm[w][g]);
    float L = 0.f, O = 0.f;
    for (int w = 0; w < kWaves; ++w) {
      if (mm[w][g] == ninf) continue;     // a wave that had no chunk
      const float f = expf(mm[w][g] - M);
      L += ml[w][g] * f;
      O += mo[w][g][d] * f;
    }
    part[g * (kD + 2) + 2 + d] = O;
    if (d == 0) {
      part[g * (kD + 2)] = M;
      part[g * (kD + 2) + 1] = L;
    }
  }
}

// o[b][h] = the splits' partials merged in split order
__global__ __launch_bounds__(kD) void attn_combine_kernel(AttnArgs a) {
  const int d = threadIdx.x, h = blockIdx.x, b = blockIdx.y;
  const int G = a.G, kvh = h / G, g = h - kvh * G;
  const float *base = a.work + ((int64_t)b * a.Hkv + kvh) * a.splits * G * (kD + 2);
  float M = -__builtin_inff();
  for (int s = 0; s < a.splits; ++s) M = fmaxf(M, base[((int64_t)s * G + g) * (kD + 2)]);
  float L = 0.f, O = 0.f;
  for (int s = 0; s < a.splits; ++s) {
    const float *p = base + ((int64_t)s * G + g) * (kD + 2);
    const float f = expf(p[0] - M);
    L += p[1] * f;
    O += p[2 + d] * f;
  }
  a.o[((int64_t)b * a.Hq + h) * kD + d] = O / L;
}

template <int N4, int N6, int N8>
void launch_t(const AttnArgs &a, hipStream_t s) {
  hipLaunchKernelGGL((attn_decode_kernel<N4, N6, N8>),
                     dim3((unsigned)a.splits, (unsigned)a.Hkv, (unsigned)a.B), dim3(kThreads), 0,
                     s, a);
}

}  // namespace

int64_t attn_tokens_per_split(int64_t B, int64_t Hkv, int64_t T) {
  // about 512 workgroups (two per compute unit), whole chunks of 64 tokens
  const int64_t chunks = (T + 63) / 64;
  int64_t s = (512 + B * Hkv - 1) / (B * Hkv);
  if (s > chunks) s = chunks;
  if (s < 1) s = 1;
  return (chunks + s - 1) / s * 64;
}

hipError_t launch_attn_decode(const AttnArgs &a, hipStream_t s) {
  switch (a.n4 * 25 + a.n6 * 5 + a.n8) {
    case 100: launch_t<4, 0, 0>(a, s); break;
    case 80: launch_t<3, 1, 0>(a, s); break;
    case 76: launch_t<3, 0, 1>(a, s); break;
    case 60: launch_t<2, 2, 0>(a, s); break;
    case 56: launch_t<2, 1, 1>(a, s); break;
    case 52: launch_t<2, 0, 2>(a, s); break;
    case 40: launch_t<1, 3, 0>(a, s); break;
    case 36: launch_t<1, 2, 1>(a, s); break;
    case 32: launch_t<1, 1, 2>(a, s); break;
    case 28: launch_t<1, 0, 3>(a, s); break;
    case 20: launch_t<0, 4, 0>(a, s); break;
    case 16: launch_t<0, 3, 1>(a, s); break;
    case 12: launch_t<0, 2, 2>(a, s); break;
    case 8: launch_t<0, 1, 3>(a, s); break;
    case 4: launch_t<0, 0, 4>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_combine_kernel, dim3((unsigned)a.Hq, (unsigned)a.B), dim3(kD), 0, s, a);
  return hipGetLastError();
}

}  // namespace mxq
