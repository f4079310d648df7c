// gemm.hip -- MXINT GEMM on int8 matrix cores (prefill tiling) and the
// per-block int32 partial-sum kernel.
//
// Y[i][j] = sum_b P[i][j][b] * 2^(sa[i][b] + sw[j][b])   (MXSens, arXiv
// 2607.17733, Section 2: integer block products, power-of-two block scales;
// Section 6: mixed widths on an integer datapath).
//
// Each 32-wide block is one V_MFMA_I32_16X16X32_I8 per 16x16 output tile, so
// its int32 sum is exact.  Packed 4/6/8-bit mantissas of both operands are
// unpacked to int8 (placed at the top of the byte) into LDS once per
// workgroup tile and read back as matrix-core operands; every width takes
// the same scale formula 2^(Ea + Ew - 266).
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, kThreads = 256;

template <bool PARTIALS>
__global__ __launch_bounds__(kThreads) void gemm_prefill_kernel(GemmArgs g) {
  __shared__ uint64_t As[BM][4];
  __shared__ uint64_t Ws[BN][4];
  __shared__ float Sa[BM], Sw[BN];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t row0 = (int64_t)blockIdx.y * BM, col0 = (int64_t)blockIdx.x * BN;
  const int wm = wave >> 1, wn = wave & 1;
  const int i16 = lane & 15, kq = lane >> 4;
  const Segs s{g.n4, g.n6, g.n8};
  const int nb = g.n4 + g.n6 + g.n8;
  const int64_t sbytes = slab_bytes(s);

  float acc[4][4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[a][b][r] = 0.f;

  for (int b = 0; b < nb; ++b) {
    const BlockInfo bi = block_info(s, b);
    __syncthreads();
    {
      const int r = t >> 1;
      const int64_t i = row0 + r;
      const int64_t j = col0 + r;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int kg = (t & 1) * 2 + h;
        As[r][kg] = i < g.M ? load_act_operand(g.a_mant + i * g.a_rb, bi, kg) : 0;
        Ws[r][kg] = j < g.npad
                        ? load_w_operand(g.w_mant + (j >> 4) * sbytes, s, bi, kg,
                                         (int)(j & 15))
                        : 0;
      }
      if (t < BM) {
        const int64_t ii = row0 + t;
        Sa[t] = ii < g.M ? block_scale(g.a_exp[ii * g.a_erb + b]) : 0.f;
      } else {
        const int64_t jj = col0 + (t - BM);
        Sw[t - BM] = jj < g.npad ? block_scale(g.w_exp[(int64_t)b * g.npad + jj]) : 0.f;
      }
    }
    __syncthreads();

    long af[4], wf[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) af[m] = (long)As[wm * 64 + m * 16 + i16][kq];
#pragma unroll
    for (int n = 0; n < 4; ++n) wf[n] = (long)Ws[wn * 64 + n * 16 + i16][kq];
    const int shift = 2 * (8 - bi.m);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        const v4i zero = {0, 0, 0, 0};
        const v4i P = __builtin_amdgcn_mfma_i32_16x16x32_i8(af[m], wf[n], zero, 0, 0, 0);
        const int cl = wn * 64 + n * 16 + i16;
        if (PARTIALS) {
          const int64_t j = col0 + cl;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int64_t i = row0 + wm * 64 + m * 16 + kq * 4 + r;
            if (i < g.M && j < g.N)
              g.p[(i * g.N + j) * nb + b] = P[r] >> shift;
          }
        } else {
          const float sw = Sw[cl];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float sa = Sa[wm * 64 + m * 16 + kq * 4 + r];
            acc[m][n][r] += (float)P[r] * (sa * sw);
          }
        }
      }
    }
  }
  if (PARTIALS) return;
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t j = col0 + wn * 64 + n * 16 + i16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t i = row0 + wm * 64 + m * 16 + kq * 4 + r;
        if (i < g.M && j < g.N) g.y[i * g.ldy + j] = acc[m][n][r];
      }
    }
}

// Decode shapes (M <= 16): one workgroup per 16-column weight slab, its four
// waves splitting the slab's blocks; the 16 activation rows fill one matrix
// core tile.  The waves' fp32 partials are reduced through LDS.
__global__ __launch_bounds__(kThreads) void gemm_decode_kernel(GemmArgs g) {
  __shared__ float red[4][64][4];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int i16 = lane & 15, kq = lane >> 4;
  const int64_t slab = blockIdx.x;
  const Segs s{g.n4, g.n6, g.n8};
  const int nb = g.n4 + g.n6 + g.n8;
  const uint8_t *wslab = g.w_mant + slab * slab_bytes(s);
  const int64_t col = slab * 16 + i16;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int b = wave; b < nb; b += 4) {
    const BlockInfo bi = block_info(s, b);
    const long av = i16 < g.M ? (long)load_act_operand(g.a_mant + i16 * g.a_rb, bi, kq) : 0;
    const long wv = (long)load_w_operand(wslab, s, bi, kq, i16);
    const v4i zero = {0, 0, 0, 0};
    const v4i P = __builtin_amdgcn_mfma_i32_16x16x32_i8(av, wv, zero, 0, 0, 0);
    const float sw = block_scale(g.w_exp[(int64_t)b * g.npad + col]);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = kq * 4 + r;
      const float sa = row < g.M ? block_scale(g.a_exp[row * g.a_erb + b]) : 0.f;
      acc[r] += (float)P[r] * (sa * sw);
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) red[wave][lane][r] = acc[r];
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float v = red[0][lane][r] + red[1][lane][r] + red[2][lane][r] +
                      red[3][lane][r];
      const int row = kq * 4 + r;
      if (row < g.M && col < g.N) g.y[row * g.ldy + col] = v;
    }
  }
}

}  // namespace

hipError_t launch_gemm_prefill(const GemmArgs &a, hipStream_t stream) {
  dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + BM - 1) / BM));
  hipLaunchKernelGGL(gemm_prefill_kernel<false>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_gemm_partials(const GemmArgs &a, hipStream_t stream) {
  dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + BM - 1) / BM));
  hipLaunchKernelGGL(gemm_prefill_kernel<true>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_gemm_decode(const GemmArgs &a, hipStream_t stream) {
  dim3 grid((unsigned)(a.npad / 16));
  hipLaunchKernelGGL(gemm_decode_kernel, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
