// decode.hip -- MXINT GEMM for decode shapes (M <= 16): streams the packed
// weights.
//
// Y[i][j] = sum_b P[i][j][b] * 2^(sa[i][b] + sw[j][b])   (MXSens, arXiv
// 2607.17733, Section 2: integer block products, power-of-two block scales).
// Each 32-wide block is one V_MFMA_I32_16X16X32_I8 (exact int32), rescaled
// in fp32 with 2^(Ea + Ew - 266) (every width is unpacked to the top of the
// int8 byte).
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

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
    const float sw = block_scale(g.w_exp[col * g.w_erb + b]);
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

hipError_t launch_gemm_decode(const GemmArgs &a, hipStream_t stream) {
  dim3 grid((unsigned)(a.npad / 16));
  hipLaunchKernelGGL(gemm_decode_kernel, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
