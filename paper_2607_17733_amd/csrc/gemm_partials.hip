// gemm_partials.hip -- the exact integer block sums of the GEMM:
// P[i][j][b] = sum over the 32 elements k of block b of qa[i][k] * qw[j][k]
// (MXSens, arXiv 2607.17733, Section 2: the integer product of one block).
//
// A verification kernel, not on the hot path: one wave per 16x16 output
// tile walks every block with one V_MFMA_I32_16X16X32_I8 (exact int32) over
// mantissas unpacked from the packed activation row and the packed weight
// slab.  The unpacked operands sit at the top of the int8 byte (each carries
// 2^(8 - m)), so the int32 result is shifted right by 2(8 - m), exactly.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(64) void gemm_partials_kernel(GemmArgs g) {
  const int lane = threadIdx.x, i16 = lane & 15, kq = lane >> 4;
  const int64_t slab = blockIdx.x, rt = blockIdx.y;
  const Segs s{g.n4, g.n6, g.n8};
  const int nb = g.n4 + g.n6 + g.n8;
  const uint8_t *wslab = g.w_mant + slab * slab_bytes(s);
  const int64_t arow = rt * 16 + i16;
  const uint8_t *ap = g.a_mant + (arow < g.M ? arow : g.M - 1) * g.a_rb;
  const int64_t col = slab * 16 + i16;
  for (int b = 0; b < nb; ++b) {
    const BlockInfo bi = block_info(s, b);
    const long av = (long)load_act_operand(ap, bi, kq);
    const long wv = (long)load_w_operand(wslab, s, bi, kq, i16);
    const v4i zero = {0, 0, 0, 0};
    const v4i P = __builtin_amdgcn_mfma_i32_16x16x32_i8(av, wv, zero, 0, 0, 0);
    const int sh = 2 * (8 - bi.m);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t i = rt * 16 + kq * 4 + r;
      if (i < g.M && col < g.N) g.p[(i * g.N + col) * nb + b] = P[r] >> sh;
    }
  }
}

}  // namespace

hipError_t launch_gemm_partials(const GemmArgs &a, hipStream_t stream) {
  dim3 grid((unsigned)(a.npad / 16), (unsigned)((a.M + 15) / 16));
  hipLaunchKernelGGL(gemm_partials_kernel, grid, dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
