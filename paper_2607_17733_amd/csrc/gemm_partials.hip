// gemm_partials.hip -- the exact integer block sums of the GEMM:
// P[i][j][b] = sum over the 32 elements t of block b of qa[i][t] * qw[j][t]
// (MXSens, arXiv 2607.17733, Section 2: the integer product of one block).
//
// A verification kernel, not on the hot path: one thread per (i, j, b)
// reads the mantissas from the canonical packed activation row and from the
// weight layout, and sums the 32 products in int32 (|P| < 2^19, exact).
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void gemm_partials_kernel(GemmArgs g) {
  const int nb = g.n4 + g.n6 + g.n8;
  const int64_t f = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (f >= g.M * g.N * nb) return;
  const int b = (int)(f % nb);
  const int64_t ij = f / nb;
  const int64_t i = ij / g.N, j = ij - i * g.N;
  const Segs s{g.n4, g.n6, g.n8, g.n3};
  const BlockInfo bi = block_info(s, b);
  const LGeo lg(g.n3, g.n4, g.n6, g.n8);
  const uint8_t *arow = g.a_mant + i * g.a_rb;
  int acc = 0;
  for (int t = 0; t < kBlock; ++t)
    acc += act_elem(arow, bi, t) * w_elem(g.w_mant, lg, g.full != 0, j, b, t);
  g.p[f] = acc;
}

}  // namespace

hipError_t launch_gemm_partials(const GemmArgs &a, hipStream_t stream) {
  const int64_t total = a.M * a.N * (a.n4 + a.n6 + a.n8);
  if (total <= 0) return hipSuccess;
  const unsigned grid = (unsigned)((total + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(gemm_partials_kernel, dim3(grid), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
