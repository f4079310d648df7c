// unpack.hip -- debug decode of the stored mantissas back to int8 values in
// permuted order, plus the exponents: the canonical packed activation rows,
// and the weight layout of the GEMMs.  Used for parity checks; not on the
// hot path.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

constexpr int kThreads = 256;

// One thread per (row, block): the 32 mantissas and the exponent.
template <bool WEIGHTS>
__global__ __launch_bounds__(kThreads) void unpack_kernel(UnpackArgs a) {
  const int nb = (int)(a.K / kBlock);
  const int64_t f = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (f >= a.rows * nb) return;
  const int64_t row = f / nb;
  const int b = (int)(f - row * nb);
  int8_t *out = a.q + row * a.K + (int64_t)b * kBlock;
  if (!WEIGHTS) {
    const Segs s{a.n4, a.n6, a.n8, a.n3};
    const BlockInfo bi = block_info(s, b);
    const uint8_t *p = a.mant + row * a.a_rb;
    for (int t = 0; t < kBlock; ++t) out[t] = (int8_t)act_elem(p, bi, t);
    a.e[row * nb + b] = a.exp[row * a.a_erb + b];
  } else {
    const LGeo lg(a.n3, a.n4, a.n6, a.n8);
    for (int t = 0; t < kBlock; ++t) out[t] = (int8_t)w_elem(a.mant, lg, a.full != 0, row, b, t);
    a.e[row * nb + b] = (uint8_t)w_exp_of(a.exp, lg, row, b);
  }
}

}  // namespace

hipError_t launch_unpack(const UnpackArgs &a, bool weights, hipStream_t stream) {
  const int64_t total = a.rows * (a.K / kBlock);
  if (total <= 0) return hipSuccess;
  const unsigned grid = (unsigned)((total + kThreads - 1) / kThreads);
  if (weights)
    hipLaunchKernelGGL(unpack_kernel<true>, dim3(grid), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(unpack_kernel<false>, dim3(grid), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
