// unpack.hip -- debug decode of packed MXINT mantissas back to canonical
// int8 values in permuted order, plus the exponents.  Used for parity
// checks of the packed activation rows and the weight slabs; not on the hot
// path.
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
  const Segs s{a.n4, a.n6, a.n8};
  const BlockInfo bi = block_info(s, b);
  int8_t *out = a.q + row * a.K + (int64_t)b * kBlock;
  if (!WEIGHTS) {
    const uint8_t *p = a.mant + row * a.a_rb;
    for (int t = 0; t < kBlock; ++t) out[t] = (int8_t)act_elem(p, bi, t);
  } else {
    const DGeo dg(a.n4, a.n6, a.n8);
    const uint8_t *slab = a.mant + (row >> 4) * wd_slab_bytes(dg);
    for (int t = 0; t < kBlock; ++t)
      out[t] = (int8_t)wstream_elem(slab, dg, bi, (int)(row & 15), t, a.sm != 0);
  }
  a.e[row * nb + b] = a.exp[row * a.a_erb + b];
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
