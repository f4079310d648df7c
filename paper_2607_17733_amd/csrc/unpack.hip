// unpack.hip -- debug decode of packed MXINT mantissas back to canonical
// int8 values in permuted order, plus the exponents.  Used for parity
// checks of the packed activation and weight layouts; not on the hot path.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

constexpr int kThreads = 256;

__device__ inline int sext(uint32_t v, int bits) {
  const int sh = 32 - bits;
  return ((int)(v << sh)) >> sh;
}

// Decode the 8 elements of one lane group from its nibble dword / top-bit
// word / raw bytes into canonical order.
__device__ inline void decode_group(int m, uint32_t lo, uint32_t hi_or_top,
                                    int8_t *out) {
  if (m == 8) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      out[u] = (int8_t)(lo >> (8 * u));
      out[4 + u] = (int8_t)(hi_or_top >> (8 * u));
    }
    return;
  }
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint32_t nib = (lo >> (4 * u)) & 15u;
    if (m == 4) {
      out[u] = (int8_t)sext(nib, 4);
    } else {
      // top bits of element u of this (even-aligned) group: byte u/2,
      // bits 6-7 for even u and 4-5 for odd u
      const uint32_t top = (hi_or_top >> (8 * (u >> 1) + ((u & 1) ? 4 : 6))) & 3u;
      out[u] = (int8_t)sext(nib | (top << 4), 6);
    }
  }
}

template <bool WEIGHTS>
__global__ __launch_bounds__(kThreads) void unpack_kernel(UnpackArgs a) {
  const int nb = (int)(a.K / kBlock);
  const int64_t f = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (f >= a.rows * 4 * nb) return;
  const int64_t row = f / (4 * nb);
  const int g = (int)(f - row * 4 * nb);
  const int b = g >> 2, kg = g & 3;
  const Segs s{a.n4, a.n6, a.n8};
  const BlockInfo bi = block_info(s, b);
  uint32_t lo, second = 0;
  uint8_t E;
  if (!WEIGHTS) {
    const uint8_t *p = a.mant + row * a.a_rb + bi.aoff;
    if (bi.m == 8) {
      lo = *(const uint32_t *)(p + 8 * kg);
      second = *(const uint32_t *)(p + 8 * kg + 4);
    } else {
      lo = *(const uint32_t *)(p + 4 * kg);
      if (bi.m == 6) second = *(const uint32_t *)(p + 16 + 4 * (kg >> 1));
    }
    E = a.exp[row * a.a_erb + b];
  } else {
    const uint8_t *slab = a.mant + (row >> 4) * slab_bytes(s);
    const WLoc w = w_loc(s, bi, kg, (int)(row & 15));
    lo = *(const uint32_t *)(slab + w.lo);
    if (bi.m == 8) second = *(const uint32_t *)(slab + w.lo + 4);
    if (bi.m == 6) second = *(const uint32_t *)(slab + w.hi);
    E = a.exp[row * a.a_erb + b];
  }
  if (bi.m == 6 && (kg & 1)) second <<= 4;
  int8_t out[8];
  decode_group(bi.m, lo, second, out);
#pragma unroll
  for (int u = 0; u < 8; ++u) a.q[row * a.K + (int64_t)b * kBlock + 8 * kg + u] = out[u];
  if (kg == 0) a.e[row * nb + b] = E;
}

}  // namespace

hipError_t launch_unpack(const UnpackArgs &a, bool weights, hipStream_t stream) {
  const int64_t total = a.rows * 4 * (a.K / kBlock);
  if (total <= 0) return hipSuccess;
  const unsigned grid = (unsigned)((total + kThreads - 1) / kThreads);
  if (weights)
    hipLaunchKernelGGL(unpack_kernel<true>, dim3(grid), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(unpack_kernel<false>, dim3(grid), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
