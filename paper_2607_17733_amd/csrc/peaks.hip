// peaks.hip -- achievable-peak microbenchmarks for the roofline figures.
//
// Not part of the quantize / GEMM path: the benchmark prices its kernels
// against the datasheet peaks and against what these loops reach on the
// same box.
//   stream read: every byte of a buffer read once with 16-byte
//     non-temporal loads, four in flight per thread, sixteen waves per CU;
//   matrix-core loops: register-resident operands, eight independent
//     accumulators per wave, sixteen waves per CU, for the dense int8
//     32x32x32 product and the block-scaled 32x32x64 FP6 (e3m2) and FP8
//     (e4m3) products the prefill GEMM issues.
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef unsigned u4 __attribute__((ext_vector_type(4)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kPeakThreads = 256;
constexpr int kPeakBlocks = 4096;   // 16 waves per CU on 256 CUs, four rounds

__global__ __launch_bounds__(kPeakThreads) void stream_read_kernel(const u4 *__restrict__ p,
                                                                   int64_t n, uint32_t *sink) {
  const int64_t stride = (int64_t)gridDim.x * kPeakThreads * 4;
  u4 acc = {0u, 0u, 0u, 0u};
  for (int64_t i = (int64_t)blockIdx.x * kPeakThreads * 4 + threadIdx.x; i < n; i += stride) {
    u4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t j = i + u * kPeakThreads;
      v[u] = j < n ? __builtin_nontemporal_load(p + j) : u4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= v[u];
  }
  sink[(int64_t)blockIdx.x * kPeakThreads + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

// KIND 0: int8 32x32x32; 1: FP6 32x32x64 (block-scaled); 2: FP8 32x32x64.
template <int KIND>
__global__ __launch_bounds__(kPeakThreads) void mfma_loop_kernel(int64_t iters, float *sink) {
  const int t = threadIdx.x;
  float s = 0.f;
  if (KIND == 0) {
    const v4i a = {t, t + 1, t + 2, t + 3}, b = {t ^ 5, t ^ 6, t ^ 7, t ^ 9};
    v16i c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = v16i{};
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
      for (int i = 0; i < 8; ++i) c[i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c[i], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) s += (float)c[i][t & 15];
  } else {
    constexpr int kFmt = KIND == 1 ? 3 : 0;
    // bytes below 0x40: finite FP8 codes (no e4m3 NaN), small FP6 values
    const int m = 0x3F3F3F3F;
    const v8i a = {t & m, (t + 1) & m, (t + 2) & m, (t + 3) & m, (t + 4) & m, (t + 5) & m,
                   (t + 6) & m, (t + 7) & m};
    const v8i b = {(t ^ 5) & m, (t ^ 6) & m, (t ^ 7) & m, (t ^ 9) & m, (t ^ 3) & m, (t ^ 1) & m,
                   (t ^ 2) & m, (t ^ 4) & m};
    v16f c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = v16f{};
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        c[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c[i], kFmt, kFmt, 0, 127, 0,
                                                               127);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) s += c[i][t & 15];
  }
  sink[(int64_t)blockIdx.x * kPeakThreads + t] = s;
}

}  // namespace

int64_t peak_sink_words() { return (int64_t)kPeakBlocks * kPeakThreads; }

int64_t peak_mfma_ops(int kind, int64_t iters) {
  const int64_t per = kind == 0 ? 2LL * 32 * 32 * 32 : 2LL * 32 * 32 * 64;
  return per * 8 * iters * (int64_t)kPeakBlocks * (kPeakThreads / 64);
}

hipError_t launch_peak_stream(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t s) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(kPeakBlocks), dim3(kPeakThreads), 0, s,
                     (const u4 *)buf, bytes / 16, sink);
  return hipGetLastError();
}

hipError_t launch_peak_mfma(int kind, int64_t iters, float *sink, hipStream_t s) {
  if (kind == 0)
    hipLaunchKernelGGL(mfma_loop_kernel<0>, dim3(kPeakBlocks), dim3(kPeakThreads), 0, s, iters,
                       sink);
  else if (kind == 1)
    hipLaunchKernelGGL(mfma_loop_kernel<1>, dim3(kPeakBlocks), dim3(kPeakThreads), 0, s, iters,
                       sink);
  else
    hipLaunchKernelGGL(mfma_loop_kernel<2>, dim3(kPeakBlocks), dim3(kPeakThreads), 0, s, iters,
                       sink);
  return hipGetLastError();
}

}  // namespace mxq
