// calib.hip -- on-GPU calibration: the offline step that produces the
// path's inputs, the column permutation and the per-block width map.
//
// MXSens (arXiv 2607.17733), Section 3, Algorithm 1: a column's sensitivity
// is the diagonal of the Hessian approximation H = sum over calibration
// samples of X^T X, i.e. the sum of its squared activations.  Section 4.2,
// Algorithm 2: sort a layer's columns by descending sensitivity; the top 32
// get 8-bit mantissas, the next N6 6-bit, the rest 4-bit.
//
// Sensitivities are float64 and computed in a fixed order, one thread per
// column: a sample's rows are summed in row order from zero (every square of
// a bf16 value is exact in float64), and the sample's sum is then added to
// the running total.  The sort is by counting: a column's rank is the number
// of columns that sort before it (larger sensitivity, or equal with a lower
// index; a NaN counts as +inf), which fixes a unique order without a
// parallel sort.  The rank then places the column in the permutation: the
// 4-bit columns first, then the 6-bit and the 8-bit ones, each in sorted
// order.
#include "mxq_internal.h"

namespace mxq {

namespace {

constexpr int kCalThreads = 256;

__device__ inline double bf16_to_f64(uint16_t v) {
  return (double)__uint_as_float((uint32_t)v << 16);
}

__global__ __launch_bounds__(kCalThreads) void colsq_kernel(const uint16_t *__restrict__ x,
                                                            int64_t rows, int64_t ld, int64_t K,
                                                            double *s, int accumulate) {
  const int64_t k = (int64_t)blockIdx.x * kCalThreads + threadIdx.x;
  if (k >= K) return;
  const uint16_t *p = x + k;
  double part = 0.0;
  int64_t r = 0;
  for (; r + 8 <= rows; r += 8) {
    uint16_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = p[(r + u) * ld];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const double d = bf16_to_f64(v[u]);
      part += d * d;
    }
  }
  for (; r < rows; ++r) {
    const double d = bf16_to_f64(p[r * ld]);
    part += d * d;
  }
  s[k] = accumulate ? s[k] + part : part;
}

// Several samples at once (blockIdx.y = sample): each sample's sums, in row
// order, go to its row of `part`; then the samples are added in order.
__global__ __launch_bounds__(kCalThreads) void colsq_samples_kernel(
    const uint16_t *__restrict__ x, int64_t rows, int64_t ld, int64_t sample_stride, int64_t K,
    double *part) {
  const int64_t k = (int64_t)blockIdx.x * kCalThreads + threadIdx.x;
  if (k >= K) return;
  const uint16_t *p = x + (int64_t)blockIdx.y * sample_stride + k;
  double sum = 0.0;
  int64_t r = 0;
  for (; r + 8 <= rows; r += 8) {
    uint16_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = p[(r + u) * ld];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const double d = bf16_to_f64(v[u]);
      sum += d * d;
    }
  }
  for (; r < rows; ++r) {
    const double d = bf16_to_f64(p[r * ld]);
    sum += d * d;
  }
  part[(int64_t)blockIdx.y * K + k] = sum;
}

__global__ __launch_bounds__(kCalThreads) void add_samples_kernel(const double *__restrict__ part,
                                                                  int64_t n, int64_t K, double *s,
                                                                  int accumulate) {
  const int64_t k = (int64_t)blockIdx.x * kCalThreads + threadIdx.x;
  if (k >= K) return;
  double acc = accumulate ? s[k] + part[k] : part[k];
  for (int64_t i = 1; i < n; ++i) acc = acc + part[i * K + k];
  s[k] = acc;
}

__device__ inline double sort_key(double v) { return v != v ? __builtin_inf() : v; }

__global__ __launch_bounds__(kCalThreads) void rank_perm_kernel(const double *__restrict__ s,
                                                                int64_t K, int64_t n4,
                                                                int64_t n6, int64_t n8,
                                                                int32_t *perm) {
  __shared__ double tile[kCalThreads];
  const int t = threadIdx.x;
  const int64_t i = (int64_t)blockIdx.x * kCalThreads + t;
  const double si = i < K ? sort_key(s[i]) : 0.0;
  int64_t before = 0;
  for (int64_t j0 = 0; j0 < K; j0 += kCalThreads) {
    __syncthreads();
    if (j0 + t < K) tile[t] = sort_key(s[j0 + t]);
    __syncthreads();
    const int jn = (int)(K - j0 < kCalThreads ? K - j0 : kCalThreads);
    for (int jj = 0; jj < jn; ++jj) {
      const double sj = tile[jj];
      before += (sj > si) || (sj == si && j0 + jj < i);
    }
  }
  if (i >= K) return;
  const int64_t c8 = 32 * n8, c6 = 32 * n6, c4 = 32 * n4;
  int64_t pos;
  if (before < c8) pos = c4 + c6 + before;                   // 8-bit: the last blocks
  else if (before < c8 + c6) pos = c4 + (before - c8);       // 6-bit
  else pos = before - c8 - c6;                               // 4-bit: the first blocks
  perm[pos] = (int32_t)i;
}

}  // namespace

hipError_t launch_calib_colsq(const uint16_t *x, int64_t rows, int64_t ld, int64_t K, double *s,
                              bool accumulate, hipStream_t stream) {
  const int64_t blocks = (K + kCalThreads - 1) / kCalThreads;
  hipLaunchKernelGGL(colsq_kernel, dim3((unsigned)blocks), dim3(kCalThreads), 0, stream, x, rows,
                     ld, K, s, accumulate ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_calib_colsq_samples(const uint16_t *x, int64_t n, int64_t rows, int64_t ld,
                                      int64_t sample_stride, int64_t K, double *part, double *s,
                                      bool accumulate, hipStream_t stream) {
  const int64_t blocks = (K + kCalThreads - 1) / kCalThreads;
  hipLaunchKernelGGL(colsq_samples_kernel, dim3((unsigned)blocks, (unsigned)n), dim3(kCalThreads),
                     0, stream, x, rows, ld, sample_stride, K, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(add_samples_kernel, dim3((unsigned)blocks), dim3(kCalThreads), 0, stream,
                     part, n, K, s, accumulate ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_calib_perm(const double *s, int64_t K, int64_t n6, int64_t n8, int32_t *perm,
                             hipStream_t stream) {
  const int64_t blocks = (K + kCalThreads - 1) / kCalThreads;
  hipLaunchKernelGGL(rank_perm_kernel, dim3((unsigned)blocks), dim3(kCalThreads), 0, stream, s,
                     K, K / 32 - n6 - n8, n6, n8, perm);
  return hipGetLastError();
}

}  // namespace mxq
