// quantize.hip -- fused MXINT quantize + bit-pack of bf16 rows.
//
// One kernel serves the online activation quantizer (canonical packed rows)
// and the offline weight packer (GEMM-tiled slabs).  MXSens (arXiv
// 2607.17733) Section 2 and Section 4.1: every 32-element block of the
// permuted row gets one shared exponent and one mantissa width.
//
// Work decomposition: a thread owns 8 consecutive elements of a block (a
// "group"), so the 4 threads of a block are adjacent lanes; the block
// maximum is a 2-step xor-shuffle reduction of integer |bf16| bit patterns.
// A workgroup owns one row (K >= 2048) or several whole rows (short K, e.g.
// the 128-wide KV-cache rows).  With a column permutation the workgroup first
// stages its source rows in LDS with 16-byte coalesced loads and gathers from
// LDS, so the permutation never turns into scattered global loads.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

constexpr int kThreads = 256;

template <bool WEIGHTS>
__global__ __launch_bounds__(kThreads) void quantize_kernel(QuantArgs q) {
  extern __shared__ uint16_t srow[];         // [rows_per_wg][K] when staged
  const int t = threadIdx.x;
  const int64_t K = q.K;
  const int nb = (int)(K / kBlock);
  const int G = 4 * nb;                      // groups per row
  const int R = q.rows_per_wg;
  const int64_t row0 = (int64_t)blockIdx.x * R;
  const Segs s{q.n4, q.n6, q.n8};

  // Stage the workgroup's source rows in LDS (permuted path only).
  if (q.stage) {
    const int64_t total = (int64_t)R * K;
    if (q.vec16) {
      for (int64_t v = t; v < total / 8; v += kThreads) {
        const int lr = (int)(v * 8 / K);
        const int64_t col = v * 8 - (int64_t)lr * K;
        const int64_t row = row0 + lr;
        uint4 d = make_uint4(0, 0, 0, 0);
        if (row < q.src_rows)
          d = *(const uint4 *)(q.src + row * q.ld + col);
        *(uint4 *)(srow + (int64_t)lr * K + col) = d;
      }
    } else {
      for (int64_t v = t; v < total; v += kThreads) {
        const int lr = (int)(v / K);
        const int64_t col = v - (int64_t)lr * K;
        const int64_t row = row0 + lr;
        srow[v] = row < q.src_rows ? q.src[row * q.ld + col] : (uint16_t)0;
      }
    }
    __syncthreads();
  }

  for (int64_t f = t; f < (int64_t)R * G; f += kThreads) {
    const int lr = (int)(f / G);
    const int g = (int)(f - (int64_t)lr * G);
    const int64_t row = row0 + lr;
    const bool live = row < q.out_rows;      // a whole block shares `live`
    const int b = g >> 2, kg = g & 3;
    const BlockInfo bi = block_info(s, b);

    // Gather the 8 source elements of the group.
    uint32_t bits[8];
    const int64_t p0 = (int64_t)b * kBlock + 8 * kg;
    if (!live || row >= q.src_rows) {
#pragma unroll
      for (int u = 0; u < 8; ++u) bits[u] = 0;
    } else if (q.perm) {
      const int4 pa = *(const int4 *)(q.perm + p0);
      const int4 pb = *(const int4 *)(q.perm + p0 + 4);
      const int src[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bool ok = src[u] >= 0 && (int64_t)src[u] < K;
        uint32_t v = 0;
        if (ok)
          v = q.stage ? srow[(int64_t)lr * K + src[u]]
                      : q.src[row * q.ld + src[u]];
        bits[u] = v;
      }
    } else if (q.vec16) {
      const uint4 d = *(const uint4 *)(q.src + row * q.ld + p0);
      const uint32_t w[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        bits[2 * u] = w[u] & 0xFFFFu;
        bits[2 * u + 1] = w[u] >> 16;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 8; ++u) bits[u] = q.src[row * q.ld + p0 + u];
    }

    // Block maximum of |x| on the integer bit patterns.
    uint32_t amax = 0;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t mag = bits[u] & 0x7FFFu;
      amax = mag > amax ? mag : amax;
    }
    uint32_t o = __shfl_xor(amax, 1);
    amax = o > amax ? o : amax;
    o = __shfl_xor(amax, 2);
    amax = o > amax ? o : amax;
    const int E = block_exponent(amax);

    int qv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      qv[u] = quant_elem(bits[u], E, bi.m, q.ties_away, q.full_clamp);

    const uint32_t nib = pack_nibbles(qv);
    uint32_t top = 0;
    if (bi.m == 6) {
      top = pack_top2(qv, kg & 1);
      top |= __shfl_xor(top, 1);             // merge the lane pair's word
    }
    if (!live) continue;

    if (!WEIGHTS) {
      uint8_t *dst = q.mant + row * q.out_rb + bi.aoff;
      if (bi.m == 4) {
        *(uint32_t *)(dst + 4 * kg) = nib;
      } else if (bi.m == 6) {
        *(uint32_t *)(dst + 4 * kg) = nib;
        if (!(kg & 1)) *(uint32_t *)(dst + 16 + 4 * (kg >> 1)) = top;
      } else {
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          lo |= ((uint32_t)qv[u] & 255u) << (8 * u);
          hi |= ((uint32_t)qv[4 + u] & 255u) << (8 * u);
        }
        *(uint2 *)(dst + 8 * kg) = make_uint2(lo, hi);
      }
      if (kg == 0) q.exp[row * q.out_erb + b] = (uint8_t)E;
      if (g == 0) {                          // zero the row padding
        for (int64_t z = q.row_used; z < q.out_rb; ++z)
          q.mant[row * q.out_rb + z] = 0;
        for (int64_t z = nb; z < q.out_erb; ++z) q.exp[row * q.out_erb + z] = 0;
      }
    } else {
      const int64_t slab = row >> 4;
      const int c = (int)(row & 15);
      uint8_t *base = q.mant + slab * slab_bytes(s);
      const WLoc w = w_loc(s, bi, kg, c);
      if (bi.m == 4) {
        *(uint32_t *)(base + w.lo) = nib;
      } else if (bi.m == 6) {
        *(uint32_t *)(base + w.lo) = nib;
        if (!(kg & 1)) *(uint32_t *)(base + w.hi) = top;
      } else {
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          lo |= ((uint32_t)qv[u] & 255u) << (8 * u);
          hi |= ((uint32_t)qv[4 + u] & 255u) << (8 * u);
        }
        *(uint32_t *)(base + w.lo) = lo;
        *(uint32_t *)(base + w.lo + 4) = hi;
      }
      if (kg == 0) q.exp[(int64_t)b * q.out_rows + row] = (uint8_t)E;
    }
  }
}

}  // namespace

hipError_t launch_quantize(const QuantArgs &args, bool weights,
                           hipStream_t stream) {
  const int64_t K = args.K;
  const int nb = (int)(K / kBlock);
  const int G = 4 * nb;
  QuantArgs a = args;
  a.rows_per_wg = G >= kThreads ? 1 : kThreads / G;
  const int64_t lds = a.stage ? (int64_t)a.rows_per_wg * K * 2 : 0;
  const int64_t grid = (a.out_rows + a.rows_per_wg - 1) / a.rows_per_wg;
  if (grid <= 0) return hipSuccess;
  if (weights)
    hipLaunchKernelGGL(quantize_kernel<true>, dim3((unsigned)grid), dim3(kThreads),
                       (size_t)lds, stream, a);
  else
    hipLaunchKernelGGL(quantize_kernel<false>, dim3((unsigned)grid), dim3(kThreads),
                       (size_t)lds, stream, a);
  return hipGetLastError();
}

}  // namespace mxq
