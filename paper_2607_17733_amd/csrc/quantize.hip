// quantize.hip -- fused MXINT quantize + bit-pack of bf16 rows.
//
// One kernel serves the online activation quantizer and the offline weight
// packer.  MXSens (arXiv 2607.17733) Section 2 and Section 4.1: every
// 32-element block of the permuted row gets one shared exponent and one
// mantissa width.
//
// Work decomposition: a thread owns 8 consecutive elements of a block (a
// "group"), so the 4 threads of a block are adjacent lanes; the block
// maximum is a 2-step xor-shuffle reduction of integer |bf16| bit patterns.
// A workgroup owns one row (K >= 2048) or several whole rows (short K, e.g.
// the 128-wide KV-cache rows).  With a column permutation the workgroup first
// stages its source rows in LDS with 16-byte coalesced loads and gathers from
// LDS, so the permutation never turns into scattered global loads.
//
// Activations additionally get a matrix-core operand image (second pass):
// every mantissa unpacked to int8 and shifted to a per-(row, chunk) reference
// exponent, so the prefill GEMM reads ready operands instead of unpacking the
// same row once per column tile.  A chunk is up to 16 blocks of one width; its
// blocks share the reference ref = max E when max E - min E <= 8 - m (the
// spare top bits of the byte), else each block keeps ref = E.  The operand of
// element q is q * 2^(8 - m - (ref - E)), exact, and the block's value is
// operand * 2^(ref - 133).
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

constexpr int kThreads = 256;
constexpr int kChunk = 16;

// Arithmetic right shift of every byte of v by s in [0, 4] (low s bits of
// every byte are zero).
__device__ inline uint32_t sar8(uint32_t v, uint32_t s) {
  const uint32_t S = v & 0x80808080u;
  return (v >> s) | ((S - (S >> s)) << 1);
}

template <bool WEIGHTS>
__global__ __launch_bounds__(kThreads) void quantize_kernel(QuantArgs q) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int t = threadIdx.x;
  const int64_t K = q.K;
  const int nb = (int)(K / kBlock);
  const int G = 4 * nb;                      // groups per row
  const int R = q.rows_per_wg;
  const int64_t row0 = (int64_t)blockIdx.x * R;
  const Segs s{q.n4, q.n6, q.n8};
  // LDS: [R][K] staged bf16 source (permuted path), then for activations
  // [R][K] int8 mantissas, [R][nb] exponents, [R][nb] reference exponents.
  uint16_t *srow = (uint16_t *)smem;
  int8_t *qrow = (int8_t *)(smem + (q.stage ? (int64_t)R * K * 2 : 0));
  uint8_t *erow = (uint8_t *)(qrow + (WEIGHTS ? 0 : (int64_t)R * K));
  uint8_t *rrow = erow + (int64_t)R * nb;

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

    uint32_t lo8 = 0, hi8 = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      lo8 |= ((uint32_t)qv[u] & 255u) << (8 * u);
      hi8 |= ((uint32_t)qv[4 + u] & 255u) << (8 * u);
    }
    if (!WEIGHTS) {
      uint8_t *dst = q.mant + row * q.out_rb + bi.aoff;
      if (bi.m == 4) {
        *(uint32_t *)(dst + 4 * kg) = nib;
      } else if (bi.m == 6) {
        *(uint32_t *)(dst + 4 * kg) = nib;
        if (!(kg & 1)) *(uint32_t *)(dst + 16 + 4 * (kg >> 1)) = top;
      } else {
        *(uint2 *)(dst + 8 * kg) = make_uint2(lo8, hi8);
      }
      if (kg == 0) q.exp[row * q.out_erb + b] = (uint8_t)E;
      if (g == 0) {                          // zero the row padding
        for (int64_t z = q.row_used; z < q.canon_rb; ++z)
          q.mant[row * q.out_rb + z] = 0;
        for (int64_t z = nb; z < q.canon_erb; ++z) {
          q.exp[row * q.out_erb + z] = 0;
          q.exp[row * q.out_erb + q.canon_erb + z] = 0;
        }
      }
      // keep the mantissas and the exponent for the operand pass
      *(uint2 *)(qrow + (int64_t)lr * K + p0) = make_uint2(lo8, hi8);
      if (kg == 0) erow[lr * nb + b] = (uint8_t)E;
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
        *(uint32_t *)(base + w.lo) = lo8;
        *(uint32_t *)(base + w.lo + 4) = hi8;
      }
      if (kg == 0) q.exp[row * q.out_erb + b] = (uint8_t)E;
      if (g == 0)                            // zero the exponent row padding
        for (int64_t z = nb; z < q.out_erb; ++z) q.exp[row * q.out_erb + z] = 0;
      if (row == 0 && g == 0)                // and the buffer's tail padding
        for (int z = 0; z < q.tail_pad; ++z)
          q.mant[(q.out_rows >> 4) * slab_bytes(s) + z] = 0;
    }
  }
  if (WEIGHTS) return;

  // ---- operand image: chunk references, then shifted int8 operands.
  __syncthreads();
  const int c4 = (q.n4 + kChunk - 1) / kChunk, c6 = (q.n6 + kChunk - 1) / kChunk;
  const int nch = c4 + c6 + (q.n8 + kChunk - 1) / kChunk;
  for (int f = t; f < R * nch; f += kThreads) {
    const int lr = f / nch, c = f - lr * nch;
    int b0, b1, H;
    if (c < c4) { b0 = c * kChunk; b1 = min(q.n4, b0 + kChunk); H = 4; }
    else if (c < c4 + c6) { b0 = q.n4 + (c - c4) * kChunk; b1 = min(q.n4 + q.n6, b0 + kChunk); H = 2; }
    else { b0 = q.n4 + q.n6 + (c - c4 - c6) * kChunk; b1 = min(nb, b0 + kChunk); H = 0; }
    int emin = 255, emax = 0;
    for (int b = b0; b < b1; ++b) {
      const int e = erow[lr * nb + b];
      emin = min(emin, e);
      emax = max(emax, e);
    }
    const bool shared = emax - emin <= H;
    for (int b = b0; b < b1; ++b)
      rrow[lr * nb + b] = (uint8_t)(shared ? emax : erow[lr * nb + b]);
  }
  __syncthreads();
  for (int64_t f = t; f < (int64_t)R * G; f += kThreads) {
    const int lr = (int)(f / G);
    const int g = (int)(f - (int64_t)lr * G);
    const int64_t row = row0 + lr;
    if (row >= q.out_rows) continue;
    const int b = g >> 2, kg = g & 3;
    const BlockInfo bi = block_info(s, b);
    const int E = erow[lr * nb + b], ref = rrow[lr * nb + b];
    const uint32_t sh = (uint32_t)(ref - E);
    const uint2 qq = *(const uint2 *)(qrow + (int64_t)lr * K + (int64_t)b * kBlock + 8 * kg);
    uint32_t ev, od;
    if (bi.m == 8) {
      ev = qq.x;
      od = qq.y;
    } else {
      // even / odd elements of the group, placed at the top of the byte
      ev = __builtin_amdgcn_perm(qq.y, qq.x, 0x06040200u);
      od = __builtin_amdgcn_perm(qq.y, qq.x, 0x07050301u);
      if (bi.m == 4) {
        ev = sar8((ev << 4) & 0xF0F0F0F0u, sh);
        od = sar8((od << 4) & 0xF0F0F0F0u, sh);
      } else {
        ev = sar8((ev << 2) & 0xFCFCFCFCu, sh);
        od = sar8((od << 2) & 0xFCFCFCFCu, sh);
      }
    }
    *(uint2 *)(q.mant + row * q.out_rb + q.canon_rb + (int64_t)b * kBlock + 8 * kg) =
        make_uint2(ev, od);
    if (kg == 0) q.exp[row * q.out_erb + q.canon_erb + b] = (uint8_t)ref;
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
  const int64_t grid = (a.out_rows + a.rows_per_wg - 1) / a.rows_per_wg;
  if (grid <= 0) return hipSuccess;
  if (weights) {
    const int64_t lds = a.stage ? (int64_t)a.rows_per_wg * K * 2 : 0;
    if (lds > kMaxLds) return hipErrorInvalidValue;
    (void)hipFuncSetAttribute((const void *)quantize_kernel<true>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
    hipLaunchKernelGGL(quantize_kernel<true>, dim3((unsigned)grid), dim3(kThreads),
                       (size_t)lds, stream, a);
  } else {
    const int64_t lds = quantize_act_lds(a.stage, a.rows_per_wg, K);
    if (lds > kMaxLds) return hipErrorInvalidValue;
    (void)hipFuncSetAttribute((const void *)quantize_kernel<false>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
    hipLaunchKernelGGL(quantize_kernel<false>, dim3((unsigned)grid), dim3(kThreads),
                       (size_t)lds, stream, a);
  }
  return hipGetLastError();
}

int64_t quantize_act_lds(int stage, int rows_per_wg, int64_t K) {
  const int64_t nb = K / kBlock;
  return (int64_t)rows_per_wg * ((stage ? 2 * K : 0) + K + 2 * nb);
}

int quantize_rows_per_wg(int64_t K) {
  const int64_t G = 4 * (K / kBlock);
  return G >= kThreads ? 1 : (int)(kThreads / G);
}

}  // namespace mxq
