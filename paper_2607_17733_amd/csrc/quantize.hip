// quantize.hip -- offline MXINT quantize + pack of bf16 weight rows.
//
// MXSens (arXiv 2607.17733) Section 2 and Section 4.1: every 32-element
// block of the permuted weight row (one output column) gets one shared
// exponent and one mantissa width, the same quantizer as the activations.
//
// Work decomposition: a thread owns 8 consecutive elements of a block (a
// "group"), so the 4 threads of a block are adjacent lanes; the block
// maximum is a 2-step xor-shuffle reduction of integer |bf16| bit patterns.
// A workgroup owns one row (K >= 2048) or several whole rows (short K, e.g.
// the 128-wide KV-cache rows).  With a column permutation the workgroup first
// stages its source rows in LDS with 16-byte coalesced loads and gathers from
// LDS, so the permutation never turns into scattered global loads.
//
// Every column is written twice: into the 16-column slabs of the stream
// layout (packed mantissas in the decode GEMM's lane order, see DGeo), and
// into the 128-column tiles of the matrix-core operand image (FP6/FP8
// digits of each mantissa, the layout described with OpGeo) with their E8M0
// scale bytes, which the prefill GEMM reads.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void quantize_kernel(QuantArgs q) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int t = threadIdx.x;
  const int64_t K = q.K;
  const int nb = (int)(K / kBlock);
  const int G = 4 * nb;                      // groups per row
  const int R = q.rows_per_wg;
  const int64_t row0 = (int64_t)blockIdx.x * R;
  const Segs s{q.n4, q.n6, q.n8};
  // LDS: [R][K] staged bf16 source rows (permuted path only).
  uint16_t *srow = (uint16_t *)smem;
  const OpGeo og(q.n4, q.n6, q.n8);

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
      qv[u] = b < q.n3 ? 2 * quant_elem(bits[u], E, 3, q.ties_away, q.full_clamp)
                       : quant_elem(bits[u], E, bi.m, q.ties_away, q.full_clamp);

    // stream-layout nibble codes, and (6-bit) the 2-bit codes of the half's
    // 16 elements: element 8d+k of the half at bits 8(k%4) + 4d + 2(k/4)
    const bool sm = !q.full_clamp;
    const uint32_t nib = stream_nibbles(qv, bi.m, sm);
    uint32_t top = 0;
    if (bi.m == 6) {
      const int dd = kg & 1;
#pragma unroll
      for (int k = 0; k < 8; ++k)
        top |= stream_top2(qv[k], sm) << (8 * (k & 3) + 4 * dd + 2 * (k >> 2));
      top |= __shfl_xor(top, 1);             // merge the lane pair's word
    }
    if (!live) continue;

    uint32_t lo8 = 0, hi8 = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      lo8 |= ((uint32_t)qv[u] & 255u) << (8 * u);
      hi8 |= ((uint32_t)qv[4 + u] & 255u) << (8 * u);
    }
    // digit codes of the 8 mantissas (MXINT -> FP6 / FP8 elements)
    uint32_t d0[8], d1[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) mxint_digits(qv[u], bi.m, d0[u], d1[u]);
    // step, lane half and (4-bit) pair of this block
    int st, h, j = 0;
    if (bi.m == 4) { st = bi.idx >> 2; h = bi.idx & 1; j = (bi.idx >> 1) & 1; }
    else if (bi.m == 6) { st = og.s4 + (bi.idx >> 1); h = bi.idx & 1; }
    else { st = og.s4 + og.s6 + bi.idx; h = kg >> 1; }

    {
      const int c = (int)(row % kOpCols);
      uint8_t *tile = q.mant + q.w_op + (row / kOpCols) * q.w_tile;
      if (row < q.slab_rows) {
        // stream layout of the 16-column slab (decode GEMM)
        const DGeo dg(q.n4, q.n6, q.n8);
        const int c16 = (int)(row & 15);
        uint8_t *slab = q.mant + (row >> 4) * wd_slab_bytes(dg);
        const DLoc L = d_loc(bi.seg, bi.idx);
        const int sd = wd_step_data(bi.seg);
        uint8_t *segp = slab + wd_seg_off(dg, bi.seg);
        uint8_t *chunk = segp + step_data_off(L.st, sd);
        const int dd = kg & 1;
        const int ln = 16 * (L.g0 + (kg >> 1)) + c16;
        if (bi.m == 4) {
          *(uint32_t *)(chunk + 16 * ln + L.region + 4 * dd) = nib;
        } else if (bi.m == 6) {
          *(uint32_t *)(chunk + 8 * ln + 4 * dd) = nib;
          if (dd == 0) *(uint32_t *)(chunk + 512 + 4 * ln) = top;
        } else {
          *(uint32_t *)(chunk + 16 * ln + 8 * dd) = lo8;
          *(uint32_t *)(chunk + 16 * ln + 8 * dd + 4) = hi8;
        }
        if (kg == 0) {
          segp[step_scale_off(L.st, sd, 16 * L.sg0 + c16)] = (uint8_t)E;
          if (bi.seg) segp[step_scale_off(L.st, sd, 16 * L.sg1 + c16)] = (uint8_t)E;
          q.exp[row * q.out_erb + b] = (uint8_t)E;
        }
        if (g == 0) {
          for (int64_t z = nb; z < q.out_erb; ++z) q.exp[row * q.out_erb + z] = 0;
          // zero the stream padding blocks of this column
          const int nseg[3] = {dg.n4, dg.n6, dg.n8};
          const int npad[3] = {4 * dg.S[0], 2 * dg.S[1], 2 * dg.S[2]};
          for (int sg = 0; sg < 3; ++sg) {
            const int psd = wd_step_data(sg);
            uint8_t *pseg = slab + wd_seg_off(dg, sg);
            for (int idx = nseg[sg]; idx < npad[sg]; ++idx) {
              const DLoc P = d_loc(sg, idx);
              uint8_t *pc = pseg + step_data_off(P.st, psd);
              for (int hh = 0; hh < 2; ++hh) {
                const int pl = 16 * (P.g0 + hh) + c16;
                if (sg == 0) {
                  *(uint2 *)(pc + 16 * pl + P.region) = make_uint2(0, 0);
                } else if (sg == 1) {
                  *(uint2 *)(pc + 8 * pl) = make_uint2(0, 0);
                  *(uint32_t *)(pc + 512 + 4 * pl) = 0;
                } else {
                  *(uint4 *)(pc + 16 * pl) = make_uint4(0, 0, 0, 0);
                }
              }
              pseg[step_scale_off(P.st, psd, 16 * P.sg0 + c16)] = 0;
              if (sg) pseg[step_scale_off(P.st, psd, 16 * P.sg1 + c16)] = 0;
            }
            // the unused scale bytes of a short last group
            const int S = dg.S[sg];
            for (int st = S; st < (S + kStreamGroup - 1) / kStreamGroup * kStreamGroup; ++st)
              for (int gg = 0; gg < 4; ++gg) pseg[step_scale_off(st, psd, 16 * gg + c16)] = 0;
          }
        }
      }
      if (row == 0 && g == 0)                // the packed section's tail padding
        for (int z = 0; z < q.tail_pad; ++z)
          q.mant[q.slab_rows / 16 * wd_slab_bytes(DGeo(q.n4, q.n6, q.n8)) + z] = 0;
      // operand image (128-column tiles of per-step chunks)
      if (bi.m == 8) {
        uint32_t h0 = 0, h1 = 0, l0 = 0, l1 = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          h0 |= d0[u] << (8 * u); h1 |= d0[4 + u] << (8 * u);
          l0 |= d1[u] << (8 * u); l1 |= d1[4 + u] << (8 * u);
        }
        const int o = 8 * (kg & 1);
        *(uint2 *)(tile + w_op_loc(st, h, c, o)) = make_uint2(h0, h1);
        *(uint2 *)(tile + w_op_loc(st, h, c, 16 + o)) = make_uint2(l0, l1);
        *(uint2 *)(tile + w_op_loc(st, h, c, 32 + o)) = make_uint2(h0, h1);
      } else {
        uint64_t v0 = 0, v1 = 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          v0 |= (uint64_t)d0[u] << (6 * u);
          v1 |= (uint64_t)d1[u] << (6 * u);
        }
        const int o = (bi.m == 4 ? 24 * j : 0) + 6 * kg;
#pragma unroll
        for (int k = 0; k < 3; ++k)
          *(uint16_t *)(tile + w_op_loc(st, h, c, o + 2 * k)) = (uint16_t)(v0 >> (16 * k));
        if (bi.m == 6)
#pragma unroll
          for (int k = 0; k < 3; ++k)
            *(uint16_t *)(tile + w_op_loc(st, h, c, 24 + o + 2 * k)) = (uint16_t)(v1 >> (16 * k));
      }
      if (kg == 0) {                         // scale dword of the lane: bytes su0, su1, 0, 0
        if (bi.m == 4) {
          uint8_t *sp = tile + w_op_scale(st, h, c);
          sp[j] = (uint8_t)E;
          if (j == 0) *(uint16_t *)(sp + 2) = 0;
        } else if (bi.m == 6) {
          *(uint32_t *)(tile + w_op_scale(st, h, c)) = (uint32_t)E;
        } else {
          *(uint32_t *)(tile + w_op_scale(st, 0, c)) = (uint32_t)E;
          *(uint32_t *)(tile + w_op_scale(st, 1, c)) = (uint32_t)E;
        }
      }
      if (g == 0) {                          // zero the pad blocks of the column
        for (int i = og.n4; i < og.n4p; ++i) {
          const int pst = i >> 2, ph = i & 1, pj = (i >> 1) & 1;
          for (int z = 0; z < 24; z += 2)
            *(uint16_t *)(tile + w_op_loc(pst, ph, c, 24 * pj + z)) = 0;
          uint8_t *sp = tile + w_op_scale(pst, ph, c);
          sp[pj] = 0;
          if (pj == 0) *(uint16_t *)(sp + 2) = 0;
        }
        if (og.n6p > og.n6) {
          const int pst = og.s4 + (og.n6 >> 1);
          for (int z = 0; z < 48; z += 2)
            *(uint16_t *)(tile + w_op_loc(pst, 1, c, z)) = 0;
          *(uint32_t *)(tile + w_op_scale(pst, 1, c)) = 0;
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_quantize(const QuantArgs &args, bool weights,
                           hipStream_t stream) {
  if (!weights) return hipErrorInvalidValue;     // activations: launch_quantize_act
  const int64_t K = args.K;
  const int nb = (int)(K / kBlock);
  const int G = 4 * nb;
  QuantArgs a = args;
  a.rows_per_wg = G >= kThreads ? 1 : kThreads / G;
  const int64_t grid = (a.out_rows + a.rows_per_wg - 1) / a.rows_per_wg;
  if (grid <= 0) return hipSuccess;
  const int64_t lds = a.stage ? (int64_t)a.rows_per_wg * K * 2 : 0;
  if (lds > kMaxLds) return hipErrorInvalidValue;
  (void)hipFuncSetAttribute((const void *)quantize_kernel,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  hipLaunchKernelGGL(quantize_kernel, dim3((unsigned)grid), dim3(kThreads),
                     (size_t)lds, stream, a);
  return hipGetLastError();
}

int quantize_rows_per_wg(int64_t K) {
  const int64_t G = 4 * (K / kBlock);
  return G >= kThreads ? 1 : (int)(kThreads / G);
}

}  // namespace mxq
