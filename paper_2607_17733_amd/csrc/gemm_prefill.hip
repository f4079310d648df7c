// gemm_prefill.hip -- MXINT GEMM for prefill shapes on int8 matrix cores,
// with exponent-aligned block groups; also the exact per-block partial-sum
// kernel (same tiles and operands, every block its own group).
//
// Y[i][j] = sum_b P[i][j][b] * 2^(sa[i][b] + sw[j][b])   (MXSens, arXiv
// 2607.17733, Section 2: integer block products and power-of-two block
// scales; Section 6: mixed widths on an integer datapath).
//
// Each 32-wide block is one V_MFMA_I32_32X32X32_I8 per 32x32 output tile, so
// its int32 sum is exact.  Converting every block sum to fp32 and scaling it
// costs about four vector instructions per output, several times the
// matrix-core time of the block itself.  Consecutive blocks of one width (a
// "group") are therefore accumulated in one int32 sum after aligning their
// mantissas to a common exponent by exact shifts inside int8:
//   operand = q * 2^(8 - m - (ref - E)),  0 <= ref - E <= 8 - m,
// so that block b contributes exactly P' * 2^(ref_a + ref_w - 266) for its
// int8 operand product P'.  One fp32 rescale per group remains.
//
// Operands:
//   - A comes as the operand image written by the activation quantizer
//     (already unpacked and aligned per (row, chunk); its reference exponent
//     per block is in the exponent buffer).  Each wave loads its 64 rows
//     straight from global memory into matrix-core registers, three blocks
//     ahead; nothing of A goes through LDS.
//   - W is unpacked from the packed weight layout once per workgroup into LDS
//     (double-buffered, one unit of up to 4 blocks per step, raw loads two
//     units ahead), shifted to a per-(column, chunk) reference min E + 8 - m.
// A chunk (up to 16 blocks of one width) is one group when every row of the
// tile has a single reference over it and every column's exponent spread
// fits the headroom (prologue); otherwise each block is its own group.
//
// Tiling: 256x128 outputs per workgroup of four waves (one per SIMD), each
// wave 64 rows x 128 columns = 2x4 tiles of 32x32.  Workgroup ids are
// remapped so that each XCD works on a contiguous range of row tiles.
#include "mxq_device.h"
#include "mxq_internal.h"

namespace mxq {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 256, BN = 128, NT = 256;
constexpr int GC = 16;        // blocks per alignment chunk (a multiple of 4)
constexpr int MAXCH = 128;    // chunks tracked per tile; later ones are per-block

__device__ inline int headroom(int m) { return 8 - m; }

// Arithmetic right shift of every byte of v by s in [0, 4]; the low s bits
// of each byte are zero, so no bits cross between bytes.
__device__ inline uint32_t sar8(uint32_t v, uint32_t s) {
  const uint32_t S = v & 0x80808080u;
  return (v >> s) | ((S - (S >> s)) << 1);
}

struct Geo {
  int n4, n6, n8;
  int u4, u6, u8;             // units (4 blocks of one width) per segment
  int c4, c6, c8;             // chunks per segment
  __device__ Geo(int a, int b, int c)
      : n4(a), n6(b), n8(c), u4((a + 3) / 4), u6((b + 3) / 4), u8((c + 3) / 4),
        c4((a + GC - 1) / GC), c6((b + GC - 1) / GC), c8((c + GC - 1) / GC) {}
  __device__ int units() const { return u4 + u6 + u8; }
  __device__ int chunks() const { return c4 + c6 + c8; }
  // Unit u: width m, first block b0, rg blocks, its chunk and whether the
  // unit ends that chunk.  A unit is one quad of the packed weight layout.
  __device__ void unit(int u, int &m, int &b0, int &rg, int &ch, bool &chunk_end) const {
    int seg_b0, nseg, cbase, first;
    if (u < u4) { m = 4; seg_b0 = 0; nseg = n4; cbase = 0; first = 4 * u; }
    else if (u < u4 + u6) { m = 6; seg_b0 = n4; nseg = n6; cbase = c4; first = 4 * (u - u4); }
    else { m = 8; seg_b0 = n4 + n6; nseg = n8; cbase = c4 + c6; first = 4 * (u - u4 - u6); }
    b0 = seg_b0 + first;
    rg = min(4, nseg - first);
    ch = cbase + first / GC;
    chunk_end = ((first + 4) % GC == 0) || (first + 4 >= nseg);
  }
  __device__ void chunk_range(int c, int &b0, int &b1) const {
    if (c < c4) { b0 = c * GC; b1 = min(n4, b0 + GC); }
    else if (c < c4 + c6) { b0 = n4 + (c - c4) * GC; b1 = min(n4 + n6, b0 + GC); }
    else { b0 = n4 + n6 + (c - c4 - c6) * GC; b1 = min(n4 + n6 + n8, b0 + GC); }
  }
  __device__ int chunk_width(int c) const { return c < c4 ? 4 : (c < c4 + c6 ? 6 : 8); }
};

// Raw (still packed) weight data of one unit for this thread (its half of one
// W column: two lanes of the quad chunk, plus the 6-bit top-bit words), the
// column's exponents and the A row's reference (and, for partials, block)
// exponents.  Loaded with a fixed number of unconditional 16-byte loads, so
// the loads of different steps can be waited for individually.
struct Stage {
  uint4 w[5];
  uint32_t ew, ra, ea;
};

__device__ inline uint32_t byte_of(uint32_t v, int j) { return (v >> (8 * j)) & 255u; }
__device__ inline uint32_t dw(const uint4 &v, int k) {
  return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
}

template <bool PARTIALS>
__global__ __launch_bounds__(NT, 1) void gemm_prefill_kernel(GemmArgs g, int mtiles,
                                                             int ntiles) {
  __shared__ __attribute__((aligned(16))) uint4 Ws[2][4][2][BN];
  __shared__ __attribute__((aligned(16))) float Sa[2][4][BM];
  __shared__ __attribute__((aligned(16))) float Sw[2][4][BN];
  __shared__ uint32_t valid[MAXCH / 32];
  __shared__ uint8_t wbase[BN][MAXCH];        // per-(column, chunk) minimum exponent
  __shared__ uint8_t Sh[PARTIALS ? 2 : 1][4][BM];   // partials: int8-operand product shift

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int T = mtiles * ntiles;
  int tile = blockIdx.x;
  if ((T & 7) == 0) tile = (tile & 7) * (T >> 3) + (tile >> 3);
  const int mt = tile / ntiles, nt = tile - mt * ntiles;
  const int64_t row0 = (int64_t)mt * BM, col0 = (int64_t)nt * BN;
  const Segs s{g.n4, g.n6, g.n8};
  const int nb = g.n4 + g.n6 + g.n8;
  const Geo geo(g.n4, g.n6, g.n8);
  const int nunits = geo.units();
  const int nchb = min(geo.chunks(), MAXCH);
  const int64_t sbytes = slab_bytes(s);

  // Thread roles: A row t (reference exponents); W column t/2, element groups
  // 2*(t&1) and 2*(t&1)+1 (unpack).  Rows / columns past the end read a
  // valid row (results never stored; their scales are zero).
  const int64_t arow = row0 + t;
  const bool arow_ok = arow < g.M;
  const uint8_t *aref_p = g.a_exp + (arow_ok ? arow : g.M - 1) * g.a_erb + g.a_ref;
  const int wl = t >> 1, wkh = t & 1;
  const int64_t wcol = col0 + wl;
  const bool wcol_ok = wcol < g.npad;
  const int64_t wcol_c = wcol_ok ? wcol : g.npad - 1;
  const uint8_t *wslab = g.w_mant + (wcol_c >> 4) * sbytes;
  const uint8_t *wexp_p = g.w_exp + wcol_c * g.w_erb;
  const int wc = (int)(wcol_c & 15);

  // ---- prologue: which chunks form one group for the whole tile, and each
  // column's minimum exponent per chunk.
  if (t < MAXCH / 32) valid[t] = PARTIALS ? 0u : 0xFFFFFFFFu;
  __syncthreads();
  if (!PARTIALS && nchb > 0) {
    int c = 0, b0, b1;
    geo.chunk_range(0, b0, b1);
    int H = headroom(geo.chunk_width(0));
    int aref0 = -1, wmin = 255, wmax = 0;
    bool aok = true;
    uint4 ac = make_uint4(0, 0, 0, 0), wcache = make_uint4(0, 0, 0, 0);
    const bool wown = wcol_ok && wkh == 0;
    for (int b = 0; b < nb && c < nchb; ++b) {
      if ((b & 15) == 0) {
        if (arow_ok) ac = *(const uint4 *)(aref_p + b);
        if (wown) wcache = *(const uint4 *)(wexp_p + b);
      }
      const int sh = 8 * (b & 3), wi = (b >> 2) & 3;
      const int ra = (dw(ac, wi) >> sh) & 255, ew = (dw(wcache, wi) >> sh) & 255;
      if (aref0 < 0) aref0 = ra;
      aok = aok && (ra == aref0);
      wmin = min(wmin, ew);
      wmax = max(wmax, ew);
      if (b + 1 == b1) {
        if ((arow_ok && !aok) || (wown && wmax - wmin > H))
          atomicAnd(&valid[c >> 5], ~(1u << (c & 31)));
        if (wkh == 0) wbase[wl][c] = (uint8_t)(wcol_ok ? wmin : 0);
        ++c;
        if (c < nchb) {
          geo.chunk_range(c, b0, b1);
          H = headroom(geo.chunk_width(c));
        }
        aref0 = -1; aok = true; wmin = 255; wmax = 0;
      }
    }
  }
  __syncthreads();

  auto chunk_ok = [&](int c) -> bool {
    return c < nchb && ((valid[c >> 5] >> (c & 31)) & 1u);
  };

  // Raw W loads of unit u (clamped to the last unit): five 16-byte loads,
  // the lane data of element groups kg0 = 2*wkh and kg0+1 (up to 32 bytes
  // each) and the 6-bit top-bit words, each from an address clamped into
  // the slab; plus the exponent bytes.
  auto load_unit = [&](int uu, Stage &st) {
    const int u = min(uu, nunits - 1);
    int m, b0, rg, ch;
    bool ce;
    geo.unit(u, m, b0, rg, ch, ce);
    const BlockInfo bi = block_info(s, b0);
    const int gq = bi.idx >> 2;
    const int64_t chunk = seg_base(s, bi.seg) + 256LL * m * gq;
    const int l0 = 2 * wkh * 16 + wc, l1 = l0 + 16;
    const int lb = m == 6 ? 4 : m;             // nibble-plane bytes per block and lane
    const int64_t o0 = chunk + (int64_t)l0 * rg * lb, o1 = chunk + (int64_t)l1 * rg * lb;
    const int64_t ot = chunk + 256LL * rg + (int64_t)(wkh * 16 + wc) * rg * 4;
    // Reads may run up to 32 bytes past a lane's data (into the next lane,
    // chunk or slab, or the buffer's tail padding); those bytes are unused.
    st.w[0] = *(const uint4 *)(wslab + o0);
    st.w[1] = *(const uint4 *)(wslab + o0 + 16);
    st.w[2] = *(const uint4 *)(wslab + o1);
    st.w[3] = *(const uint4 *)(wslab + o1 + 16);
    st.w[4] = *(const uint4 *)(wslab + ot);
    st.ew = 0;
    st.ra = 0;
    st.ea = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int bj = min(b0 + j, nb - 1);
      st.ew |= (uint32_t)wexp_p[bj] << (8 * j);
      st.ra |= (uint32_t)aref_p[bj] << (8 * j);
      if (PARTIALS) st.ea |= (uint32_t)aref_p[bj - g.a_ref] << (8 * j);
    }
  };

  // Unpack the W data of unit u into LDS buffer u&1 and write the unit's
  // per-block group scales of this thread's A row and W column.
  auto prep = [&](int u, const Stage &st) {
    int m, b0, rg, ch;
    bool ce;
    geo.unit(u, m, b0, rg, ch, ce);
    const int buf = u & 1;
    const bool grouped = chunk_ok(ch);
    const int H = headroom(m);
    const int bw = grouped ? wbase[wl][ch] : 0;
    // lane data: 4-bit: dword j of w[0] (kg0) / w[2] (kg1); 8-bit: dwords
    // 2j, 2j+1 of w[0..1] / w[2..3]; 6-bit: nibble dword j of w[0] / w[2],
    // top word j of w[4].
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j >= rg) break;
      const int ra = (int)byte_of(st.ra, j);
      Sa[buf][j][t] = arow_ok ? (ra == 255 ? __builtin_nanf("") : ldexpf(1.0f, ra - 133)) : 0.f;
      if (PARTIALS)   // A operand carries 2^(H - (ref - E)), W operand 2^H
        Sh[buf][j][t] = (uint8_t)(2 * H - (ra - (int)byte_of(st.ea, j)));
      const int ew = (int)byte_of(st.ew, j);
      const int ref_w = grouped ? bw + H : ew;
      const uint32_t sw = (uint32_t)(ref_w - ew) & 7u;
      if (wkh == 0)
        Sw[buf][j][wl] = wcol_ok ? ((grouped ? bw : ew) == 255 ? __builtin_nanf("")
                                                               : ldexpf(1.0f, ref_w - 133))
                                 : 0.f;
      uint32_t wv[4];
      if (m == 4) {
        const uint32_t x0 = dw(st.w[0], j), x1 = dw(st.w[2], j);
        wv[0] = sar8((x0 << 4) & 0xF0F0F0F0u, sw);
        wv[1] = sar8(x0 & 0xF0F0F0F0u, sw);
        wv[2] = sar8((x1 << 4) & 0xF0F0F0F0u, sw);
        wv[3] = sar8(x1 & 0xF0F0F0F0u, sw);
      } else if (m == 6) {
        const uint32_t y = dw(st.w[4], j);
        const uint64_t v0 = unpack6(dw(st.w[0], j), y);
        const uint64_t v1 = unpack6(dw(st.w[2], j), y << 4);
        wv[0] = sar8((uint32_t)v0, sw);
        wv[1] = sar8((uint32_t)(v0 >> 32), sw);
        wv[2] = sar8((uint32_t)v1, sw);
        wv[3] = sar8((uint32_t)(v1 >> 32), sw);
      } else {
        const uint4 &p0 = st.w[j >> 1], &p1 = st.w[2 + (j >> 1)];
        wv[0] = dw(p0, 2 * (j & 1));
        wv[1] = dw(p0, 2 * (j & 1) + 1);
        wv[2] = dw(p1, 2 * (j & 1));
        wv[3] = dw(p1, 2 * (j & 1) + 1);
      }
      Ws[buf][j][wkh][wl] = make_uint4(wv[0], wv[1], wv[2], wv[3]);
    }
  };

  v16i acc_i[2][4];
  float acc_f[2][4][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int n = 0; n < 4; ++n) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        acc_i[a][n][r] = 0;
        acc_f[a][n][r] = 0.f;
      }
    }

  const int l32 = lane & 31, lh = lane >> 5;
  // This lane's A operand rows (two 32-row tiles of the wave's 64 rows).
  const int64_t r_a0 = row0 + wave * 64 + l32, r_a1 = r_a0 + 32;
  const uint8_t *aop0 = g.a_mant + min(r_a0, g.M - 1) * g.a_rb + g.a_op + 16 * lh;
  const uint8_t *aop1 = g.a_mant + min(r_a1, g.M - 1) * g.a_rb + g.a_op + 16 * lh;
  // A operands of unit u (clamped to valid blocks): 4 blocks x 2 row tiles.
  auto load_a = [&](int uu, v4i (&x)[4][2]) {
    const int u = min(uu, nunits - 1);
    int m, b0, rg, ch;
    bool ce;
    geo.unit(u, m, b0, rg, ch, ce);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t off = (int64_t)min(b0 + j, nb - 1) * kBlock;
      x[j][0] = *(const v4i *)(aop0 + off);
      x[j][1] = *(const v4i *)(aop1 + off);
    }
  };

  // Fold the int32 group sums into fp32 (or store them as exact block sums)
  // with the scales of block j of the unit in buffer buf.
  auto flush = [&](int buf, int j, int b) {
#pragma unroll
    for (int tm = 0; tm < 2; ++tm) {
#pragma unroll
      for (int tn = 0; tn < 4; ++tn) {
        const int cl = tn * 32 + l32;
        const float swv = Sw[buf][j][cl];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int rl = wave * 64 + tm * 32 + 8 * q + 4 * lh;
          const float4 sav = *(const float4 *)&Sa[buf][j][rl];
          const float sa4[4] = {sav.x, sav.y, sav.z, sav.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int r = 4 * q + u;
            if (PARTIALS) {
              const int64_t i = row0 + rl + u, jj = col0 + cl;
              if (i < g.M && jj < g.N)
                g.p[(i * g.N + jj) * nb + b] = acc_i[tm][tn][r] >> Sh[buf][j][rl + u];
            } else {
              acc_f[tm][tn][r] += (float)acc_i[tm][tn][r] * (sa4[u] * swv);
            }
          }
        }
      }
    }
  };

  // One K step: multiply unit u (A operands in x, W operands in LDS), then
  // refill x with unit u+2.
  bool fresh = true;          // the int32 accumulators hold no group yet
  auto step = [&](int u, v4i (&x)[4][2], Stage &st_use) {
    int m, b0, rg, ch;
    bool ce;
    geo.unit(u, m, b0, rg, ch, ce);
    const bool grouped = chunk_ok(ch);
    const int buf = u & 1;
    __syncthreads();
    if (u + 1 < nunits) {
      prep(u + 1, st_use);
      load_unit(u + 3, st_use);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j >= rg) break;
      v4i w4[4];
#pragma unroll
      for (int tn = 0; tn < 4; ++tn)
        w4[tn] = *(const v4i *)&Ws[buf][j][lh][tn * 32 + l32];
      if (fresh) {
        const v4i zero = {0, 0, 0, 0};
        const v16i z16 = {};
        (void)zero;
#pragma unroll
        for (int tn = 0; tn < 4; ++tn) {
          acc_i[0][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(x[j][0], w4[tn], z16, 0, 0, 0);
          acc_i[1][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(x[j][1], w4[tn], z16, 0, 0, 0);
        }
      } else {
#pragma unroll
        for (int tn = 0; tn < 4; ++tn) {
          acc_i[0][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(x[j][0], w4[tn], acc_i[0][tn], 0, 0, 0);
          acc_i[1][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(x[j][1], w4[tn], acc_i[1][tn], 0, 0, 0);
        }
      }
      fresh = false;
      if (!grouped || (ce && j == rg - 1)) {
        flush(buf, j, b0 + j);
        fresh = true;
      }
    }
    load_a(u + 2, x);
  };

  Stage st0, st1;
  v4i xa[4][2], xb[4][2];
  load_unit(0, st0);
  load_a(0, xa);
  load_a(1, xb);
  load_unit(1, st1);
  prep(0, st0);
  load_unit(2, st0);

  for (int u = 0; u < nunits; u += 2) {
    step(u, xa, st1);                          // prep(u+1) uses the stage of u+1
    if (u + 1 < nunits) step(u + 1, xb, st0);
  }
  if (PARTIALS) return;
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int tn = 0; tn < 4; ++tn) {
      const int64_t j = col0 + tn * 32 + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t i = row0 + wave * 64 + tm * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (i < g.M && j < g.N) g.y[i * g.ldy + j] = acc_f[tm][tn][r];
      }
    }
}

template <bool PARTIALS>
hipError_t launch(const GemmArgs &a, hipStream_t stream) {
  const int mtiles = (int)((a.M + BM - 1) / BM), ntiles = (int)((a.N + BN - 1) / BN);
  hipLaunchKernelGGL(gemm_prefill_kernel<PARTIALS>, dim3((unsigned)(mtiles * ntiles)),
                     dim3(NT), 0, stream, a, mtiles, ntiles);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_prefill(const GemmArgs &a, hipStream_t stream) {
  return launch<false>(a, stream);
}

hipError_t launch_gemm_partials(const GemmArgs &a, hipStream_t stream) {
  return launch<true>(a, stream);
}

}  // namespace mxq
