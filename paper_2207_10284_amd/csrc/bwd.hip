// Gradients of the MRA-2 output with the selection held fixed (Sec. 4.2 eq.
// actual_approx_mat_form, Sec. 4.3 Alg. 2; R = {b, 1}, b = 32).
//
// Query i of block-row x takes a softmax over the fine logits P_ij = c Q_i.K_j
// of the columns j of its refined blocks T_x and, with the low-resolution
// term, over the coarse logits S~[x,y] + ln b of the other blocks y, applied
// to the rows V_j and V~_y. With L_i its log normaliser (saved by the
// forward), G = dZ and delta_i = G_i . Z_i, each logit's gradient is its
// probability times (G_i . value - delta_i):
//   fine:   dP_ij = e^{P_ij - L_i} (G_i . V_j - delta_i)
//           dQ_i += c sum_j dP_ij K_j,   dK_j += c sum_i dP_ij Q_i,
//           dV_j += sum_i e^{P_ij - L_i} G_i
//   coarse: the 32 queries of block-row x share S~[x,y]. For a reference m_x,
//           W[x,y] = b e^{S~[x,y] - m_x} (0 for y in T_x),
//           G^_x = sum_{i in x} e^{m_x - L_i} G_i,  d^_x = sum e^{m_x - L_i} delta_i:
//           dS~[x,y] = W[x,y] (V~_y . G^_x - d^_x),   dV~_y = sum_x W[x,y] G^_x,
//           dQ~_x = c sum_y dS~[x,y] K~_y,           dK~_y = c sum_x dS~[x,y] Q~_x.
//           A pooled row is a block mean, so its gradient reaches each of the
//           block's 32 rows divided by 32.
// m_x = min_{i in x} L_i keeps both exponentials at most 1: every L_i is at
// least each coarse logit S~[x,y] + ln b of its own row.
//
// Kernels, in launch order (after the packing pass of pool.hip):
//  * bwd_rows_kernel: per block-row (a wave; 16 per workgroup): a 256-byte
//    record of the 32 log normalisers (log2 units) and the 32 deltas, the
//    selection as a bitmap; with the coarse
//    term also G^, d^ and the row's W, dS~ and dQ~ (K~ and V~ staged through
//    LDS 64 blocks at a time).
//  * bwd_cols_kernel: per column block (a wave; 16 per workgroup): dK~, dV~.
//  * bwd_dq_(stream_)kernel: per block-row (a wave), over its refined tiles: the
//    products K_y Q_x^T and V_y G_x^T on the matrix cores, then
//    dQ^T += K_y^T dP^T.
//  * bwd_dkdv_(stream_)kernel: per column block (a wave), over the block-rows that
//    refined it (ascending): dV^T += G_x^T A, dK^T += c Q_x^T dP. For raw
//    tiles the row pass also writes, per query, the bfloat16 triples of
//    -L_i/c and -delta_i, which enter the products as one more contraction
//    step, so a lane holding 16 queries needs no per-query registers.
// Tile operands: for bfloat16 raw 32-row tiles of the inputs (copied into LDS
// under a swizzle that serves row and transposed reads); for float32 packed
// copies in the layouts of tile_ops.h.
#include "common.h"
#include "kernels.h"
#include "tile_ops.h"

namespace mra {

constexpr int kBwdRows = 16;              // waves (block-rows) per workgroup of the row pass
constexpr int kBwdTileWaves = 4;          // waves per workgroup of the tile passes
constexpr int kBwdCols = 16;              // column blocks per workgroup of the column pass
// Raw-tile slots per wave of the bfloat16 gradient passes: one (the next tile
// is copied once the current one is in registers) measured faster than two.
constexpr int kDqSlots = 1;
constexpr int kDkdvSlots = 1;

template <int DT>
__device__ __forceinline__ float elem_lo(uint32_t w) {
  return DT == BF16 ? bf16_to_f32(w & 0xFFFFu) : __uint_as_float(w);
}

__device__ __forceinline__ f32x4 mfma16x4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// x as hi + mid + lo, each rounded to bfloat16 in turn (the two differences
// are exact in float32, so the sum is x to about 2^-24 |x|).
__device__ __forceinline__ uint32_t split3_bf16(float x, uint32_t& mid_lo) {
  const __bf16 hi = (__bf16)x;
  const float r1 = x - (float)hi;
  const __bf16 mid = (__bf16)r1;
  const __bf16 lo = (__bf16)(r1 - (float)mid);
  mid_lo = (uint32_t)__builtin_bit_cast(uint16_t, mid) | ((uint32_t)__builtin_bit_cast(uint16_t, lo) << 16);
  return __builtin_bit_cast(uint16_t, hi);
}

// One query's bias operand for the column pass: the bfloat16 elements
// [hi(x), mid(x), lo(x), hi(y), mid(y), lo(y), 0, 0].
__device__ __forceinline__ u32x4 bias_operand(float x, float y) {
  uint32_t xm, ym;
  const uint32_t xh = split3_bf16(x, xm), yh = split3_bf16(y, ym);
  return u32x4{xh | (xm << 16), (xm >> 16) | (yh << 16), ym, 0u};
}

// ---------------------------------------------------------------------------
// Row pass: one wave per block-row x for the per-row terms (the record, the
// bitmap, G^_x, d^_x), then with the coarse term the 16 rows of the
// workgroup together, 128 column blocks per step, on the float32 matrix cores
// (v_mfma_f32_16x16x4_f32; A: 16 rows x 4, B: 4 x 16 columns, lane l holds
// A[l%16][l/16] and B[l/16][l%16], and D[4(l/16)+r][l%16] in register r):
//  1. S~ = Q~_x K~_y^T and G^_x V~_y^T: one 16 x 16 tile per wave, the
//     contraction over dims taken four at a time from 16-byte loads;
//  2. W and dS~ for the 16 x 128 entries (two per thread), written out;
//  3. dQ~_x += dS~ K~_y: wave (dim tile, part of the step's columns), the
//     partial sums added in part order at the end.
template <int DT, int D, bool COARSE>
__global__ __launch_bounds__(kBwdRows * kWave) __attribute__((amdgpu_waves_per_eu(8, 8))) void bwd_rows_kernel(
    const void* __restrict__ gin, const void* __restrict__ zin, const float* __restrict__ lse,
    const int32_t* __restrict__ idx, const float* __restrict__ qp, const float* __restrict__ kp,
    const float* __restrict__ vp, float* __restrict__ ld, uint32_t* __restrict__ bias,
    uint32_t* __restrict__ bits, float* __restrict__ gh, float* __restrict__ Wout,
    float* __restrict__ dSout, float* __restrict__ dqp, int nb, int m, float scale) {
  using Cfg = TileCfg<DT, D>;
  using elem = typename Cfg::elem;
  constexpr int KC = Cfg::kKChunks;                        // 16-byte chunks per half row
  constexpr int PQ = D + 4;                                 // LDS pitch of the Q~, G^ rows
  constexpr int YC = 128;                                   // column blocks per step
  constexpr int PP = YC + 1, PD = YC + 4;
  constexpr int NTD = D / 16, KQ = kBwdRows / NTD, YK = YC / KQ;
  static_assert(KQ * kBwdRows * D <= 2 * kBwdRows * PP, "dQ~ partials fit the step buffer");
  __shared__ __attribute__((aligned(16))) float Qx[COARSE ? kBwdRows * PQ : 1];
  __shared__ __attribute__((aligned(16))) float Gx[COARSE ? kBwdRows * PQ : 1];
  __shared__ float Pst[COARSE ? 2 * kBwdRows * PP : 1];    // a step's S~, G^V~^T; then dQ~ partials
  __shared__ float Ds[COARSE ? kBwdRows * PD : 1];
  __shared__ float wq[kBwdRows][32];
  __shared__ float rowm[kBwdRows], rowd[kBwdRows];
  __shared__ uint32_t bm_all[kBwdRows][64];                 // nb <= 2048 bits

  const int tid = threadIdx.x;
  const int w = wave_uniform(tid / kWave);
  const int lane = lane_id(), j = lane & 31, h = lane >> 5;
  const int groups = (nb + kBwdRows - 1) / kBwdRows;
  const long long lwg = xcd_remap(blockIdx.x, gridDim.x);
  const long long bh = lwg / groups;
  const int x0 = (int)(lwg - bh * groups) * kBwdRows;
  const bool active = x0 + w < nb;                          // wave-uniform
  const long long g = bh * nb + x0 + w;                     // this wave's block-row
  const int nbw = (nb + 31) / 32;
  uint32_t* bm = bm_all[w];

  if (active) {
    // the first 64 selection entries and the log normaliser are requested
    // first, so their latency overlaps the delta's loads
    const int ysel0 = lane < m ? idx[g * m + lane] : -1;
    const float L = lse[g * 32 + j];
    // delta_i = G_i . Z_i: lane (h, j) takes half h of row j
    const long long roff = (g * 32 + j) * D + (D / 2) * h;
    const u32x4* gp = reinterpret_cast<const u32x4*>(reinterpret_cast<const elem*>(gin) + roff);
    const u32x4* zp = reinterpret_cast<const u32x4*>(reinterpret_cast<const elem*>(zin) + roff);
    float part = 0.0f;
#pragma unroll 4
    for (int s = 0; s < KC; ++s) {
      const u32x4 gw = gp[s], zw = zp[s];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        part = fmaf(elem_lo<DT>(gw[e]), elem_lo<DT>(zw[e]), part);
        if constexpr (DT == BF16) part = fmaf(bf16_to_f32(gw[e] >> 16), bf16_to_f32(zw[e] >> 16), part);
      }
    }
    const float dl = halves_sum(part);
    if (h == 0) {                                           // the block-row's record
      ld[g * 64 + j] = L * kLog2e;
      ld[g * 64 + 32 + j] = dl;
      if (bias != nullptr)
        *reinterpret_cast<u32x4*>(bias + (g * 32 + j) * 4) = bias_operand(-L / scale, -dl);
    }
    // the selection as a bitmap (entries outside [0, nb) ignored)
    for (int i = lane; i < nbw; i += kWave) bm[i] = 0u;
    wave_lds_sync();
    if (ysel0 >= 0 && ysel0 < nb) atomicOr(&bm[ysel0 >> 5], 1u << (ysel0 & 31));
    for (int i0 = kWave; i0 < m; i0 += kWave) {
      const int y = i0 + lane < m ? idx[g * m + i0 + lane] : -1;
      if (y >= 0 && y < nb) atomicOr(&bm[y >> 5], 1u << (y & 31));
    }
    wave_lds_sync();
    for (int i = lane; i < nbw; i += kWave) bits[g * nbw + i] = bm[i];
    if constexpr (COARSE) {
      const float mref = -wave_max(-L);                     // min over the 32 queries
      const float wi = exp2f((mref - L) * kLog2e);
      const float dhat = wave_sum(h == 0 ? wi * dl : 0.0f);
      if (h == 0) wq[w][j] = wi;
      if (lane == 0) {
        rowm[w] = mref;
        rowd[w] = dhat;
      }
      wave_lds_sync();
      // G^_x: lanes over the dims, rows in order
      const elem* G = reinterpret_cast<const elem*>(gin) + g * 32 * D;
      for (int dd = lane; dd < D; dd += kWave) {
        float acc = 0.0f;
        for (int i = 0; i < 32; ++i) {
          float gv;
          if constexpr (DT == BF16) gv = bf16_to_f32(G[i * D + dd]);
          else gv = G[i * D + dd];
          acc = fmaf(wq[w][i], gv, acc);
        }
        Gx[w * PQ + dd] = acc;
        gh[g * D + dd] = acc;
        Qx[w * PQ + dd] = qp[g * D + dd];
      }
    }
  } else if constexpr (COARSE) {
    for (int dd = lane; dd < D; dd += kWave) Gx[w * PQ + dd] = Qx[w * PQ + dd] = 0.0f;
  }
  if constexpr (!COARSE) return;
  __syncthreads();                                          // Q~, G^, rowm, rowd, bitmaps

  // K~, V~ of the head as buffers: loads past row nb read as zero
  const unsigned hbytes = (unsigned)nb * D * (unsigned)sizeof(float);
  const i32x4 krs = buffer_rsrc(kp + bh * (long long)nb * D, hbytes);
  const i32x4 vrs = buffer_rsrc(vp + bh * (long long)nb * D, hbytes);
  const int lr = lane & 15, lg = lane >> 4;
  const int kind = w >> 3, t = w & 7;                       // step 1: S~ (0) or G^V~^T (1), columns 16t..
  const float* arow = (kind ? Gx : Qx) + lr * PQ + 4 * lg;
  const i32x4 brs = kind ? vrs : krs;
  const int nt = w % NTD, kq = w / NTD;                     // step 3: dims 16nt.., columns kq*YK..
  const int b1lane = ((16 * t + lr) * D + 4 * lg) * (int)sizeof(float);
  const int b3lane = ((kq * YK + lg) * D + 16 * nt + lr) * (int)sizeof(float);
  f32x4 accq = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int y0 = 0; y0 < nb; y0 += YC) {
    const int ystep = y0 * D * (int)sizeof(float);
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    constexpr int UG = D / 16 < 4 ? D / 16 : 4;             // 16-byte loads in flight per group
#pragma unroll
    for (int u0 = 0; u0 < D / 16; u0 += UG) {
      f32x4 bq[UG];
#pragma unroll
      for (int u = 0; u < UG; ++u)
        bq[u] = mra_raw_buffer_load_f32x4(brs, b1lane + ystep + 16 * (u0 + u) * (int)sizeof(float), 0, 0);
#pragma unroll
      for (int u = 0; u < UG; ++u) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(arow + 16 * (u0 + u));
#pragma unroll
        for (int e = 0; e < 4; ++e) acc = mfma16x4(a[e], bq[u][e], acc);   // dims 16(u0+u) + 4(l/16) + e
      }
    }
    __syncthreads();                                        // the previous step's Pst, Ds consumed
#pragma unroll
    for (int r = 0; r < 4; ++r) Pst[(kind * kBwdRows + 4 * lg + r) * PP + 16 * t + lr] = acc[r];
    __syncthreads();
    for (int e = tid; e < kBwdRows * YC; e += kBwdRows * kWave) {
      const int i = e / YC, yl = e % YC, y = y0 + yl;
      float dsv = 0.0f;
      if (x0 + i < nb && y < nb) {
        float wv = 0.0f;
        if (!((bm_all[i][y >> 5] >> (y & 31)) & 1u)) {
          wv = (float)kBlock * exp2f(fmaf(Pst[i * PP + yl], scale, -rowm[i]) * kLog2e);
          dsv = wv * (Pst[(kBwdRows + i) * PP + yl] - rowd[i]);
        }
        const long long gi = bh * nb + x0 + i;
        Wout[gi * nb + y] = wv;
        dSout[gi * nb + y] = dsv;
      }
      Ds[i * PD + yl] = dsv;
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < YK / 4; ++s) {
      const int yl = kq * YK + 4 * s + lg;
      const float b = mra_raw_buffer_load_f32(krs, b3lane + ystep + 4 * s * D * (int)sizeof(float), 0, 0);
      accq = mfma16x4(Ds[lr * PD + yl], b, accq);
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 4; ++r) Pst[(kq * kBwdRows + 4 * lg + r) * D + 16 * nt + lr] = accq[r];
  __syncthreads();
  if (active) {
    for (int dd = lane; dd < D; dd += kWave) {
      float sum = Pst[w * D + dd];
#pragma unroll
      for (int q = 1; q < KQ; ++q) sum += Pst[(q * kBwdRows + w) * D + dd];
      dqp[g * D + dd] = sum * scale;
    }
  }
}

// The block-rows x whose selection holds column block y (bit y of row x's
// bitmap), ascending, into list (LDS); returns their count (wave-uniform).
// The bitmap words of kColBatch groups of 64 rows are all requested before
// the first is used (rows past nb read row nb - 1's word and are dropped).
constexpr int kColBatch = 8;
__device__ __forceinline__ int column_list(const uint32_t* __restrict__ bits, long long hb, int nbw, int y,
                                           int nb, int32_t* list) {
  const int lane = lane_id();
  int cnt = 0;
  for (int x0 = 0; x0 < nb; x0 += kColBatch * kWave) {
    uint32_t wv[kColBatch];
#pragma unroll
    for (int u = 0; u < kColBatch; ++u) {
      const int x = min(x0 + kWave * u + lane, nb - 1);
      wv[u] = bits[(hb + x) * nbw + (y >> 5)];
    }
#pragma unroll
    for (int u = 0; u < kColBatch; ++u) {
      const int x = x0 + kWave * u + lane;
      const bool ok = x < nb && ((wv[u] >> (y & 31)) & 1u);
      const uint64_t mk = __ballot(ok);
      if (ok) list[cnt + bits_below(mk)] = x;
      cnt += __popcll(mk);
    }
  }
  wave_lds_sync();
  return wave_uniform(cnt);
}

// ---------------------------------------------------------------------------
// Column pass: dK~_y = c sum_x dS~[x,y] Q~_x and dV~_y = sum_x W[x,y] G^_x for
// 16 column blocks per workgroup on the float32 matrix cores, the contraction
// over the block-rows x in ascending order, four per matrix-core step. A wave
// takes one quantity and TW = min(4, D/16) dim tiles at once, with the dims
// permuted inside its group of 16 TW: tile t, column n is dim 16 TW g +
// TW n + t, so each lane reads its TW consecutive dims of a row of Q~ or G^
// with one load (and stores its TW dims of an output row with one store),
// and the column of W or dS serves all TW products.
constexpr int kColsBatch = 8;                             // matrix-core steps per batch of loads

template <int D>
struct ColsCfg {
  static constexpr int kTW = D / 16 < 4 ? D / 16 : 4;      // dim tiles per wave
  static constexpr int kGroups = D / (16 * kTW);            // dim groups
  static constexpr int kWaves = 2 * kGroups;                // (quantity, group) per wave
};

template <int TW>
__device__ __forceinline__ void load_tw(i32x4 rs, int off, float (&b)[TW]) {
  if constexpr (TW == 4) {
    const f32x4 v = mra_raw_buffer_load_f32x4(rs, off, 0, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) b[t] = v[t];
  } else if constexpr (TW == 2) {
    const f32x2 v = mra_raw_buffer_load_f32x2(rs, off, 0, 0);
    b[0] = v[0];
    b[1] = v[1];
  } else {
    b[0] = mra_raw_buffer_load_f32(rs, off, 0, 0);
  }
}

template <int D>
__global__ __launch_bounds__(ColsCfg<D>::kWaves * kWave) void bwd_cols_kernel(
    const float* __restrict__ qp, const float* __restrict__ gh, const float* __restrict__ W,
    const float* __restrict__ dS, float* __restrict__ dkp, float* __restrict__ dvp, int nb,
    float scale) {
  constexpr int TW = ColsCfg<D>::kTW;
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id(), lr = lane & 15, lg = lane >> 4;
  const int groups = (nb + kBwdCols - 1) / kBwdCols;
  const long long lwg = xcd_remap(blockIdx.x, gridDim.x);
  const long long bh = lwg / groups;
  const int y0 = (int)(lwg - bh * groups) * kBwdCols;
  const long long hb = bh * nb;                             // first block of the head
  const int y = y0 + lr;
  const int kind = w / ColsCfg<D>::kGroups, dg = w % ColsCfg<D>::kGroups;
  const int d0 = 16 * TW * dg + TW * lr;                    // this lane's first dim
  // A[y][x] = A[x * nb + y] (column y) and B[x][d0 ..] of the head as
  // buffers: reads past the head's last row or column come back as zero
  // (those columns' outputs are not stored)
  const i32x4 ars = buffer_rsrc((kind ? W : dS) + hb * nb, (unsigned)nb * nb * (unsigned)sizeof(float));
  const i32x4 brs = buffer_rsrc((kind ? gh : qp) + hb * D, (unsigned)nb * D * (unsigned)sizeof(float));
  int ao = (lg * nb + y) * (int)sizeof(float), bo = (lg * D + d0) * (int)sizeof(float);
  f32x4 acc[TW];
#pragma unroll
  for (int t = 0; t < TW; ++t) acc[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  // kColsBatch steps of four block-rows per batch, every load of a batch in
  // flight before its products (rows past nb read as zero)
  for (int xs = 0; xs < nb; xs += 4 * kColsBatch) {
    float a[kColsBatch], b[kColsBatch][TW];
#pragma unroll
    for (int u = 0; u < kColsBatch; ++u) {
      a[u] = mra_raw_buffer_load_f32(ars, ao + u * 4 * nb * (int)sizeof(float), 0, 0);
      load_tw<TW>(brs, bo + u * 4 * D * (int)sizeof(float), b[u]);
    }
#pragma unroll
    for (int u = 0; u < kColsBatch; ++u)
#pragma unroll
      for (int t = 0; t < TW; ++t) acc[t] = mfma16x4(a[u], b[u][t], acc[t]);
    ao += 4 * kColsBatch * nb * (int)sizeof(float);
    bo += 4 * kColsBatch * D * (int)sizeof(float);
  }
  // lane: rows y0 + 4 lg + r, dims d0 + t
  float* out = kind ? dvp : dkp;
  const float f = kind ? 1.0f : scale;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int yy = y0 + 4 * lg + r;
    if (yy >= nb) continue;
    float* o = out + (hb + yy) * D + d0;
    if constexpr (TW == 4) {
      *reinterpret_cast<f32x4*>(o) = f32x4{acc[0][r] * f, acc[1][r] * f, acc[2][r] * f, acc[3][r] * f};
    } else {
#pragma unroll
      for (int t = 0; t < TW; ++t) o[t] = acc[t][r] * f;
    }
  }
}

// Stores a 32 x D block from d-major tiles acc (lane: row j; register r of
// tile t: dim 32t + 8(r/4) + 4h + r%4) as acc * a + (add ? add[dim] / 32 : 0).
// The add terms are loaded first, all at once. bfloat16: lanes l and l^32
// hold dims 4h..4h+3 of the groups rg (even, odd); they exchange one group so
// that each stores 8 contiguous dims (16 bytes).
template <int DT, int D>
__device__ __forceinline__ void store_block(typename TileCfg<DT, D>::elem* dst,
                                            const f32x16 (&acc)[D / 32], float a,
                                            const float* add) {
  constexpr int NT = D / 32;
  const int lane = lane_id(), j = lane & 31, h = lane >> 5;
  auto* row = dst + (long long)j * D;
  constexpr float inv = 1.0f / kBlock;
  f32x4 c4[NT][4];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg)
      c4[t][rg] = add != nullptr ? *reinterpret_cast<const f32x4*>(add + 32 * t + 8 * rg + 4 * h)
                                 : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    u32x2 pend = {0u, 0u};
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int d0 = 32 * t + 8 * rg + 4 * h;
      float z[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) z[e] = fmaf(acc[t][4 * rg + e], a, c4[t][rg][e] * inv);
      if constexpr (DT == BF16) {
        const u32x2 pr = {pack_bf16x2(z[0], z[1]), pack_bf16x2(z[2], z[3])};
        if ((rg & 1) == 0) {
          pend = pr;
        } else {
          const u32x2 send = h ? pend : pr;                 // h = 0 sends its odd group, h = 1 its even one
          u32x2 recv;
          recv[0] = (uint32_t)__shfl_xor((int)send[0], 32);
          recv[1] = (uint32_t)__shfl_xor((int)send[1], 32);
          const u32x4 st = h ? u32x4{recv[0], recv[1], pr[0], pr[1]} : u32x4{pend[0], pend[1], recv[0], recv[1]};
          *reinterpret_cast<u32x4*>(row + 32 * t + 8 * (rg - 1) + 8 * h) = st;
        }
      } else {
        const f32x4 st = {z[0], z[1], z[2], z[3]};
        *reinterpret_cast<f32x4*>(row + d0) = st;
      }
    }
  }
}

// bfloat16 pairs of 16 float32 values in register order (the B operand of
// mfma_acc_bf16).
__device__ __forceinline__ void pack16(const float (&v)[16], uint32_t (&pk)[8]) {
#pragma unroll
  for (int rr = 0; rr < 8; ++rr) {
    bf16x2 pb;
    pb[0] = (__bf16)v[2 * rr];
    pb[1] = (__bf16)v[2 * rr + 1];
    pk[rr] = __builtin_bit_cast(uint32_t, pb);
  }
}

// C = X0 Y0^T + A B^T (bfloat16, row layout): the product of one more
// contraction step x0, y0 (16 elements of each row) followed by the KC chunks
// of a and b.
template <int KC>
__device__ __forceinline__ f32x16 mfma_abt_from(const u32x4 (&a)[KC], const u32x4 (&b)[KC], u32x4 x0, u32x4 y0) {
  f32x16 c;
#pragma unroll
  for (int r = 0; r < 16; ++r) c[r] = 0.0f;
  c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, x0), __builtin_bit_cast(bf16x8, y0), c, 0, 0, 0);
#pragma unroll
  for (int k = 0; k < KC; ++k)
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[k]), __builtin_bit_cast(bf16x8, b[k]), c, 0, 0, 0);
  return c;
}

// ---------------------------------------------------------------------------
// dQ: one wave per block-row x. For each refined block y (ascending):
// S^T = K_y Q_x^T and (V_y G_x^T) on the matrix cores (lane: query, 16 keys),
// dP^T = e^{S^T c - L} o (V G^T - delta), dQ^T += K_y^T dP^T. The epilogue
// scales by c and adds dQ~_x / 32. Operand loads for the next tile are issued
// before the current tile is computed (past the last one they re-read it).
template <int DT, int D, bool COARSE>
__global__ __launch_bounds__(kBwdTileWaves * kWave) void bwd_dq_kernel(
    const void* __restrict__ qin, const void* __restrict__ gin, const void* __restrict__ krow,
    const void* __restrict__ vrow, const void* __restrict__ kt, const int32_t* __restrict__ idx,
    const float* __restrict__ ld, const float* __restrict__ dqp, void* __restrict__ dq, int nb,
    int m, long long rows, float scale, float scale_log2) {
  using Cfg = TileCfg<DT, D>;
  using elem = typename Cfg::elem;
  constexpr int KC = Cfg::kKChunks, VC = Cfg::kVChunks, NT = Cfg::kNT;
  extern __shared__ int32_t sidx_all[];
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id(), jq = lane & 31;
  const long long g = xcd_remap(blockIdx.x, gridDim.x) * (long long)kBwdTileWaves + w;
  if (g >= rows) return;                                    // no workgroup barriers below
  const long long bh = g / nb;
  int32_t* myidx = sidx_all + w * m;
  const int cnt = stage_selection(idx + g * m, m, nb, myidx);

  u32x4 qf[KC], gf[KC];
  load_rows<DT, D>(reinterpret_cast<const elem*>(qin) + g * 32 * D, qf);
  load_rows<DT, D>(reinterpret_cast<const elem*>(gin) + g * 32 * D, gf);
  const float lq = ld[g * 64 + jq], dl = ld[g * 64 + 32 + jq];
  f32x16 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.0f;

  const u32x4* kr = reinterpret_cast<const u32x4*>(krow) + bh * nb * KC * 64 + lane;
  const u32x4* vr = reinterpret_cast<const u32x4*>(vrow) + bh * nb * KC * 64 + lane;
  const u32x4* ktp = reinterpret_cast<const u32x4*>(kt) + bh * nb * VC * 64 + lane;
  struct Ops {
    u32x4 k[KC], v[KC], t[VC];
  };
  auto load = [&](int y, Ops& o) {
#pragma unroll
    for (int c = 0; c < KC; ++c) o.k[c] = kr[((long long)y * KC + c) * 64];
#pragma unroll
    for (int c = 0; c < KC; ++c) o.v[c] = vr[((long long)y * KC + c) * 64];
#pragma unroll
    for (int c = 0; c < VC; ++c) o.t[c] = ktp[((long long)y * VC + c) * 64];
  };
  Ops cur, nxt;
  if (cnt > 0) load(wave_uniform(myidx[0]), cur);
  for (int i = 0; i < cnt; ++i) {
    load(wave_uniform(myidx[min(i + 1, cnt - 1)]), nxt);
    const f32x16 s = mfma_abt<DT, KC>(cur.k, qf);
    const f32x16 pv = mfma_abt<DT, KC>(cur.v, gf);
    float ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
      ds[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -lq)) * (pv[r] - dl);
    if constexpr (DT == BF16) {
      uint32_t pk[8];
      pack16(ds, pk);
      mfma_acc_bf16<NT>(acc, pk, [&](int c) { return cur.t[c]; });
    } else {
      mfma_acc_f32<NT>(acc, ds, [&](int c) { return cur.t[c]; });
    }
    cur = nxt;
  }
  store_block<DT, D>(reinterpret_cast<elem*>(dq) + g * 32 * D, acc, scale,
                     COARSE ? dqp + g * D : nullptr);
}

// ---------------------------------------------------------------------------
// dK, dV: one wave per column block y. For each block-row x whose selection
// holds y (ascending): S = Q_x K_y^T and G_x V_y^T (lane: key, 16 queries),
// A = e^{S c - L}, dP = A o (G V^T - delta), dV^T += G_x^T A,
// dK^T += Q_x^T dP. The epilogue scales dK by c and adds dK~_y / 32 and
// dV~_y / 32.
template <int DT, int D, bool COARSE, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void bwd_dkdv_kernel(
    const void* __restrict__ kin, const void* __restrict__ vin, const void* __restrict__ qrow,
    const void* __restrict__ grow, const void* __restrict__ qt, const void* __restrict__ gt,
    const uint32_t* __restrict__ bits, const float* __restrict__ ld,
    const float* __restrict__ dkp, const float* __restrict__ dvp, void* __restrict__ dk,
    void* __restrict__ dv, int nb, long long rows, float scale, float scale_log2) {
  using Cfg = TileCfg<DT, D>;
  using elem = typename Cfg::elem;
  constexpr int KC = Cfg::kKChunks, VC = Cfg::kVChunks, NT = Cfg::kNT;
  extern __shared__ int32_t sidx_all[];
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id(), h = lane >> 5;
  const long long gy = xcd_remap(blockIdx.x, gridDim.x) * (long long)WAVES + w;
  if (gy >= rows) return;                                   // no workgroup barriers below
  const long long bh = gy / nb;
  const int y = (int)(gy - bh * nb);
  const long long hb = bh * nb;
  const int nbw = (nb + 31) / 32;

  // block-rows whose selection holds y, ascending
  int32_t* myx = sidx_all + w * nb;
  const int cnt = column_list(bits, hb, nbw, y, nb, myx);

  u32x4 kf[KC], vf[KC];
  load_rows<DT, D>(reinterpret_cast<const elem*>(kin) + gy * 32 * D, kf);
  load_rows<DT, D>(reinterpret_cast<const elem*>(vin) + gy * 32 * D, vf);
  f32x16 ak[NT], av[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) ak[t][r] = av[t][r] = 0.0f;

  const u32x4* qr = reinterpret_cast<const u32x4*>(qrow) + hb * KC * 64 + lane;
  const u32x4* gr = reinterpret_cast<const u32x4*>(grow) + hb * KC * 64 + lane;
  const u32x4* qtp = reinterpret_cast<const u32x4*>(qt) + hb * VC * 64 + lane;
  const u32x4* gtp = reinterpret_cast<const u32x4*>(gt) + hb * VC * 64 + lane;
  struct Ops {
    u32x4 q[KC], g[KC], qt[VC], gt[VC];
    f32x4 l[4], d[4];
  };
  auto load = [&](int x, Ops& o) {
#pragma unroll
    for (int c = 0; c < KC; ++c) o.q[c] = qr[((long long)x * KC + c) * 64];
#pragma unroll
    for (int c = 0; c < KC; ++c) o.g[c] = gr[((long long)x * KC + c) * 64];
#pragma unroll
    for (int c = 0; c < VC; ++c) o.qt[c] = qtp[((long long)x * VC + c) * 64];
#pragma unroll
    for (int c = 0; c < VC; ++c) o.gt[c] = gtp[((long long)x * VC + c) * 64];
    // queries 8rg + 4h + e of block-row x (the rows of this lane's registers)
    const float* lx = ld + (hb + x) * 64 + 4 * h;
    const float* dx = lx + 32;
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      o.l[rg] = *reinterpret_cast<const f32x4*>(lx + 8 * rg);
      o.d[rg] = *reinterpret_cast<const f32x4*>(dx + 8 * rg);
    }
  };
  Ops cur, nxt;
  if (cnt > 0) load(wave_uniform(myx[0]), cur);
  for (int i = 0; i < cnt; ++i) {
    load(wave_uniform(myx[min(i + 1, cnt - 1)]), nxt);
    const f32x16 s = mfma_abt<DT, KC>(cur.q, kf);
    const f32x16 pv = mfma_abt<DT, KC>(cur.g, vf);
    float a[16], ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      a[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -cur.l[r / 4][r % 4]));
      ds[r] = a[r] * (pv[r] - cur.d[r / 4][r % 4]);
    }
    if constexpr (DT == BF16) {
      uint32_t pa[8], pd[8];
      pack16(a, pa);
      pack16(ds, pd);
      mfma_acc_bf16<NT>(av, pa, [&](int c) { return cur.gt[c]; });
      mfma_acc_bf16<NT>(ak, pd, [&](int c) { return cur.qt[c]; });
    } else {
      mfma_acc_f32<NT>(av, a, [&](int c) { return cur.gt[c]; });
      mfma_acc_f32<NT>(ak, ds, [&](int c) { return cur.qt[c]; });
    }
    cur = nxt;
  }
  store_block<DT, D>(reinterpret_cast<elem*>(dk) + gy * 32 * D, ak, scale,
                     COARSE ? dkp + gy * D : nullptr);
  store_block<DT, D>(reinterpret_cast<elem*>(dv) + gy * 32 * D, av, 1.0f,
                     COARSE ? dvp + gy * D : nullptr);
}

// ---------------------------------------------------------------------------
// Streaming forms of the two tile passes (tiles whose chunks fit the load's
// immediate offset: bf16 d <= 64, f32 d = 32). A wave's next tile is copied
// HBM/L2 -> LDS with direct-to-LDS loads while the current one is computed.
// Each wave owns a slot split into parts that are consumed at different
// times (separate LDS objects, so reading one part does not wait for loads in
// flight into another); a part is refilled with the next tile's operands as
// soon as it has been read into registers. Loads complete in issue order, so
// "part P of tile i has landed" is a wait until at most the number of loads
// issued after it are outstanding.
template <int N>
__device__ __forceinline__ void wait_loads() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// dQ, one wave per block-row. Part A: K_y and V_y in the row layout (the
// products with Q_x and G_x); part B: K_y in the transposed layout.
template <int DT, int D, bool COARSE, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void bwd_dq_stream_kernel(
    const void* __restrict__ qin, const void* __restrict__ gin, const void* __restrict__ krow,
    const void* __restrict__ vrow, const void* __restrict__ kt, const int32_t* __restrict__ idx,
    const float* __restrict__ ld, const float* __restrict__ dqp, void* __restrict__ dq, int nb,
    int m, long long rows, float scale, float scale_log2) {
  using Cfg = TileCfg<DT, D>;
  using elem = typename Cfg::elem;
  constexpr int KC = Cfg::kKChunks, VC = Cfg::kVChunks, NT = Cfg::kNT;
  constexpr int NA = 2 * KC, NB = VC;                      // loads per part
  static_assert(KC <= 4 && VC <= 4, "chunk offsets fit the immediate field");
  __shared__ __attribute__((aligned(16))) u32x4 partA[WAVES][NA * 64];
  __shared__ __attribute__((aligned(16))) u32x4 partB[WAVES][NB * 64];
  extern __shared__ int32_t sidx_all[];
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id(), jq = lane & 31;
  const long long g = xcd_remap(blockIdx.x, gridDim.x) * (long long)WAVES + w;
  if (g >= rows) return;                                    // no workgroup barriers below
  const long long bh = g / nb;
  int32_t* myidx = sidx_all + w * m;
  const int cnt = stage_selection(idx + g * m, m, nb, myidx);

  u32x4 qf[KC], gf[KC];
  load_rows<DT, D>(reinterpret_cast<const elem*>(qin) + g * 32 * D, qf);
  load_rows<DT, D>(reinterpret_cast<const elem*>(gin) + g * 32 * D, gf);
  const float lq = ld[g * 64 + jq], dl = ld[g * 64 + 32 + jq];
  f32x16 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.0f;

  const unsigned loff = lane * 16u;
  const char* ks = static_cast<const char*>(krow) + (size_t)bh * nb * KC * 1024 + loff;
  const char* vs = static_cast<const char*>(vrow) + (size_t)bh * nb * KC * 1024 + loff;
  const char* ts = static_cast<const char*>(kt) + (size_t)bh * nb * VC * 1024 + loff;
  const lptr_t la = (lptr_t)partA[w];
  const lptr_t lb = (lptr_t)partB[w];
  const uint32_t aA = lds_addr(partA[w]) + loff, aB = lds_addr(partB[w]) + loff;
  auto issueA = [&](int y) {
    load_chunks_lds<KC>((gptr_t)(ks + (size_t)y * KC * 1024), la);
    load_chunks_lds<KC>((gptr_t)(vs + (size_t)y * KC * 1024), la + KC * 1024);
  };
  auto issueB = [&](int y) { load_chunks_lds<VC>((gptr_t)(ts + (size_t)y * VC * 1024), lb); };
  if (cnt > 0) {
    const int y0 = wave_uniform(myidx[0]);
    issueA(y0);
    issueB(y0);
  }
  for (int i = 0; i < cnt; ++i) {
    const bool more = i + 1 < cnt;                          // wave-uniform
    const int yn = more ? wave_uniform(myidx[i + 1]) : 0;
    wait_loads<NB>();                                       // A(i) landed; B(i) may not have
    u32x4 kf[KC], vf[KC];
    lds_read_chunks<KC>(aA, kf);
    lds_read_chunks<KC, KC>(aA, vf);
    lds_done(kf);
    lds_done(vf);
    if (more) issueA(yn);
    const f32x16 s = mfma_abt<DT, KC>(kf, qf);
    const f32x16 pv = mfma_abt<DT, KC>(vf, gf);
    float ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
      ds[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -lq)) * (pv[r] - dl);
    if (more) wait_loads<NA>();                             // B(i) landed; A(i+1) may not have
    else wait_loads<0>();
    u32x4 tf[VC];
    lds_read_chunks<VC>(aB, tf);
    lds_done(tf);
    if (more) issueB(yn);
    if constexpr (DT == BF16) {
      uint32_t pk[8];
      pack16(ds, pk);
      mfma_acc_bf16<NT>(acc, pk, [&](int c) { return tf[c]; });
    } else {
      mfma_acc_f32<NT>(acc, ds, [&](int c) { return tf[c]; });
    }
  }
  store_block<DT, D>(reinterpret_cast<elem*>(dq) + g * 32 * D, acc, scale,
                     COARSE ? dqp + g * D : nullptr);
}

// dK, dV, one wave per column block. Part A: Q_x and G_x in the row layout;
// part X: block-row x's record (log normalisers and deltas, 256 bytes, one
// dword per lane); part B: Q_x and G_x in the transposed layout.
template <int DT, int D, bool COARSE, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void bwd_dkdv_stream_kernel(
    const void* __restrict__ kin, const void* __restrict__ vin, const void* __restrict__ qrow,
    const void* __restrict__ grow, const void* __restrict__ qt, const void* __restrict__ gt,
    const uint32_t* __restrict__ bits, const float* __restrict__ ld,
    const float* __restrict__ dkp, const float* __restrict__ dvp, void* __restrict__ dk,
    void* __restrict__ dv, int nb, long long rows, float scale, float scale_log2) {
  using Cfg = TileCfg<DT, D>;
  using elem = typename Cfg::elem;
  constexpr int KC = Cfg::kKChunks, VC = Cfg::kVChunks, NT = Cfg::kNT;
  constexpr int NA = 2 * KC, NX = 1, NB = 2 * VC;          // loads per part
  static_assert(KC <= 4 && VC <= 4, "chunk offsets fit the immediate field");
  __shared__ __attribute__((aligned(16))) u32x4 partA[WAVES][NA * 64];
  __shared__ __attribute__((aligned(16))) u32x4 partB[WAVES][NB * 64];
  __shared__ __attribute__((aligned(16))) float partX[WAVES][64];
  extern __shared__ int32_t sidx_all[];
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id(), h = lane >> 5;
  const long long gy = xcd_remap(blockIdx.x, gridDim.x) * (long long)WAVES + w;
  if (gy >= rows) return;                                   // no workgroup barriers below
  const long long bh = gy / nb;
  const int y = (int)(gy - bh * nb);
  const long long hb = bh * nb;
  const int nbw = (nb + 31) / 32;

  // block-rows whose selection holds y, ascending
  int32_t* myx = sidx_all + w * nb;
  const int cnt = column_list(bits, hb, nbw, y, nb, myx);

  u32x4 kf[KC], vf[KC];
  load_rows<DT, D>(reinterpret_cast<const elem*>(kin) + gy * 32 * D, kf);
  load_rows<DT, D>(reinterpret_cast<const elem*>(vin) + gy * 32 * D, vf);
  f32x16 ak[NT], av[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) ak[t][r] = av[t][r] = 0.0f;

  const unsigned loff = lane * 16u;
  const char* qs = static_cast<const char*>(qrow) + (size_t)hb * KC * 1024 + loff;
  const char* gs = static_cast<const char*>(grow) + (size_t)hb * KC * 1024 + loff;
  const char* qts = static_cast<const char*>(qt) + (size_t)hb * VC * 1024 + loff;
  const char* gts = static_cast<const char*>(gt) + (size_t)hb * VC * 1024 + loff;
  const char* xs = reinterpret_cast<const char*>(ld + hb * 64) + lane * 4u;
  const lptr_t la = (lptr_t)partA[w];
  const lptr_t lb = (lptr_t)partB[w];
  const lptr_t lx = (lptr_t)partX[w];
  const uint32_t aA = lds_addr(partA[w]) + loff, aB = lds_addr(partB[w]) + loff;
  const uint32_t aX = lds_addr(partX[w]) + 16u * h;          // this half's queries
  auto issueA = [&](int x) {
    load_chunks_lds<KC>((gptr_t)(qs + (size_t)x * KC * 1024), la);
    load_chunks_lds<KC>((gptr_t)(gs + (size_t)x * KC * 1024), la + KC * 1024);
  };
  auto issueX = [&](int x) { __builtin_amdgcn_global_load_lds((gptr_t)(xs + (size_t)x * 256), lx, 4, 0, 0); };
  auto issueB = [&](int x) {
    load_chunks_lds<VC>((gptr_t)(qts + (size_t)x * VC * 1024), lb);
    load_chunks_lds<VC>((gptr_t)(gts + (size_t)x * VC * 1024), lb + VC * 1024);
  };
  if (cnt > 0) {
    const int x0 = wave_uniform(myx[0]);
    issueA(x0);
    issueX(x0);
    issueB(x0);
  }
  for (int i = 0; i < cnt; ++i) {
    const bool more = i + 1 < cnt;                          // wave-uniform
    const int xn = more ? wave_uniform(myx[i + 1]) : 0;
    wait_loads<NX + NB>();                                  // A(i) landed
    u32x4 qa[KC], ga[KC];
    lds_read_chunks<KC>(aA, qa);
    lds_read_chunks<KC, KC>(aA, ga);
    lds_done(qa);
    lds_done(ga);
    if (more) issueA(xn);
    const f32x16 s = mfma_abt<DT, KC>(qa, kf);             // lane: key, 16 queries
    const f32x16 pv = mfma_abt<DT, KC>(ga, vf);
    if (more) wait_loads<NB + NA>();                        // X(i) landed
    else wait_loads<NB>();
    u32x4 xr[8];                                            // queries 8rg + 4h + e
    xr[0] = lds_read16<0>(aX);
    xr[1] = lds_read16<32>(aX);
    xr[2] = lds_read16<64>(aX);
    xr[3] = lds_read16<96>(aX);
    xr[4] = lds_read16<128>(aX);
    xr[5] = lds_read16<160>(aX);
    xr[6] = lds_read16<192>(aX);
    xr[7] = lds_read16<224>(aX);
    lds_done(xr);
    if (more) issueX(xn);
    f32x4 lq[4], dl[4];
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      lq[rg] = __builtin_bit_cast(f32x4, xr[rg]);
      dl[rg] = __builtin_bit_cast(f32x4, xr[4 + rg]);
    }
    float a[16], ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      a[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -lq[r / 4][r % 4]));
      ds[r] = a[r] * (pv[r] - dl[r / 4][r % 4]);
    }
    if (more) wait_loads<NA + NX>();                        // B(i) landed
    else wait_loads<0>();
    u32x4 qb[VC], gb[VC];
    lds_read_chunks<VC>(aB, qb);
    lds_read_chunks<VC, VC>(aB, gb);
    lds_done(qb);
    lds_done(gb);
    if (more) issueB(xn);
    if constexpr (DT == BF16) {
      uint32_t pa8[8], pd8[8];
      pack16(a, pa8);
      pack16(ds, pd8);
      mfma_acc_bf16<NT>(av, pa8, [&](int c) { return gb[c]; });
      mfma_acc_bf16<NT>(ak, pd8, [&](int c) { return qb[c]; });
    } else {
      mfma_acc_f32<NT>(av, a, [&](int c) { return gb[c]; });
      mfma_acc_f32<NT>(ak, ds, [&](int c) { return qb[c]; });
    }
  }
  store_block<DT, D>(reinterpret_cast<elem*>(dk) + gy * 32 * D, ak, scale,
                     COARSE ? dkp + gy * D : nullptr);
  store_block<DT, D>(reinterpret_cast<elem*>(dv) + gy * 32 * D, av, 1.0f,
                     COARSE ? dvp + gy * D : nullptr);
}

// ---------------------------------------------------------------------------
// bfloat16 forms that read the transposed operands straight from the
// row-layout copy in LDS with gfx950's transposing read ds_read_b64_tr_b16:
// within each group of 16 lanes, lane i receives as value k (k = 0..3) the
// 16-bit element i%4 of the 8 bytes at the address that lane 4k + i/4 of the
// group supplies (lane layout checked on the device). Chunk (u, t) of the
// transposed operand X^T for lane l = 32h + j holds X[16u + 8(s/4) + 4h + s%4]
// [32t + j], s = 0..7; so each lane supplies, for each half e = 0, 1, the
// address of X[16u + 8e + 4(l/32) + (l%16)/4][32t + 16((l/16)&1) + 4(l&3)]
// (four consecutive columns of one row, 8 bytes) and two reads fill a chunk.
// Only the row-layout copies are then loaded per tile (dQ: K_y, V_y, 8 KB;
// dK/dV: Q_x, G_x and the record, 8.25 KB), and each wave keeps two whole
// tiles in flight in two LDS slots while it computes a third from registers.

// In LDS each 1 KB chunk of a row-layout block is followed by 64 bytes of
// padding, so the four chunks a transposing read touches start 16 banks apart:
// its 32 lanes per pass then hit 64 distinct banks (without the padding, lanes
// whose addresses differ by whole chunks share banks).
constexpr int kChunkPad = 64;
constexpr int kChunkStride = 1024 + kChunkPad;

// Byte offset of X[r][c] in a padded row-layout block (bf16, D columns) in LDS.
template <int D>
__host__ __device__ constexpr int row_layout_offset(int r, int c) {
  return ((c % (D / 2)) / 8) * kChunkStride + (32 * (c / (D / 2)) + r) * 16 + (c % 8) * 2;
}

// C consecutive 1 KB chunks HBM/L2 -> LDS at kChunkStride apart: the load's
// immediate offset steps both addresses by 1 KB, the LDS base adds the pad.
template <int C>
__device__ __forceinline__ void load_chunks_lds_padded(gptr_t src, lptr_t dst) {
  if constexpr (C > 0) {
    load_chunks_lds_padded<C - 1>(src, dst);
    __builtin_amdgcn_global_load_lds(src, dst + (C - 1) * kChunkPad, 16, (C - 1) * 1024, 0);
  }
}

// v[i] = padded chunk C0 + i for this lane, i < C
template <int I, int C, int C0>
struct LdsChunksPadded {
  static __device__ __forceinline__ void run(uint32_t addr, u32x4* v) {
    v[I] = lds_read16<(C0 + I) * kChunkStride>(addr);
    LdsChunksPadded<I + 1, C, C0>::run(addr, v);
  }
};
template <int C, int C0>
struct LdsChunksPadded<C, C, C0> {
  static __device__ __forceinline__ void run(uint32_t, u32x4*) {}
};

// this lane's address term for the transposed reads of a row-layout block
template <int D>
__device__ __forceinline__ uint32_t tr_lane_offset() {
  const int l = lane_id();
  return (uint32_t)row_layout_offset<D>(4 * (l >> 5) + ((l & 15) >> 2), 16 * ((l >> 4) & 1) + 4 * (l & 3));
}

// Transposed chunks c = u*NT + t (c < VC) of the row-layout block at `base`
// (+ this lane's tr_lane_offset); the caller completes them with lds_done().
template <int D, int C, int VC>
struct TrChunks {
  static constexpr int NT = D / 32;
  static __device__ __forceinline__ void run(uint32_t addr, u32x4* v) {
    if constexpr (C < VC) {
      constexpr int u = C / NT, t = C % NT;
      constexpr int o0 = row_layout_offset<D>(16 * u, 32 * t) - row_layout_offset<D>(0, 0);
      constexpr int o1 = row_layout_offset<D>(16 * u + 8, 32 * t) - row_layout_offset<D>(0, 0);
      const u32x2 a = lds_read_tr16<o0>(addr);
      const u32x2 b = lds_read_tr16<o1>(addr);
      v[C] = u32x4{a[0], a[1], b[0], b[1]};
      TrChunks<D, C + 1, VC>::run(addr, v);
    }
  }
};

// bfloat16: the passes read raw 32-row tiles of the inputs themselves, no
// packed copies. A tile (32 consecutive rows, 2d bytes each) is
// copied with direct-to-LDS loads of whole rows, every lane fetching the
// 16-byte block that belongs at its LDS position under an XOR swizzle of the
// blocks within a row (raw_offset / raw_copy_offset), and read both in the row
// layout (ds_read_b128: 16 lanes = 16 rows per pass) and transposed
// (ds_read_b64_tr_b16: 32 lanes = 4 rows x 64 bytes per pass). One swizzle
// serves both: for d = 64 the even rows of 16 consecutive rows take 8
// different block positions, and so do the odd ones (row reads), and rows r
// and r + 2 of a group of four take positions in opposite halves of the row
// (transposed reads); for d = 32 rows r, r + 4, r + 8, r + 12 take 4
// different positions; for d = 128 see the d = 128 kernels below. The
// swizzle has period 16 in the row, so the transposed reads 16 rows further
// use the same lane address plus an immediate offset; reads 8 rows further
// need a second address. The copy offsets repeat with period 4 (d = 128),
// 2 (d = 64) or 1 (d = 32) in the copy index.
template <int D>
__host__ __device__ constexpr int raw_swz_b(int r) {
  return D == 128 ? 4 * (r & 3) + ((r >> 2) & 3) : (D == 64 ? 4 * ((r >> 1) & 1) + ((r >> 2) & 3) : (r >> 2) & 3);
}

// This lane's offsets for the raw tiles of the gradient passes.
template <int D>
struct RawB {
  static constexpr int KC = D / 16, NT = D / 32;
  static constexpr int TB = 64 * D;                           // bytes of a 32-row tile
  static constexpr int KP = D == 128 ? 4 : (D == 64 ? 2 : 1); // period of the copy offsets
  unsigned cp[KP];                                            // copy sources of copies i mod KP (less their KB)
  uint32_t rr[KC];                                            // row-layout chunk c
  uint32_t tr[NT][2];                                         // transposed column tile t, half e
  __device__ __forceinline__ void init() {
    const int lane = lane_id(), h = lane >> 5, j = lane & 31, i16 = lane & 15;
#pragma unroll
    for (int q = 0; q < KP; ++q) cp[q] = (unsigned)(raw_copy_offset<D, raw_swz_b<D>>(q, lane) - q * 1024);
#pragma unroll
    for (int c = 0; c < KC; ++c) rr[c] = (uint32_t)raw_offset<D, raw_swz_b<D>>(j, (D / 2) * h + 8 * c);
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int e = 0; e < 2; ++e)
        tr[t][e] = (uint32_t)raw_offset<D, raw_swz_b<D>>(4 * h + i16 / 4 + 8 * e,
                                                         32 * t + 16 * ((lane >> 4) & 1) + 4 * (i16 & 3));
  }
};

// Two raw tiles, C 1 KB copies each, as buffer loads to LDS: the heads' rows
// are the resources ra and rb, the tiles' byte offsets ta and tb go in the
// scalar offset (outside the hardware range check: callers copy validated
// blocks only), this lane's swizzled source offset of copy i (cp[i mod KP],
// the offsets repeat with period KP) in the vector offset.
template <int C, int KP>
__device__ __forceinline__ void copy_raw_pair_buf(i32x4 ra, i32x4 rb, unsigned ta, unsigned tb,
                                                  const unsigned (&cp)[KP], lptr_t as, lptr_t bs) {
  if constexpr (C > 0) {
    copy_raw_pair_buf<C - 1, KP>(ra, rb, ta, tb, cp, as, bs);
    constexpr int i = C - 1;
    buffer_load_lds16(ra, as + i * 1024, cp[i % KP], ta + i * 1024);
    buffer_load_lds16(rb, bs + i * 1024, cp[i % KP], tb + i * 1024);
  }
}

// One raw tile, C 1 KB copies, as buffer loads to LDS (as copy_raw_pair_buf).
template <int C, int KP>
__device__ __forceinline__ void copy_raw_buf(i32x4 rs, unsigned t, const unsigned (&cp)[KP], lptr_t dst) {
#pragma unroll
  for (int i = 0; i < C; ++i) buffer_load_lds16(rs, dst + i * 1024, cp[i % KP], t + i * 1024);
}

// Row-layout chunks of the raw tile at base + OFF.
template <int OFF, int KC>
__device__ __forceinline__ void raw_rows(uint32_t base, const uint32_t (&rr)[KC], u32x4 (&v)[KC]) {
#pragma unroll
  for (int c = 0; c < KC; ++c) v[c] = lds_read16<OFF>(base + rr[c]);
}

// Transposed chunks c = u*NT + t (c < VC) of the raw tile at base + OFF: two
// transposing reads each, the halves 8 rows apart, 16 u rows further on.
template <int D, int OFF, int C, int VC>
struct RawTrB {
  static constexpr int NT = D / 32;
  static __device__ __forceinline__ void run(uint32_t base, const uint32_t (&tr)[NT][2], u32x4* v) {
    if constexpr (C < VC) {
      constexpr int u = C / NT, t = C % NT, o = OFF + 16 * u * 2 * D;
      const u32x2 a = lds_read_tr16<o>(base + tr[t][0]);
      const u32x2 b = lds_read_tr16<o>(base + tr[t][1]);
      v[C] = u32x4{a[0], a[1], b[0], b[1]};
      RawTrB<D, OFF, C + 1, VC>::run(base, tr, v);
    }
  }
};

// dQ (bf16, d <= 64): one wave per block-row; a slot holds the raw tiles K_y
// and V_y (K^T is read transposed from the K tile). SLOTS tiles in flight per
// wave: with one slot the next tile is copied once the current one is in
// registers.
template <int D, bool COARSE, int WAVES, int SLOTS>
__global__ __launch_bounds__(WAVES * kWave) void bwd_dq_tr_kernel(
    const void* __restrict__ qin, const void* __restrict__ gin, const void* __restrict__ kin,
    const void* __restrict__ vin, const int32_t* __restrict__ idx,
    const float* __restrict__ ld, const float* __restrict__ dqp, void* __restrict__ dq, int nb,
    int m, long long rows, float scale, float scale_log2) {
  using Cfg = TileCfg<BF16, D>;
  using elem = typename Cfg::elem;
  using R = RawB<D>;
  constexpr int KC = Cfg::kKChunks, VC = Cfg::kVChunks, NT = Cfg::kNT;
  constexpr int TB = R::TB, N = 2 * KC;                     // loads per tile
  constexpr int SLOT = 2 * TB;
  static_assert(KC == R::KC && KC <= 4 && VC <= 4, "raw tiles of d <= 64");
  static_assert(SLOTS == 1 || SLOTS == 2, "tiles in flight per wave");
  __shared__ __attribute__((aligned(16))) unsigned char slots[WAVES][SLOTS][SLOT];
  __shared__ __attribute__((aligned(16))) float addl[WAVES][COARSE ? add_lds_floats(D) : 1];
  extern __shared__ int32_t sidx_all[];
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id(), jq = lane & 31;
  const long long g = xcd_remap(blockIdx.x, gridDim.x) * (long long)WAVES + w;
  if (g >= rows) return;                                    // no workgroup barriers below
  const long long bh = g / nb;
  if constexpr (COARSE) prefetch_vec_lds<D>(dqp + g * D, (lptr_t)addl[w]);
  int32_t* myidx = sidx_all + w * m;
  const int cnt = stage_selection(idx + g * m, m, nb, myidx);

  u32x4 qf[KC], gf[KC];
  load_rows<BF16, D>(reinterpret_cast<const elem*>(qin) + g * 32 * D, qf);
  load_rows<BF16, D>(reinterpret_cast<const elem*>(gin) + g * 32 * D, gf);
  const float lq = ld[g * 64 + jq], dl = ld[g * 64 + 32 + jq];
  f32x16 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.0f;

  R ro;
  ro.init();
  const i32x4 krs = buffer_rsrc(static_cast<const char*>(kin) + (size_t)bh * nb * TB, (unsigned)nb * TB);
  const i32x4 vrs = buffer_rsrc(static_cast<const char*>(vin) + (size_t)bh * nb * TB, (unsigned)nb * TB);
  const uint32_t a0 = lds_addr(slots[w][0]);
  auto issue = [&](int y, int sl) {
    const lptr_t dst = (lptr_t)slots[w][sl];
    copy_raw_pair_buf<KC, R::KP>(krs, vrs, (unsigned)y * TB, (unsigned)y * TB, ro.cp, dst, dst + TB);
  };
#pragma unroll
  for (int t = 0; t < SLOTS; ++t)
    if (cnt > t) issue(wave_uniform(myidx[t]), t);
  for (int i = 0; i < cnt; ++i) {
    if (SLOTS == 2 && i + 1 < cnt) wait_loads<N>();         // tile i landed, i+1 may not have
    else wait_loads<0>();
    const uint32_t base = a0 + (uint32_t)((i % SLOTS) * SLOT);
    u32x4 kf[KC], vf[KC], tf[VC];
    raw_rows<0>(base, ro.rr, kf);
    raw_rows<TB>(base, ro.rr, vf);
    RawTrB<D, 0, 0, VC>::run(base, ro.tr, tf);
    lds_done(kf);
    lds_done(vf);
    lds_done(tf);
    if (i + SLOTS < cnt) issue(wave_uniform(myidx[i + SLOTS]), i % SLOTS);
    const f32x16 s = mfma_abt<BF16, KC>(kf, qf);
    const f32x16 pv = mfma_abt<BF16, KC>(vf, gf);
    float ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
      ds[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -lq)) * (pv[r] - dl);
    uint32_t pk[8];
    pack16(ds, pk);
    mfma_acc_bf16<NT>(acc, pk, [&](int c) { return tf[c]; });
  }
  wait_loads<0>();
  store_block<BF16, D>(reinterpret_cast<elem*>(dq) + g * 32 * D, acc, scale, COARSE ? addl[w] : nullptr);
}

// dK, dV (bf16, d <= 64): one wave per column block; a slot holds the raw
// tiles Q_x and G_x and block-row x's bias operands (Q^T and G^T are read
// transposed). The log normalisers and deltas enter the two products of a
// tile through one more matrix-core step each (A: the queries' bias operands,
// B: ones at the positions of the first or of the second triple), so the
// products come out as Q_i.K_j - L_i/c and G_i.V_j - delta_i, and each lane
// needs one 16-byte read for the 16 queries it holds.
template <int D, bool COARSE, int WAVES, int SLOTS>
__global__ __launch_bounds__(WAVES * kWave) void bwd_dkdv_tr_kernel(
    const void* __restrict__ kin, const void* __restrict__ vin, const void* __restrict__ qin,
    const void* __restrict__ gin, const uint32_t* __restrict__ bits,
    const uint32_t* __restrict__ bias, const float* __restrict__ dkp, const float* __restrict__ dvp,
    void* __restrict__ dk, void* __restrict__ dv, int nb, long long rows, float scale,
    float scale_log2) {
  using Cfg = TileCfg<BF16, D>;
  using elem = typename Cfg::elem;
  using R = RawB<D>;
  constexpr int KC = Cfg::kKChunks, VC = Cfg::kVChunks, NT = Cfg::kNT;
  constexpr int TB = R::TB, RB = 32 * 16;                   // bytes of a raw tile, of a block-row's bias operands
  constexpr int N = 2 * KC + 2;                             // loads per tile
  constexpr int SLOT = 2 * TB + RB;
  static_assert(KC == R::KC && KC <= 4 && VC <= 4, "raw tiles of d <= 64");
  static_assert(SLOTS == 1 || SLOTS == 2, "tiles in flight per wave");
  __shared__ __attribute__((aligned(16))) unsigned char slots[WAVES][SLOTS][SLOT];
  __shared__ __attribute__((aligned(16))) float addl[WAVES][2][COARSE ? add_lds_floats(D) : 1];
  extern __shared__ int32_t sidx_all[];
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id();
  const long long gy = xcd_remap(blockIdx.x, gridDim.x) * (long long)WAVES + w;
  if (gy >= rows) return;                                   // no workgroup barriers below
  const long long bh = gy / nb;
  if constexpr (COARSE) {
    prefetch_vec_lds<D>(dkp + gy * D, (lptr_t)addl[w][0]);
    prefetch_vec_lds<D>(dvp + gy * D, (lptr_t)addl[w][1]);
  }
  const int y = (int)(gy - bh * nb);
  const long long hb = bh * nb;
  const int nbw = (nb + 31) / 32;

  // block-rows whose selection holds y, ascending
  int32_t* myx = sidx_all + w * nb;
  const int cnt = column_list(bits, hb, nbw, y, nb, myx);

  u32x4 kf[KC], vf[KC];
  load_rows<BF16, D>(reinterpret_cast<const elem*>(kin) + gy * 32 * D, kf);
  load_rows<BF16, D>(reinterpret_cast<const elem*>(vin) + gy * 32 * D, vf);
  f32x16 ak[NT], av[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) ak[t][r] = av[t][r] = 0.0f;
  // B operands of the bias steps: lane l holds B[k = 8 (l/32) + e][l % 32]
  const bool lo_half = lane < 32;
  const u32x4 ones_l = lo_half ? u32x4{0x3F803F80u, 0x00003F80u, 0u, 0u} : u32x4{0u, 0u, 0u, 0u};
  const u32x4 ones_d = lo_half ? u32x4{0u, 0x3F800000u, 0x3F803F80u, 0u} : u32x4{0u, 0u, 0u, 0u};

  R ro;
  ro.init();
  const i32x4 qrs = buffer_rsrc(static_cast<const char*>(qin) + (size_t)hb * TB, (unsigned)nb * TB);
  const i32x4 grs = buffer_rsrc(static_cast<const char*>(gin) + (size_t)hb * TB, (unsigned)nb * TB);
  const i32x4 brs = buffer_rsrc(reinterpret_cast<const char*>(bias) + (size_t)hb * RB, (unsigned)nb * RB);
  const uint32_t a0 = lds_addr(slots[w][0]);
  const uint32_t boff = (uint32_t)(2 * TB) + 16u * (lane & 31);   // this lane's query's bias operand
  auto issue = [&](int x, int sl) {
    const lptr_t dst = (lptr_t)slots[w][sl];
    copy_raw_pair_buf<KC, R::KP>(qrs, grs, (unsigned)x * TB, (unsigned)x * TB, ro.cp, dst, dst + TB);
    mra_raw_buffer_load_lds(brs, dst + 2 * TB, 4, lane * 4, x * RB, 0, 0);
    mra_raw_buffer_load_lds(brs, dst + 2 * TB + 256, 4, lane * 4, x * RB + 256, 0, 0);
  };
#pragma unroll
  for (int t = 0; t < SLOTS; ++t)
    if (cnt > t) issue(wave_uniform(myx[t]), t);
  for (int i = 0; i < cnt; ++i) {
    if (SLOTS == 2 && i + 1 < cnt) wait_loads<N>();         // tile i landed, i+1 may not have
    else wait_loads<0>();
    const uint32_t base = a0 + (uint32_t)((i % SLOTS) * SLOT);
    u32x4 qa[KC], ga[KC], qt[VC], gtc[VC], ba[1];
    raw_rows<0>(base, ro.rr, qa);
    raw_rows<TB>(base, ro.rr, ga);
    RawTrB<D, 0, 0, VC>::run(base, ro.tr, qt);
    RawTrB<D, TB, 0, VC>::run(base, ro.tr, gtc);
    ba[0] = lds_read16<0>(base + boff);
    lds_done(qa);
    lds_done(ga);
    lds_done(qt);
    lds_done(gtc);
    lds_done(ba);
    if (i + SLOTS < cnt) issue(wave_uniform(myx[i + SLOTS]), i % SLOTS);
    const f32x16 s = mfma_abt_from<KC>(qa, kf, ba[0], ones_l);   // lane: key, 16 queries
    const f32x16 pv = mfma_abt_from<KC>(ga, vf, ba[0], ones_d);
    float a[16], ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      a[r] = __builtin_amdgcn_exp2f(s[r] * scale_log2);
      ds[r] = a[r] * pv[r];
    }
    uint32_t pa8[8], pd8[8];
    pack16(a, pa8);
    pack16(ds, pd8);
    mfma_acc_bf16<NT>(av, pa8, [&](int c) { return gtc[c]; });
    mfma_acc_bf16<NT>(ak, pd8, [&](int c) { return qt[c]; });
  }
  wait_loads<0>();
  store_block<BF16, D>(reinterpret_cast<elem*>(dk) + gy * 32 * D, ak, scale, COARSE ? addl[w][0] : nullptr);
  store_block<BF16, D>(reinterpret_cast<elem*>(dv) + gy * 32 * D, av, 1.0f, COARSE ? addl[w][1] : nullptr);
}

// bfloat16, d = 128: raw 8 KB tiles of 32 rows x 256 bytes under the same
// kind of swizzle (block b of row r at b ^ (4 (r mod 4) + (r / 4 mod 4)):
// sixteen consecutive rows take sixteen positions for the row reads, four
// consecutive rows four groups of four for the transposed reads; copy offsets
// of period 4). A tile's operands are too many registers at this width to be
// read at once, so each is read just before its products: the row chunks of
// one tile, then of the other, then the transposed chunks.

// dQ (bf16, d = 128): one wave per block-row, one slot per wave (K_y and V_y);
// the next tile is copied once the current one has been read.
template <bool COARSE, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void bwd_dq_tr128_kernel(
    const void* __restrict__ qin, const void* __restrict__ gin, const void* __restrict__ kin,
    const void* __restrict__ vin, const int32_t* __restrict__ idx,
    const float* __restrict__ ld, const float* __restrict__ dqp, void* __restrict__ dq, int nb,
    int m, long long rows, float scale, float scale_log2) {
  constexpr int D = 128;
  using Cfg = TileCfg<BF16, D>;
  using elem = typename Cfg::elem;
  using R = RawB<D>;
  constexpr int KC = Cfg::kKChunks, VC = Cfg::kVChunks, NT = Cfg::kNT;
  constexpr int TB = R::TB;
  static_assert(KC == R::KC && VC == KC, "row and transposed chunks of a tile");
  __shared__ __attribute__((aligned(16))) unsigned char slots[WAVES][2 * TB];
  __shared__ __attribute__((aligned(16))) float addl[WAVES][COARSE ? D : 1];
  extern __shared__ int32_t sidx_all[];
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id(), jq = lane & 31;
  const long long g = xcd_remap(blockIdx.x, gridDim.x) * (long long)WAVES + w;
  if (g >= rows) return;                                    // no workgroup barriers below
  const long long bh = g / nb;
  if constexpr (COARSE) prefetch_vec_lds<D>(dqp + g * D, (lptr_t)addl[w]);
  int32_t* myidx = sidx_all + w * m;
  const int cnt = stage_selection(idx + g * m, m, nb, myidx);

  u32x4 qf[KC], gf[KC];
  load_rows<BF16, D>(reinterpret_cast<const elem*>(qin) + g * 32 * D, qf);
  load_rows<BF16, D>(reinterpret_cast<const elem*>(gin) + g * 32 * D, gf);
  const float lq = ld[g * 64 + jq], dl = ld[g * 64 + 32 + jq];
  f32x16 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.0f;

  R ro;
  ro.init();
  const i32x4 krs = buffer_rsrc(static_cast<const char*>(kin) + (size_t)bh * nb * TB, (unsigned)nb * TB);
  const i32x4 vrs = buffer_rsrc(static_cast<const char*>(vin) + (size_t)bh * nb * TB, (unsigned)nb * TB);
  const uint32_t base = lds_addr(slots[w]);
  const lptr_t kdst = (lptr_t)slots[w], vdst = kdst + TB;
  // the slot's halves are refilled separately: V_y's as soon as its rows are
  // read (they are read first), K_y's once its rows and K_y^T are read
  if (cnt > 0) {
    const int y = wave_uniform(myidx[0]);
    copy_raw_buf<KC, R::KP>(vrs, (unsigned)y * TB, ro.cp, vdst);
    copy_raw_buf<KC, R::KP>(krs, (unsigned)y * TB, ro.cp, kdst);
  }
  for (int i = 0; i < cnt; ++i) {
    wait_loads<KC>();                                       // V_y landed (K_y may be in flight)
    const int yn = i + 1 < cnt ? wave_uniform(myidx[i + 1]) : 0;
    u32x4 op[KC];
    raw_rows<TB>(base, ro.rr, op);                          // V_y rows
    lds_done(op);
    if (i + 1 < cnt) {
      copy_raw_buf<KC, R::KP>(vrs, (unsigned)yn * TB, ro.cp, vdst);
      wait_loads<KC>();                                     // K_y landed
    } else {
      wait_loads<0>();
    }
    const f32x16 pv = mfma_abt<BF16, KC>(op, gf);
    raw_rows<0>(base, ro.rr, op);                           // K_y rows
    lds_done(op);
    const f32x16 s = mfma_abt<BF16, KC>(op, qf);
    RawTrB<D, 0, 0, VC>::run(base, ro.tr, op);             // K_y^T
    lds_done(op);
    if (i + 1 < cnt) copy_raw_buf<KC, R::KP>(krs, (unsigned)yn * TB, ro.cp, kdst);
    float ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
      ds[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -lq)) * (pv[r] - dl);
    uint32_t pk[8];
    pack16(ds, pk);
    mfma_acc_bf16<NT>(acc, pk, [&](int c) { return op[c]; });
  }
  wait_loads<0>();
  store_block<BF16, D>(reinterpret_cast<elem*>(dq) + g * 32 * D, acc, scale, COARSE ? addl[w] : nullptr);
}

// dK, dV (bf16, d = 128): one wave per column block, two slots (raw Q_x, G_x
// and the block-row's bias operands), the per-query terms entering the
// products as in bwd_dkdv_tr_kernel.
template <bool COARSE>
__global__ __launch_bounds__(kWave) void bwd_dkdv_tr128_kernel(
    const void* __restrict__ kin, const void* __restrict__ vin, const void* __restrict__ qin,
    const void* __restrict__ gin, const uint32_t* __restrict__ bits,
    const uint32_t* __restrict__ bias, const float* __restrict__ dkp, const float* __restrict__ dvp,
    void* __restrict__ dk, void* __restrict__ dv, int nb, long long rows, float scale,
    float scale_log2) {
  constexpr int D = 128;
  using Cfg = TileCfg<BF16, D>;
  using elem = typename Cfg::elem;
  using R = RawB<D>;
  constexpr int KC = Cfg::kKChunks, VC = Cfg::kVChunks, NT = Cfg::kNT;
  constexpr int TB = R::TB, RB = 32 * 16;
  constexpr int N = 2 * KC + 2;                             // loads per tile
  constexpr int SLOT = 2 * TB + RB;
  static_assert(KC == R::KC && VC == KC, "row and transposed chunks of a tile");
  __shared__ __attribute__((aligned(16))) unsigned char slots[2][SLOT];
  __shared__ __attribute__((aligned(16))) float addl[2][COARSE ? D : 1];
  extern __shared__ int32_t sidx_all[];
  const int lane = lane_id();
  const long long gy = xcd_remap(blockIdx.x, gridDim.x);
  if (gy >= rows) return;
  const long long bh = gy / nb;
  if constexpr (COARSE) {
    prefetch_vec_lds<D>(dkp + gy * D, (lptr_t)addl[0]);
    prefetch_vec_lds<D>(dvp + gy * D, (lptr_t)addl[1]);
  }
  const int y = (int)(gy - bh * nb);
  const long long hb = bh * nb;
  const int nbw = (nb + 31) / 32;

  // block-rows whose selection holds y, ascending
  int32_t* myx = sidx_all;
  const int cnt = column_list(bits, hb, nbw, y, nb, myx);

  u32x4 kf[KC], vf[KC];
  load_rows<BF16, D>(reinterpret_cast<const elem*>(kin) + gy * 32 * D, kf);
  load_rows<BF16, D>(reinterpret_cast<const elem*>(vin) + gy * 32 * D, vf);
  f32x16 ak[NT], av[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) ak[t][r] = av[t][r] = 0.0f;
  const bool lo_half = lane < 32;
  const u32x4 ones_l = lo_half ? u32x4{0x3F803F80u, 0x00003F80u, 0u, 0u} : u32x4{0u, 0u, 0u, 0u};
  const u32x4 ones_d = lo_half ? u32x4{0u, 0x3F800000u, 0x3F803F80u, 0u} : u32x4{0u, 0u, 0u, 0u};

  R ro;
  ro.init();
  const i32x4 qrs = buffer_rsrc(static_cast<const char*>(qin) + (size_t)hb * TB, (unsigned)nb * TB);
  const i32x4 grs = buffer_rsrc(static_cast<const char*>(gin) + (size_t)hb * TB, (unsigned)nb * TB);
  const i32x4 brs = buffer_rsrc(reinterpret_cast<const char*>(bias) + (size_t)hb * RB, (unsigned)nb * RB);
  const uint32_t a0 = lds_addr(slots[0]);
  const uint32_t boff = (uint32_t)(2 * TB) + 16u * (lane & 31);
  auto issue = [&](int x, int sl) {
    const lptr_t dst = (lptr_t)slots[sl];
    copy_raw_pair_buf<KC, R::KP>(qrs, grs, (unsigned)x * TB, (unsigned)x * TB, ro.cp, dst, dst + TB);
    mra_raw_buffer_load_lds(brs, dst + 2 * TB, 4, lane * 4, x * RB, 0, 0);
    mra_raw_buffer_load_lds(brs, dst + 2 * TB + 256, 4, lane * 4, x * RB + 256, 0, 0);
  };
  if (cnt > 0) issue(wave_uniform(myx[0]), 0);
  if (cnt > 1) issue(wave_uniform(myx[1]), 1);
  for (int i = 0; i < cnt; ++i) {
    if (i + 1 < cnt) wait_loads<N>();                       // tile i landed, i+1 may not have
    else wait_loads<0>();
    const uint32_t base = a0 + (uint32_t)((i & 1) * SLOT);
    u32x4 op[KC], ba[1];
    ba[0] = lds_read16<0>(base + boff);
    raw_rows<0>(base, ro.rr, op);                           // Q_x rows
    lds_done(ba);
    lds_done(op);
    const f32x16 s = mfma_abt_from<KC>(op, kf, ba[0], ones_l);   // lane: key, 16 queries
    raw_rows<TB>(base, ro.rr, op);                          // G_x rows
    lds_done(op);
    const f32x16 pv = mfma_abt_from<KC>(op, vf, ba[0], ones_d);
    float a[16], ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      a[r] = __builtin_amdgcn_exp2f(s[r] * scale_log2);
      ds[r] = a[r] * pv[r];
    }
    uint32_t pa8[8], pd8[8];
    pack16(a, pa8);
    pack16(ds, pd8);
    RawTrB<D, 0, 0, VC>::run(base, ro.tr, op);             // Q_x^T
    lds_done(op);
    mfma_acc_bf16<NT>(ak, pd8, [&](int c) { return op[c]; });
    RawTrB<D, TB, 0, VC>::run(base, ro.tr, op);            // G_x^T
    lds_done(op);
    if (i + 2 < cnt) issue(wave_uniform(myx[i + 2]), i & 1);   // the slot has been read
    mfma_acc_bf16<NT>(av, pa8, [&](int c) { return op[c]; });
  }
  wait_loads<0>();
  store_block<BF16, D>(reinterpret_cast<elem*>(dk) + gy * 32 * D, ak, scale, COARSE ? addl[0] : nullptr);
  store_block<BF16, D>(reinterpret_cast<elem*>(dv) + gy * 32 * D, av, 1.0f, COARSE ? addl[1] : nullptr);
}

// ---------------------------------------------------------------------------
template <int DT, int D, bool COARSE>
static void launch_tiles_t(const BwdArgs& A, hipStream_t stream) {
  using Cfg = TileCfg<DT, D>;
  const int nb = A.n / kBlock;
  const long long rows = A.bh * nb;
  const float scale = (float)(1.0 / sqrt((double)D));
  const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
  const unsigned wgs = (unsigned)((rows + kBwdTileWaves - 1) / kBwdTileWaves);
  const size_t smem_dq = (size_t)kBwdTileWaves * A.m * sizeof(int32_t);
  constexpr int W = kBwdTileWaves;
  if constexpr (DT == BF16 && Cfg::kKChunks <= 4 && Cfg::kVChunks <= 4) {
    bwd_dq_tr_kernel<D, COARSE, W, kDqSlots><<<wgs, W * kWave, smem_dq, stream>>>(
        A.q, A.dout, A.k, A.v, A.idx, A.ld, A.dqp, A.dq, nb, A.m, rows, scale, scale_log2);
    // one wave per workgroup in every column pass: column lists differ in
    // length (a workgroup keeps its resources until its longest list is
    // done), rows all have m tiles
    bwd_dkdv_tr_kernel<D, COARSE, 1, kDkdvSlots><<<(unsigned)rows, kWave, nb * sizeof(int32_t), stream>>>(
        A.k, A.v, A.q, A.dout, A.bits, A.bias, A.dkp, A.dvp, A.dk, A.dv, nb, rows, scale,
        scale_log2);
  } else if constexpr (DT == BF16 && D == 128) {
    bwd_dq_tr128_kernel<COARSE, W><<<wgs, W * kWave, smem_dq, stream>>>(
        A.q, A.dout, A.k, A.v, A.idx, A.ld, A.dqp, A.dq, nb, A.m, rows, scale, scale_log2);
    bwd_dkdv_tr128_kernel<COARSE><<<(unsigned)rows, kWave, nb * sizeof(int32_t), stream>>>(
        A.k, A.v, A.q, A.dout, A.bits, A.bias, A.dkp, A.dvp, A.dk, A.dv, nb, rows, scale, scale_log2);
  } else if constexpr (Cfg::kKChunks <= 4 && Cfg::kVChunks <= 4) {
    bwd_dq_stream_kernel<DT, D, COARSE, W><<<wgs, W * kWave, smem_dq, stream>>>(
        A.q, A.dout, A.k_row, A.v_row, A.k_t, A.idx, A.ld, A.dqp, A.dq, nb, A.m, rows, scale,
        scale_log2);
    bwd_dkdv_stream_kernel<DT, D, COARSE, 1><<<(unsigned)rows, kWave, nb * sizeof(int32_t), stream>>>(
        A.k, A.v, A.q_row, A.g_row, A.q_t, A.g_t, A.bits, A.ld, A.dkp, A.dvp, A.dk, A.dv, nb, rows,
        scale, scale_log2);
  } else {
    bwd_dq_kernel<DT, D, COARSE><<<wgs, W * kWave, smem_dq, stream>>>(
        A.q, A.dout, A.k_row, A.v_row, A.k_t, A.idx, A.ld, A.dqp, A.dq, nb, A.m, rows, scale,
        scale_log2);
    bwd_dkdv_kernel<DT, D, COARSE, 1><<<(unsigned)rows, kWave, nb * sizeof(int32_t), stream>>>(
        A.k, A.v, A.q_row, A.g_row, A.q_t, A.g_t, A.bits, A.ld, A.dkp, A.dvp, A.dk, A.dv, nb, rows,
        scale, scale_log2);
  }
}

template <int DT, int D>
static void launch_bwd_t(const BwdArgs& A, hipStream_t stream) {
  const int nb = A.n / kBlock;
  const float scale = (float)(1.0 / sqrt((double)D));
  const long long groups = (nb + kBwdRows - 1) / kBwdRows;
  const unsigned wg_rows = (unsigned)(A.bh * groups);
  if (A.coarse) {
    bwd_rows_kernel<DT, D, true><<<wg_rows, kBwdRows * kWave, 0, stream>>>(
        A.dout, A.out, A.lse, A.idx, A.qp, A.kp, A.vp, A.ld, A.bias, A.bits, A.gh, A.W, A.dS, A.dqp, nb,
        A.m, scale);
    const unsigned wg_cols = (unsigned)(A.bh * ((nb + kBwdCols - 1) / kBwdCols));
    bwd_cols_kernel<D><<<wg_cols, ColsCfg<D>::kWaves * kWave, 0, stream>>>(
        A.qp, A.gh, A.W, A.dS, A.dkp, A.dvp, nb, scale);
    launch_tiles_t<DT, D, true>(A, stream);
  } else {
    bwd_rows_kernel<DT, D, false><<<wg_rows, kBwdRows * kWave, 0, stream>>>(
        A.dout, A.out, A.lse, A.idx, A.qp, A.kp, A.vp, A.ld, A.bias, A.bits, A.gh, A.W, A.dS, A.dqp, nb,
        A.m, scale);
    launch_tiles_t<DT, D, false>(A, stream);
  }
}

hipError_t launch_bwd(const BwdArgs& A, hipStream_t stream) {
  hipError_t e = hipSuccess;
  if (A.dtype == BF16) {
    // the tile passes read raw tiles of Q, K, V and G = dZ: only the pooled
    // rows of the coarse term
    if (A.coarse && !A.pooled_in)
      e = launch_pool(A.q, A.k, A.v, A.qp, A.kp, A.vp, nullptr, A.bh, A.n, A.d, A.dtype, stream);
  } else {
    // pooled rows (unless given) and packed operands of Q, K, V and G = dZ
    const bool pool = A.coarse && !A.pooled_in;
    const PackJob jobs[4] = {{A.q, pool ? A.qp : nullptr, A.q_row, A.q_t},
                             {A.k, pool ? A.kp : nullptr, A.k_row, A.k_t},
                             {A.v, pool ? A.vp : nullptr, A.v_row, nullptr},
                             {A.dout, nullptr, A.g_row, A.g_t}};
    e = launch_pack(jobs, 4, A.bh, A.n, A.d, A.dtype, stream);
  }
  if (e != hipSuccess) return e;
  if (A.dtype == BF16) {
    if (A.d == 32) launch_bwd_t<BF16, 32>(A, stream);
    else if (A.d == 64) launch_bwd_t<BF16, 64>(A, stream);
    else launch_bwd_t<BF16, 128>(A, stream);
  } else {
    if (A.d == 32) launch_bwd_t<F32, 32>(A, stream);
    else if (A.d == 64) launch_bwd_t<F32, 64>(A, stream);
    else launch_bwd_t<F32, 128>(A, stream);
  }
  return hipGetLastError();
}

}  // namespace mra
