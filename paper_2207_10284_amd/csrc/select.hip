// Per block-row selection and the low-resolution term of MRA-2.
//
// Selection (Sec. 4.2, Alg. 1, per block-row): keep the `m` column blocks with
// the largest coarse logit S~[x, .]; equal scores prefer the lower index;
// the kept indices are written in ascending order.
//
// Low-resolution term (Sec. 4.3, Alg. 2 at scale b over the blocks that were
// not refined; eq. actual_approx_mat_form gives every such block b columns):
//   M = max S~ over unselected blocks, c = sum b e^{S~ - M},
//   L = sum b e^{S~ - M} V~_y.
//
// One workgroup owns 16 consecutive block-rows of one head: 8 waves with two
// rows each (one row per wave for heads of more than 1024 blocks). Lane l of a
// row's wave holds the row's scores for blocks y = 64j + l in registers:
// loaded from S~, or (fused modes) computed as 16 x 16 tiles on the float64
// matrix cores with the same tile routine as the coarse-logit kernel (so the
// same bits), the waves taking tiles in turn with their operands in
// registers, then passed through LDS. The selection is a radix search for the
// m-th largest order-preserving 32-bit key (32 rounds of ballot + popcount
// over the registers), then one ascending sweep that resolves ties at the
// threshold by index and compacts the kept indices with prefix popcounts. Max
// and sum use DPP / lane-swap reductions (no LDS). L = W V~ is formed on the
// float32 matrix cores (16x16x4): the weights b e^{S~ - M} (0 where selected)
// of the 16 rows go to LDS once, and the waves split the dims and the blocks
// between them, so V~ is read once per workgroup. Workgroups of one head stay
// on one XCD. Every mode runs the same arithmetic in the same order, so the
// fused forward step is bit-identical to separate score, select and
// coarse-term calls. A fused select-only mode serves MRA-2-s.
#include "coarse_tile.h"
#include "kernels.h"

namespace mra {

enum RowsMode { kSelectOnly = 0, kTermOnly = 1, kFused = 2, kFusedSelect = 3 };
constexpr int kRows = 16;                 // block-rows (waves) per workgroup
constexpr int kChunk = 64;                // score columns per register
constexpr int kU = 8;                     // coarse-term steps per batch of V~ loads (two float4 of weights)

typedef float f32x4v __attribute__((ext_vector_type(4)));

// LDS of a workgroup: the 16 rows' scores (fused modes) and then their
// weights, [16][64 JMAX] floats (zero past nb), column c of row r stored at
// c ^ 4r: rows start on the same bank, and the swizzle (bits 2-5 of the
// column, so groups of four stay contiguous and every column stays in its
// group of 64) keeps the coarse term's 16-byte operand reads across the 16
// rows free of bank conflicts without padding; followed by the partial sums
// of L ((16 / (d/16)) x 16 x d floats).
__host__ __device__ constexpr int rows_ldc(int jmax) { return 64 * jmax; }
__host__ __device__ constexpr int rows_col(int r, int c) { return c ^ ((r & 15) << 2); }

struct RowsSmem {
  size_t part_off, bytes;
};

// The select-only mode uses no LDS. In the fused modes the region after the
// score rows first holds the 16 query rows in float64 ([16][d], element c of
// row r at c ^ 2r: pairs stay contiguous, and the 16-byte reads of the 16
// rows fall on different banks), then the partial sums of L. Unpadded, the
// two regions of a 16-block-row workgroup at nb <= 1024 and d = 128 take
// exactly half of a CU's LDS, so two such workgroups share a CU.
__host__ __device__ constexpr int rows_ldq(int d) { return d; }
__host__ __device__ constexpr int rows_qcol(int r, int c) { return c ^ ((r & 15) << 1); }

static RowsSmem rows_smem(int jmax, int nw, int mode, int d) {
  RowsSmem L{};
  if (mode == kSelectOnly) return L;
  L.part_off = ((size_t)kRows * rows_ldc(jmax) * sizeof(float) + 15) & ~size_t(15);
  const size_t part = mode == kTermOnly || mode == kFused ? (size_t)nw * 16 * 16 * sizeof(float) : 0;
  const size_t qd = mode == kFused || mode == kFusedSelect ? (size_t)kRows * rows_ldq(d) * sizeof(double) : 0;
  L.bytes = L.part_off + (part > qd ? part : qd);
  return L;
}

template <int D, int MODE, int JMAX, int RPW>
__global__ __launch_bounds__(kRows / RPW * kWave) void rows_kernel(
    const float* __restrict__ S, const float* __restrict__ qp, const float* __restrict__ kp,
    int32_t* __restrict__ idx_out, const int32_t* __restrict__ idx_in,
    const float* __restrict__ vp, float* __restrict__ cmax, float* __restrict__ csum,
    float* __restrict__ cvec, int nb, int m, int part_off, double scale) {
  constexpr int NW = kRows / RPW;                                  // waves per workgroup
  constexpr int NTH = NW * kWave;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  float* Cb = reinterpret_cast<float*>(smem);                      // [16][ldc] scores, then weights
  const int tid = threadIdx.x;
  const int w = wave_uniform(tid / kWave);
  const int lane = lane_id();
  const int groups = (nb + kRows - 1) / kRows;
  const long long lwg = xcd_remap(blockIdx.x, gridDim.x);
  const long long bh = lwg / groups;
  const int x0 = (int)(lwg - bh * groups) * kRows;
  const int rows = min(kRows, nb - x0);
  const long long g0 = bh * nb + x0;                               // first global block-row
  const int J = (nb + kChunk - 1) / kChunk;
  // this wave's rows: w + NW * i, i < RPW
  auto row_of = [&](int i) { return w + NW * i; };

  // Phase 4's B operands (V~ values, kU steps per batch): for heads of up to
  // 512 blocks the first batch is loaded here so its latency hides behind
  // phases 1-3 (larger heads keep those registers for phase 1).
  constexpr bool kEarlyB = JMAX <= 8;
  constexpr int NTD = D / 16, KQ = NW / NTD;
  static_assert(KQ >= 1 && NW % NTD == 0, "waves cover the dim tiles");
  const int nt = w % NTD, kq = w / NTD;
  const int ar = lane & 15, ak = lane >> 4;
  constexpr int ldc = rows_ldc(JMAX), BPW = 2 * JMAX / KQ;            // batches per wave
  static_assert(BPW * KQ == 2 * JMAX, "whole batches");
  float ba[kU];
  // V~ rows of this wave's batch u: blocks 32 (kq + KQ u) + 8 ak + e, e < kU,
  // as buffer loads from the head's V~ (one lane offset per batch, the steps
  // in the immediate offset; rows past nb read as zero, and their weights are
  // zero too)
  i32x4 vrs = {0, 0, 0, 0};
  int vlane = 0;
  if constexpr (MODE == kFused || MODE == kTermOnly) {
    vrs = buffer_rsrc(vp + bh * (long long)nb * D, (unsigned)nb * D * (unsigned)sizeof(float));
    vlane = ((4 * kU * kq + kU * ak) * D + 16 * nt + ar) * (int)sizeof(float);
  }
  auto load_b = [&](int u, float (&b)[kU]) {
    const int vo = vlane + u * (4 * kU * KQ * D * (int)sizeof(float));
#pragma unroll
    for (int e = 0; e < kU; ++e) b[e] = mra_raw_buffer_load_f32(vrs, vo + e * D * (int)sizeof(float), 0, 0);
  };
  if constexpr ((MODE == kFused || MODE == kTermOnly) && kEarlyB) load_b(0, ba);

  // ---- phase 1: the rows' scores into registers, s[i][j] for y = 64j + lane
  float s[RPW][JMAX];
#pragma unroll
  for (int i = 0; i < RPW; ++i)
#pragma unroll
    for (int j = 0; j < JMAX; ++j) s[i][j] = 0.0f;
  if constexpr (MODE == kFused || MODE == kFusedSelect) {
    // 16 x 16 tiles of S~ (the 16 rows x 16 keys) on the float64 matrix
    // cores, tile t by wave t % NW, operands in registers straight from the
    // pooled rows, results through LDS
    constexpr int NQ = D / 16;
    const int r = lane & 15;
    const float* kh = kp + bh * (long long)nb * D;
    // the 16 query rows in float64, converted once (rows past the group
    // repeat the last one; their results are ignored)
    constexpr int LDQ = rows_ldq(D);
    double* Qd = reinterpret_cast<double*>(smem + part_off);
    for (int i = tid; i < kRows * D; i += NTH) {
      const int rr = i / D, c = i % D;
      Qd[rr * LDQ + rows_qcol(rr, c)] = (double)qp[(g0 + min(rr, rows - 1)) * D + c];
    }
    __syncthreads();
    const double* qrow = Qd + r * LDQ;
    const int qc0 = 4 * (lane >> 4), qx = rows_qcol(r, 0);
    const int ntile = (nb + 15) / 16;
    auto load_k = [&](int t, f32x4 (&kv)[NQ]) {                   // keys past nb: ignored columns
      coarse_load<D>(kh + (long long)min(16 * min(t, ntile - 1) + r, nb - 1) * D, kv);
    };
    auto tile = [&](int t, const f32x4 (&kv)[NQ]) {
      const f64x4 acc = coarse_tile_f64_qd<D>(qrow, qc0, qx, kv);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int rr = coarse_tile_row(lane, e);
        Cb[rr * ldc + rows_col(rr, 16 * t + r)] = coarse_round(acc[e], scale);
      }
    };
    // K~ one tile ahead where a wave takes several tiles and the registers
    // allow it (not at d = 128 with two rows per wave)
    if constexpr (4 * JMAX <= NW || (D == 128 && RPW == 2)) {
      for (int t = w; t < ntile; t += NW) {
        f32x4 kv[NQ];
        load_k(t, kv);
        tile(t, kv);
      }
    } else {
      f32x4 ka[NQ], kb[NQ];
      int t = w;
      if (t < ntile) load_k(t, ka);
      // unconditional loads (past the last tile: the last tile again), so the
      // load-counter waits stay exact
      while (t < ntile) {
        load_k(t + NW, kb);
        asm volatile("" ::: "memory");                            // loads stay ahead of the products
        tile(t, ka);
        t += NW;
        if (t >= ntile) break;
        load_k(t + NW, ka);
        asm volatile("" ::: "memory");
        tile(t, kb);
        t += NW;
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < JMAX; ++j) {
      if (j >= J) break;
#pragma unroll
      for (int i = 0; i < RPW; ++i)
        if (row_of(i) < rows && kChunk * j + lane < nb)
          s[i][j] = Cb[row_of(i) * ldc + rows_col(row_of(i), kChunk * j + lane)];
    }
  } else {
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
      if (row_of(i) >= rows) continue;
      const long long g = g0 + row_of(i);
#pragma unroll
      for (int j = 0; j < JMAX; ++j) {
        const int y = kChunk * j + lane;
        if (j < J && y < nb) s[i][j] = S[g * nb + y];
      }
    }
  }

  // ---- phase 2: selection flags sel[i] (bit j <-> y = 64j + lane)
  uint32_t sel[RPW];
#pragma unroll
  for (int i = 0; i < RPW; ++i) {
    sel[i] = 0;
    if (row_of(i) >= rows) continue;
    const long long g = g0 + row_of(i);
    if constexpr (MODE == kTermOnly) {
      // the row's list (any width, entries outside [0, nb) ignored) as a
      // bitmap in the row's part of the chunk buffer, 64 entries per step
      uint32_t* bm = reinterpret_cast<uint32_t*>(Cb) + row_of(i) * 64;   // nb <= 2048 bits
      bm[lane] = 0u;
      wave_lds_sync();
      for (int i0 = 0; i0 < m; i0 += kWave) {
        const int y = i0 + lane < m ? idx_in[g * m + i0 + lane] : -1;
        if (y >= 0 && y < nb) atomicOr(&bm[y >> 5], 1u << (y & 31));
      }
      wave_lds_sync();
#pragma unroll
      for (int j = 0; j < JMAX; ++j) {
        const int y = kChunk * j + lane;
        if (j < J && y < nb && ((bm[y >> 5] >> (y & 31)) & 1u)) sel[i] |= 1u << j;
      }
    } else {
      uint32_t key[JMAX];
#pragma unroll
      for (int j = 0; j < JMAX; ++j) key[j] = (j < J && kChunk * j + lane < nb) ? ordered_key(s[i][j]) : 0u;
      uint32_t T = 0;
      int need = 0;
      const bool all = (m == nb), none = (m == 0);
      if (!all && !none) {
        // Every valid key shares the bits above the highest bit in which the
        // row's largest and smallest keys differ, so the search starts there
        // with those bits set. Unused registers hold key 0, below every
        // candidate, so the counts need no range checks.
        float smax = -INFINITY, smin = INFINITY;
#pragma unroll
        for (int j = 0; j < JMAX; ++j)
          if (j < J && kChunk * j + lane < nb) {
            smax = fmaxf(smax, s[i][j]);
            smin = fminf(smin, s[i][j]);
          }
        const uint32_t kmax = __builtin_amdgcn_readfirstlane(ordered_key(wave_max(smax)));
        const uint32_t kmin = __builtin_amdgcn_readfirstlane(ordered_key(-wave_max(-smin)));
        const uint32_t diff = kmax ^ kmin;
        const int top = diff ? 31 - __builtin_clz(diff) : -1;
        T = top >= 0 ? kmax & ~((2u << top) - 1u) : kmax;
        for (int bit = top; bit >= 0; --bit) {
          const uint32_t cand = T | (1u << bit);
          int cnt = 0;
#pragma unroll
          for (int j = 0; j < JMAX; ++j) cnt += __popcll(__ballot(key[j] >= cand));
          if (cnt >= m) T = cand;
          if (cnt == m) break;               // exactly the m largest are >= T
        }
        int gt = 0;
#pragma unroll
        for (int j = 0; j < JMAX; ++j) gt += __popcll(__ballot(key[j] > T));
        need = m - gt;                       // keys equal to T still to take
      }
      int eq_seen = 0, written = 0;
#pragma unroll
      for (int j = 0; j < JMAX; ++j) {
        if (j < J) {                         // wave-uniform: unrolls fully
          const int y = kChunk * j + lane;
          const bool valid = y < nb;
          bool take;
          if (all) {
            take = valid;
          } else if (none) {
            take = false;
          } else {
            const bool eq = valid && key[j] == T;
            const uint64_t eqm = __ballot(eq);
            const int rank = eq_seen + __popcll(eqm & lanemask_lt());
            eq_seen += __popcll(eqm);
            take = valid && (key[j] > T || (eq && rank < need));
          }
          const uint64_t tm = __ballot(take);
          if (take && idx_out) idx_out[g * m + written + __popcll(tm & lanemask_lt())] = y;
          written += __popcll(tm);
          if (take) sel[i] |= 1u << j;
        }
      }
    }
  }
  if constexpr (MODE == kSelectOnly || MODE == kFusedSelect) return;

  // ---- phase 3: max, weights (kept in s[]) and their sum over unselected blocks
#pragma unroll
  for (int i = 0; i < RPW; ++i) {
    if (row_of(i) < rows) {
      const long long g = g0 + row_of(i);
      float M = -INFINITY;
#pragma unroll
      for (int j = 0; j < JMAX; ++j)
        if (j < J && kChunk * j + lane < nb && !((sel[i] >> j) & 1u)) M = fmaxf(M, s[i][j]);
      M = wave_max(M);
      const bool any = M != -INFINITY;
      float c = 0.0f;
#pragma unroll
      for (int j = 0; j < JMAX; ++j) {
        const int y = kChunk * j + lane;
        const bool unsel = j < J && y < nb && !((sel[i] >> j) & 1u);
        s[i][j] = (any && unsel) ? (float)kBlock * expf(s[i][j] - M) : 0.0f;
        c += s[i][j];
      }
      c = wave_sum(c);
      if (lane == 0) {
        cmax[g] = M;
        csum[g] = c;
      }
    } else {
#pragma unroll
      for (int j = 0; j < JMAX; ++j) s[i][j] = 0.0f;
    }
  }

  // ---- phase 4: L = W V~ on the float32 matrix cores (v_mfma_f32_16x16x4_f32,
  // A = W: 16 rows x 4 blocks from LDS, B = V~: 4 blocks x 16 dims straight
  // from the pooled rows, two batches of kU steps ahead). Wave w takes dim tile
  // nt = w % (D/16) and the 32-block batches kq + KQ u, u < BPW, for
  // kq = w / (D/16) (all 64 JMAX columns; the weights past nb are zero); the
  // per-wave partial sums are added in kq order at the end.
  __syncthreads();                                                 // every wave has read its scores
#pragma unroll
  for (int j = 0; j < JMAX; ++j) {
    if (j >= J) break;
#pragma unroll
    for (int i = 0; i < RPW; ++i)                                   // zero: inactive rows, blocks >= nb
      Cb[row_of(i) * ldc + rows_col(row_of(i), kChunk * j + lane)] = s[i][j];
  }
  for (int c = kChunk * J + lane; c < kChunk * JMAX; c += kWave)   // columns past the scores
    for (int i = 0; i < RPW; ++i) Cb[row_of(i) * ldc + rows_col(row_of(i), c)] = 0.0f;
  __syncthreads();
  if constexpr (!kEarlyB) load_b(0, ba);
  const float* wrow = Cb + ar * ldc;
  f32x4v acc = {0.0f, 0.0f, 0.0f, 0.0f};
  // batch u: step e takes block 32 (kq + KQ u) + 8 ak + e in lane group ak,
  // so each lane reads its kU weights as two 16-byte LDS reads
  auto steps = [&](int u, const float (&b)[kU]) {
    const int c0 = rows_col(ar, kU * ak + 4 * kU * (kq + KQ * u));  // c0 + 4 lands at c0 ^ 4
    const f32x4v a0 = *reinterpret_cast<const f32x4v*>(wrow + c0);
    const f32x4v a1 = *reinterpret_cast<const f32x4v*>(wrow + (c0 ^ 4));
#pragma unroll
    for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[e], b[e], acc, 0, 0, 0);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[e], b[4 + e], acc, 0, 0, 0);
  };
  // All BPW batches unrolled (no loop state for the compiler's load-counter
  // waits to merge), loads two batches ahead; the empty asm keeps the
  // compiler from sinking them below the products, which would expose their
  // latency.
  float bv[3][kU];
#pragma unroll
  for (int e = 0; e < kU; ++e) bv[0][e] = ba[e];
  if constexpr (BPW > 1) load_b(1, bv[1]);
#pragma unroll
  for (int u = 0; u < BPW; ++u) {
    if (u + 2 < BPW) load_b(u + 2, bv[(u + 2) % 3]);
    asm volatile("" ::: "memory");
    steps(u, bv[u % 3]);
  }
  // partial sums: lane holds rows 4*ak + e of dim 16*nt + ar
  float* part = reinterpret_cast<float*>(smem + part_off);         // [KQ][16][D]
#pragma unroll
  for (int e = 0; e < 4; ++e) part[(kq * kRows + 4 * ak + e) * D + 16 * nt + ar] = acc[e];
  __syncthreads();
  for (int i = tid; i < rows * D; i += NTH) {
    const int r = i / D, dm = i % D;
    float sum = part[r * D + dm];
#pragma unroll
    for (int q = 1; q < KQ; ++q) sum += part[(q * kRows + r) * D + dm];
    cvec[(g0 + r) * D + dm] = sum;
  }
}

template <int MODE, int JMAX>
static void launch_rows_j(const float* S, const float* qp, const float* kp, int32_t* idx_out,
                          const int32_t* idx_in, const float* vp, float* cmax, float* csum,
                          float* cvec, long long bh, int nb, int d, int m, hipStream_t stream) {
  const long long groups = (nb + kRows - 1) / kRows;
  const unsigned blocks = (unsigned)(bh * groups);
  constexpr int RPW = JMAX <= 16 ? 2 : 1;
  const RowsSmem L = rows_smem(JMAX, kRows / RPW, MODE, d);
  const double scale = 1.0 / sqrt((double)d);
  // two rows per wave (8 waves) while the scores fit in registers (nb <= 1024):
  // workgroups of 16 block-rows small enough that two or more share a CU, so
  // one's matrix-core phases overlap another's selection
#define MRA_ROWS_LAUNCH(DD)                                                                     \
  rows_kernel<DD, MODE, JMAX, RPW><<<blocks, 64 * kRows / RPW, L.bytes, stream>>>(            \
      S, qp, kp, idx_out, idx_in, vp, cmax, csum, cvec, nb, m, (int)L.part_off, scale)
  switch (d) {
    case 32: MRA_ROWS_LAUNCH(32); break;
    case 64: MRA_ROWS_LAUNCH(64); break;
    default: MRA_ROWS_LAUNCH(128); break;
  }
#undef MRA_ROWS_LAUNCH
}

// Score registers per lane: up to 2 (nb <= 128), 8 (nb <= 512), 16 (nb <= 1024)
// or 32 (nb <= 2048).
template <int MODE>
static hipError_t launch_rows(const float* S, const float* qp, const float* kp, int32_t* idx_out,
                              const int32_t* idx_in, const float* vp, float* cmax, float* csum,
                              float* cvec, long long bh, int nb, int d, int m, hipStream_t stream) {
  if (nb <= 128)
    launch_rows_j<MODE, 2>(S, qp, kp, idx_out, idx_in, vp, cmax, csum, cvec, bh, nb, d, m, stream);
  else if (nb <= 512)
    launch_rows_j<MODE, 8>(S, qp, kp, idx_out, idx_in, vp, cmax, csum, cvec, bh, nb, d, m, stream);
  else if (nb <= 1024)
    launch_rows_j<MODE, 16>(S, qp, kp, idx_out, idx_in, vp, cmax, csum, cvec, bh, nb, d, m, stream);
  else
    launch_rows_j<MODE, 32>(S, qp, kp, idx_out, idx_in, vp, cmax, csum, cvec, bh, nb, d, m, stream);
  return hipGetLastError();
}

hipError_t launch_select(const float* S, int32_t* idx, long long bh, int nb, int m,
                         hipStream_t stream) {
  return launch_rows<kSelectOnly>(S, nullptr, nullptr, idx, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, bh, nb, 64, m, stream);
}

hipError_t launch_coarse_term(const float* S, const int32_t* idx, const float* vp, float* cmax,
                              float* csum, float* cvec, long long bh, int nb, int d, int m,
                              hipStream_t stream) {
  return launch_rows<kTermOnly>(S, nullptr, nullptr, nullptr, idx, vp, cmax, csum, cvec, bh, nb,
                                d, m, stream);
}

hipError_t launch_select_fused(const float* qp, const float* kp, int32_t* idx, long long bh,
                               int nb, int d, int m, hipStream_t stream) {
  return launch_rows<kFusedSelect>(nullptr, qp, kp, idx, nullptr, nullptr, nullptr, nullptr,
                                   nullptr, bh, nb, d, m, stream);
}

hipError_t launch_select_term_fused(const float* qp, const float* kp, int32_t* idx,
                                    const float* vp, float* cmax, float* csum, float* cvec,
                                    long long bh, int nb, int d, int m, hipStream_t stream) {
  return launch_rows<kFused>(nullptr, qp, kp, idx, nullptr, vp, cmax, csum, cvec, bh, nb, d, m,
                             stream);
}

}  // namespace mra
