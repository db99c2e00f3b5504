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
// One workgroup (4 waves) owns RB consecutive block-rows of one head. Their
// score rows sit in LDS: loaded from S~, or (fused mode) computed there from
// the pooled rows in float64 exactly as the coarse-logit kernel does. Each
// wave then selects for its rows: a radix search for the m-th largest
// order-preserving 32-bit key (32 rounds of ballot + popcount), then one
// ascending sweep that resolves ties at the threshold by index and compacts
// the kept indices with prefix popcounts; the row's keys stay in registers
// throughout. The score row is overwritten by the weights b e^{S~ - M} (0
// where selected), and L = W V~ is formed for the RB rows at once on the
// float32 matrix cores (16x16x4), so V~ is read once per workgroup rather than
// once per row. Workgroups of one head are kept on one XCD.
// Every mode runs the same arithmetic in the same order, so the fused forward
// step is bit-identical to separate score, select and coarse-term calls.
#include "common.h"
#include "kernels.h"

namespace mra {

enum RowsMode { kSelectOnly = 0, kTermOnly = 1, kFused = 2 };
constexpr int kRowsThreads = 256;

// Block-rows per workgroup: 16, fewer for long rows (LDS holds RB x nb scores).
static int rows_per_group(int nb) {
  int rb = 16;
  while (rb > 4 && rb * nb > 8192) rb >>= 1;
  return rb;
}

typedef float f32x4v __attribute__((ext_vector_type(4)));

template <int D, int MODE, int JMAX>
__global__ __launch_bounds__(kRowsThreads) void rows_kernel(
    const float* __restrict__ S, const float* __restrict__ qp, const float* __restrict__ kp,
    int32_t* __restrict__ idx_out, const int32_t* __restrict__ idx_in,
    const float* __restrict__ vp, float* __restrict__ cmax, float* __restrict__ csum,
    float* __restrict__ cvec, int nb, int m, int rb, double scale) {
  extern __shared__ float smem[];
  const int nwords = (nb + 31) / 32;
  const int ldr = nb + 1;                                          // odd row stride: no bank conflicts
  float* srow = smem;                                              // [rb][ldr]
  uint32_t* selbits = reinterpret_cast<uint32_t*>(smem + rb * ldr); // [rb][nwords]
  const int tid = threadIdx.x;
  const int w = wave_uniform(tid / kWave);
  const int lane = lane_id();
  const int groups = (nb + rb - 1) / rb;
  const long long lwg = xcd_remap(blockIdx.x, gridDim.x);
  const long long bh = lwg / groups;
  const int x0 = (int)(lwg - bh * groups) * rb;
  const int rows = min(rb, nb - x0);
  const long long g0 = bh * nb + x0;                               // first global block-row

  // ---- phase 1: the RB score rows into LDS
  if constexpr (MODE == kFused) {
    // S~ = c Q~ K~^T in float64: 64 columns x rb rows per pass, contraction in
    // slices of 32; same fma order as the coarse-logit kernel.
    float* qs = reinterpret_cast<float*>(selbits + rb * nwords);  // [16][33]
    float* ks = qs + 16 * 33;                                       // [64][33]
    const float* qh = qp + g0 * D;
    const float* kh = kp + bh * nb * D;
    const int yl = tid & 63, rg = tid >> 6;
    for (int y0 = 0; y0 < nb; y0 += 64) {
      double acc[4] = {0.0, 0.0, 0.0, 0.0};
      for (int k0 = 0; k0 < D; k0 += 32) {
        for (int li = tid; li < 16 * 32; li += kRowsThreads) {
          const int r = li >> 5, cc = li & 31;
          qs[r * 33 + cc] = r < rows ? qh[(long long)r * D + k0 + cc] : 0.0f;
        }
        for (int li = tid; li < 64 * 32; li += kRowsThreads) {
          const int r = li >> 5, cc = li & 31;
          ks[r * 33 + cc] = (y0 + r < nb) ? kh[(long long)(y0 + r) * D + k0 + cc] : 0.0f;
        }
        __syncthreads();
#pragma unroll 4
        for (int cc = 0; cc < 32; ++cc) {
          const double b = (double)ks[yl * 33 + cc];
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (rg + 4 * i < rb) acc[i] = fma((double)qs[(rg + 4 * i) * 33 + cc], b, acc[i]);
        }
        __syncthreads();
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = rg + 4 * i;
        if (r < rows && y0 + yl < nb) srow[r * ldr + y0 + yl] = (float)(acc[i] * scale);
      }
    }
  } else {
    const float* Sg = S + g0 * nb;
    for (int i = tid; i < rows * nb; i += kRowsThreads) srow[(i / nb) * ldr + i % nb] = Sg[i];
  }
  for (int i = tid; i < rb * nwords; i += kRowsThreads) selbits[i] = 0u;
  __syncthreads();

  // ---- phase 2: selection (one wave per row)
  const int J = (nb + kWave - 1) / kWave;
  for (int r = w; r < rows; r += 4) {
    float* sr = srow + r * ldr;
    uint32_t* sb = selbits + r * nwords;
    const long long g = g0 + r;
    if constexpr (MODE == kTermOnly) {
      for (int i = lane; i < m; i += kWave) {
        const int y = idx_in[g * m + i];
        if (y >= 0 && y < nb) atomicOr(&sb[y >> 5], 1u << (y & 31));
      }
    } else {
      uint32_t key[JMAX];                    // this lane's keys, y = j*64 + lane
#pragma unroll
      for (int j = 0; j < JMAX; ++j) {
        const int y = j * kWave + lane;
        key[j] = (j < J && y < nb) ? ordered_key(sr[y]) : 0u;
      }
      uint32_t T = 0;
      int need = 0;
      const bool all = (m == nb), none = (m == 0);
      if (!all && !none) {
        for (int bit = 31; bit >= 0; --bit) {
          const uint32_t cand = T | (1u << bit);
          int cnt = 0;
#pragma unroll
          for (int j = 0; j < JMAX; ++j)
            if (j < J) cnt += __popcll(__ballot(key[j] >= cand));
          if (cnt >= m) T = cand;
        }
        int gt = 0;
#pragma unroll
        for (int j = 0; j < JMAX; ++j)
          if (j < J) gt += __popcll(__ballot(key[j] > T));
        need = m - gt;                       // >= 1 keys equal to T still to take
      }
      int eq_seen = 0, written = 0;
#pragma unroll
      for (int j = 0; j < JMAX; ++j) {
        if (j >= J) break;
        const int y = j * kWave + lane;
        const bool valid = y < nb;
        bool sel;
        if (all) {
          sel = valid;
        } else if (none) {
          sel = false;
        } else {
          const bool eq = valid && key[j] == T;
          const uint64_t eqm = __ballot(eq);
          const int rank = eq_seen + __popcll(eqm & lanemask_lt());
          eq_seen += __popcll(eqm);
          sel = valid && (key[j] > T || (eq && rank < need));
        }
        const uint64_t smk = __ballot(sel);
        if (sel && idx_out) idx_out[g * m + written + __popcll(smk & lanemask_lt())] = y;
        written += __popcll(smk);
        if (lane == 0) {
          if (j * 2 < nwords) sb[j * 2] = (uint32_t)smk;
          if (j * 2 + 1 < nwords) sb[j * 2 + 1] = (uint32_t)(smk >> 32);
        }
      }
    }
    if constexpr (MODE == kSelectOnly) continue;
    wave_lds_sync();
    // ---- phase 3: max and weights of the unselected blocks
    float M = -INFINITY;
    for (int j = 0; j < J; ++j) {
      const int y = j * kWave + lane;
      if (y < nb && !((sb[y >> 5] >> (y & 31)) & 1u)) M = fmaxf(M, sr[y]);
    }
    M = wave_max(M);
    const bool any = M != -INFINITY;
    float c = 0.0f;
    for (int j = 0; j < J; ++j) {
      const int y = j * kWave + lane;
      if (y < nb) {
        const bool unsel = !((sb[y >> 5] >> (y & 31)) & 1u);
        const float wgt = (any && unsel) ? (float)kBlock * expf(sr[y] - M) : 0.0f;
        sr[y] = wgt;                           // each lane rewrites only its own entries
        c += wgt;
      }
    }
    c = wave_sum(c);
    if (lane == 0) {
      cmax[g] = M;
      csum[g] = c;
    }
  }
  if constexpr (MODE == kSelectOnly) return;
  __syncthreads();

  // ---- phase 4: L = W V~ for the rows of this group on the float32 matrix
  // cores: v_mfma_f32_16x16x4_f32 with A = W (16 rows x 4 blocks, rows past
  // `rows` are zero), B = V~ (4 blocks x 16 dims); wave w owns the dim tiles
  // w, w+4, ...; blocks in ascending order, four per instruction.
  {
    constexpr int kNT16 = D / 16;
    const int ar = lane & 15, ak = lane >> 4;          // A: row, k;  B: dim, k
    const float* vh = vp + bh * (long long)nb * D;
    for (int nt = w; nt < kNT16; nt += 4) {
      f32x4v acc = {0.0f, 0.0f, 0.0f, 0.0f};
      const int dim = 16 * nt + ar;
#pragma unroll 4
      for (int y0 = 0; y0 < nb; y0 += 4) {
        const int y = y0 + ak;
        const float a = (ar < rows && y < nb) ? srow[ar * ldr + y] : 0.0f;
        const float b = y < nb ? vh[(long long)y * D + dim] : 0.0f;
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
      }
      // D layout: lane holds rows 4*(lane/16) + e of column lane%16
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * ak + e;
        if (r < rows) cvec[(g0 + r) * D + dim] = acc[e];
      }
    }
  }
}

static size_t rows_smem(int nb, int rb, bool fused) {
  size_t s = (size_t)rb * (nb + 1) * sizeof(float) + (size_t)rb * ((nb + 31) / 32) * sizeof(uint32_t);
  if (fused) s += (16 * 33 + 64 * 33) * sizeof(float);
  return s;
}

template <int MODE, int JMAX>
static void launch_rows_j(const float* S, const float* qp, const float* kp, int32_t* idx_out,
                          const int32_t* idx_in, const float* vp, float* cmax, float* csum,
                          float* cvec, long long bh, int nb, int d, int m, hipStream_t stream) {
  const int rb = rows_per_group(nb);
  const long long groups = (nb + rb - 1) / rb;
  const unsigned blocks = (unsigned)(bh * groups);
  const size_t smem = rows_smem(nb, rb, MODE == kFused);
  const double scale = 1.0 / sqrt((double)d);
#define MRA_ROWS_LAUNCH(DD) \
  rows_kernel<DD, MODE, JMAX><<<blocks, kRowsThreads, smem, stream>>>(S, qp, kp, idx_out, idx_in, vp, cmax, csum, cvec, nb, m, rb, scale)
  switch (d) {
    case 32: MRA_ROWS_LAUNCH(32); break;
    case 64: MRA_ROWS_LAUNCH(64); break;
    default: MRA_ROWS_LAUNCH(128); break;
  }
#undef MRA_ROWS_LAUNCH
}

// Keys per lane: up to 2 (nb <= 128), 8 (nb <= 512) or 32 (nb <= 2048).
template <int MODE>
static hipError_t launch_rows(const float* S, const float* qp, const float* kp, int32_t* idx_out,
                              const int32_t* idx_in, const float* vp, float* cmax, float* csum,
                              float* cvec, long long bh, int nb, int d, int m, hipStream_t stream) {
  if (nb <= 128)
    launch_rows_j<MODE, 2>(S, qp, kp, idx_out, idx_in, vp, cmax, csum, cvec, bh, nb, d, m, stream);
  else if (nb <= 512)
    launch_rows_j<MODE, 8>(S, qp, kp, idx_out, idx_in, vp, cmax, csum, cvec, bh, nb, d, m, stream);
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

hipError_t launch_select_term_fused(const float* qp, const float* kp, int32_t* idx,
                                    const float* vp, float* cmax, float* csum, float* cvec,
                                    long long bh, int nb, int d, int m, hipStream_t stream) {
  return launch_rows<kFused>(nullptr, qp, kp, idx, nullptr, vp, cmax, csum, cvec, bh, nb, d, m,
                             stream);
}

}  // namespace mra
