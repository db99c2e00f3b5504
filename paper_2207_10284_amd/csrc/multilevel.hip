// Any number of resolutions R = {s_0 > s_1 > ... > s_{L-1} = b, 1} (b = 32,
// each scale a multiple of the next): Sec. 4.2 Alg. 1 refined level by level
// and Sec. 4.3 Alg. 2 over the resulting set J, with a budget per block-row at
// each level. The pieces beyond the two-level path:
//
//  * pool_up_kernel: the scale-s_l means Q~_l, K~_l, V~_l as means of
//    s_l / b consecutive scale-b means (eq. recursive_pooling applied further
//    up);
//  * mask_kernel: after level l - 1's selection (per s_{l-1}-block-row), an
//    s_l-block-row may only keep s_l-blocks inside its parent row's kept
//    blocks: every other entry of its row of S~_l is set to -inf, so the
//    per-row top-m selection of select.hip picks among the candidates only
//    (the budget m_l never exceeds their number m_{l-1} s_{l-1} / s_l);
//  * coarse_term_levels_kernel: the low-resolution part of b-block-row x,
//    relative to its largest coarse logit M: s_l e^{S~_l[X_l,Y] - M} V~_l,Y
//    over, at every level l, the candidate blocks Y (all s_0-blocks at level
//    0, the children of the ancestor's kept blocks below) that its ancestor
//    X_l did not keep (each coarse block counts the columns it spans), in the
//    (M, c, L) form the tile pass merges.
//
// The coarse logits at every scale, the selections and the tile pass are the
// kernels of the two-level path.
#include "common.h"
#include "kernels.h"

namespace mra {

// dst[row, :] = mean of src rows r*row .. r*row + r - 1 (float32, in order);
// blockIdx.y picks one of three tensors (a NULL pair is skipped).
__global__ __launch_bounds__(256) void pool_up_kernel(const float* __restrict__ s0,
                                                       const float* __restrict__ s1,
                                                       const float* __restrict__ s2,
                                                       float* __restrict__ d0, float* __restrict__ d1,
                                                       float* __restrict__ d2, long long rows_out,
                                                       int d, int r) {
  const int which = blockIdx.y;
  const float* src = which == 0 ? s0 : (which == 1 ? s1 : s2);
  float* dst = which == 0 ? d0 : (which == 1 ? d1 : d2);
  if (src == nullptr) return;
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows_out * d) return;
  const long long row = t / d;
  const int c = (int)(t - row * d);
  float acc = 0.0f;
  for (int i = 0; i < r; ++i) acc += src[(row * r + i) * d + c];
  dst[t] = acc / (float)r;
}

// One wave per block-row x of a level: S[x, y] = -inf unless y / r is in
// idx1[x / r], the parent level's kept blocks (nb0 <= 1024 parent blocks).
__global__ __launch_bounds__(64) void mask_kernel(float* __restrict__ S,
                                                  const int32_t* __restrict__ idx1, int nb,
                                                  int nb0, int r, int m1) {
  __shared__ uint32_t bm[32];                               // nb0 <= 1024
  const long long g = blockIdx.x;                           // global b-block-row
  const long long bh = g / nb;
  const int x = (int)(g - bh * nb);
  const long long G0 = bh * nb0 + x / r;
  const int lane = lane_id();
  if (lane < 32) bm[lane] = 0u;
  wave_lds_sync();
  for (int i = lane; i < m1; i += kWave) {
    const int Y = idx1[G0 * m1 + i];
    if (Y >= 0 && Y < nb0) atomicOr(&bm[Y >> 5], 1u << (Y & 31));
  }
  wave_lds_sync();
  float* row = S + g * nb;
  for (int y = lane; y < nb; y += kWave) {
    const int Y = y / r;
    if (!((bm[Y >> 5] >> (Y & 31)) & 1u)) row[y] = -INFINITY;
  }
}

constexpr int kMlWaves = 4;

// One wave per b-block-row (`waves` per workgroup, no workgroup barriers).
// Per-wave LDS: the kept-block bitmaps of the row's ancestors at every level,
// then every level's candidate list (level 0: all its blocks; level l: the
// children of the level l - 1 ancestor's kept blocks, in that list's order),
// compacted to the unkept candidates with their weights.
template <int L>
__global__ __launch_bounds__(kMlWaves * kWave) void coarse_term_levels_kernel(
    LevelTerm T, float* __restrict__ cmax, float* __restrict__ csum, float* __restrict__ cvec,
    long long rows, int d, int waves) {
  extern __shared__ __attribute__((aligned(16))) uint32_t ml_smem[];
  const int nbf = T.nb[L - 1];
  int words = 0, ents = 0;
  int woff[kMaxLevels], eoff[kMaxLevels + 1];
#pragma unroll
  for (int l = 0; l < L; ++l) {
    woff[l] = words;
    words += (T.nb[l] + 31) / 32;
    eoff[l] = ents;
    ents += l == 0 ? T.nb[0] : T.m[l - 1] * (T.r[l - 1] / T.r[l]);
  }
  eoff[L] = ents;
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id();
  const long long g = (long long)blockIdx.x * waves + w;
  if (g >= rows) return;
  uint32_t* bm = ml_smem + (size_t)w * (words + 2 * ents);
  int32_t* cy = reinterpret_cast<int32_t*>(bm + words);
  float* wt = reinterpret_cast<float*>(cy + ents);
  const long long bh = g / nbf;
  const int x = (int)(g - bh * nbf);

  // the row's ancestor at every level; every level's candidate count
  long long G[L];
  int ncand[L], mmax = 0, cmaxn = 0;
#pragma unroll
  for (int l = 0; l < L; ++l) {
    G[l] = bh * T.nb[l] + x / T.r[l];
    ncand[l] = eoff[l + 1] - eoff[l];
    mmax = max(mmax, T.m[l]);
    cmaxn = max(cmaxn, ncand[l]);
  }
  // Global loads are issued for all levels before their results are used, so
  // their latencies overlap.
  for (int i = lane; i < words; i += kWave) bm[i] = 0u;
  wave_lds_sync();
  for (int i0 = 0; i0 < mmax; i0 += kWave) {
    int Yv[L];
#pragma unroll
    for (int l = 0; l < L; ++l) Yv[l] = i0 + lane < T.m[l] ? T.idx[l][G[l] * T.m[l] + i0 + lane] : -1;
#pragma unroll
    for (int l = 0; l < L; ++l)
      if (Yv[l] >= 0 && Yv[l] < T.nb[l]) atomicOr(&bm[woff[l] + (Yv[l] >> 5)], 1u << (Yv[l] & 31));
  }
  wave_lds_sync();

  auto unkept = [&](int l, int y) {
    return y >= 0 && !((bm[woff[l] + (y >> 5)] >> (y & 31)) & 1u);
  };
  // candidates (level 0: all blocks; level l: the children of the parent's
  // kept blocks, -1 for an invalid parent entry) and the unkept ones' logits,
  // held in wt until the weights replace them
  float M = -INFINITY;
  for (int c0 = 0; c0 < cmaxn; c0 += kWave) {
    const int c = c0 + lane;
    int yv[L];
    float sv[L];
#pragma unroll
    for (int l = 0; l < L; ++l) {
      if (l == 0) {
        yv[l] = c < ncand[0] ? c : -1;
      } else {
        const int p = T.r[l - 1] / T.r[l];
        const int Y = c < ncand[l] ? T.idx[l - 1][G[l - 1] * T.m[l - 1] + c / p] : -1;
        yv[l] = Y >= 0 && Y < T.nb[l - 1] ? Y * p + c % p : -1;
      }
    }
#pragma unroll
    for (int l = 0; l < L; ++l) {
      const float s = T.S[l][G[l] * T.nb[l] + (yv[l] < 0 ? 0 : yv[l])];
      sv[l] = unkept(l, yv[l]) ? s : -INFINITY;
    }
#pragma unroll
    for (int l = 0; l < L; ++l)
      if (c < ncand[l]) {
        cy[eoff[l] + c] = yv[l];
        wt[eoff[l] + c] = sv[l];
        M = fmaxf(M, sv[l]);
      }
  }
  wave_lds_sync();
  M = wave_max(M);
  const bool any = M != -INFINITY;
  // weights; the list keeps only the entries that carry one, in order
  // (kept blocks would add zero: dropping them changes no bit)
  float sum = 0.0f;
  int kept_to[kMaxLevels + 1];
  int cnt = 0;
#pragma unroll
  for (int l = 0; l < L; ++l) {
    kept_to[l] = cnt;
    const float wide = (float)(T.r[l] * kBlock);
    for (int c0 = eoff[l]; c0 < eoff[l + 1]; c0 += kWave) {
      const int c = c0 + lane;
      const int y = c < eoff[l + 1] ? cy[c] : -1;
      const float sv = c < eoff[l + 1] ? wt[c] : -INFINITY;
      const bool use = any && unkept(l, y);
      const float v = use ? wide * expf(sv - M) : 0.0f;
      sum += v;
      const uint64_t mk = __ballot(use);
      if (use) {
        const int pos = cnt + __popcll(mk & lanemask_lt());
        cy[pos] = y;                                        // pos <= c: that entry was read above
        wt[pos] = v;
      }
      cnt += __popcll(mk);
    }
  }
  kept_to[L] = cnt;
  sum = wave_sum(sum);
  wave_lds_sync();
  if (lane == 0) {
    cmax[g] = M;
    csum[g] = sum;
  }
  // weight x pooled V row, entries in list order; the rows' loads are issued
  // kBatch at a time so that their latencies overlap
  constexpr int kBatch = 32;
  for (int dd = lane; dd < d; dd += kWave) {
    float acc = 0.0f;
#pragma unroll
    for (int l = 0; l < L; ++l) {
      // the level's pooled V rows of the head as a buffer (a row's offset in
      // the vector offset; every listed y is in [0, nb_l))
      const i32x4 vrs = buffer_rsrc(T.vp[l] + bh * (long long)T.nb[l] * d, (unsigned)T.nb[l] * d * 4u);
      for (int c0 = kept_to[l]; c0 < kept_to[l + 1]; c0 += kBatch) {
        const int nc = min(kBatch, kept_to[l + 1] - c0);  // wave-uniform
        float vv[kBatch], ww[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
          const int y = j < nc ? cy[c0 + j] : 0;
          ww[j] = j < nc ? wt[c0 + j] : 0.0f;
          vv[j] = mra_raw_buffer_load_f32(vrs, (y * d + dd) * 4, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
          if (j < nc) acc = fmaf(ww[j], vv[j], acc);
      }
    }
    cvec[g * d + dd] = acc;
  }
}

hipError_t launch_pool_up(const float* qp, const float* kp, const float* vp, float* qp0,
                          float* kp0, float* vp0, long long rows_out, int d, int r,
                          hipStream_t stream) {
  const long long n = rows_out * d;
  const dim3 grid((unsigned)((n + 255) / 256), 3);
  pool_up_kernel<<<grid, 256, 0, stream>>>(qp, kp, vp, qp0, kp0, vp0, rows_out, d, r);
  return hipGetLastError();
}

hipError_t launch_mask_candidates(float* S, const int32_t* idx1, long long bh, int nb, int nb0,
                                  int r, int m1, hipStream_t stream) {
  mask_kernel<<<(unsigned)(bh * nb), kWave, 0, stream>>>(S, idx1, nb, nb0, r, m1);
  return hipGetLastError();
}

static size_t coarse_term_levels_wave_bytes(const LevelTerm& T) {
  size_t words = 0, ents = 0;
  for (int l = 0; l < T.levels; ++l) {
    words += (T.nb[l] + 31) / 32;
    ents += l == 0 ? T.nb[0] : (size_t)T.m[l - 1] * (T.r[l - 1] / T.r[l]);
  }
  return (words + 2 * ents) * sizeof(uint32_t);
}

hipError_t launch_coarse_term_levels(const LevelTerm& T, float* cmax, float* csum, float* cvec,
                                     long long bh, int d, hipStream_t stream) {
  const long long rows = bh * T.nb[T.levels - 1];
  // four waves per workgroup while their lists fit 64 KB of LDS, else one
  // (under 34 KB: every level's candidates number at most its blocks, and the
  // block counts of the levels sum to less than 2 nb <= 4096)
  const size_t per_wave = coarse_term_levels_wave_bytes(T);
  const int waves = per_wave * kMlWaves <= 65536 ? kMlWaves : 1;
  const unsigned blocks = (unsigned)((rows + waves - 1) / waves);
  const size_t smem = per_wave * waves;
  switch (T.levels) {
#define MRA_LEVELS_CASE(NL)                                                                          \
  case NL:                                                                                           \
    coarse_term_levels_kernel<NL><<<blocks, waves * kWave, smem, stream>>>(T, cmax, csum, cvec, rows, \
                                                                           d, waves);               \
    break;
    MRA_LEVELS_CASE(1)
    MRA_LEVELS_CASE(2)
    MRA_LEVELS_CASE(3)
    MRA_LEVELS_CASE(4)
    MRA_LEVELS_CASE(5)
    MRA_LEVELS_CASE(6)
    MRA_LEVELS_CASE(7)
    MRA_LEVELS_CASE(8)
#undef MRA_LEVELS_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mra
