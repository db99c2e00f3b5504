// Three resolutions R = {s0, b, 1} (b = 32, s0 = r*b): Sec. 4.2 Alg. 1 with
// two refinement levels and Sec. 4.3 Alg. 2 over the resulting set J, with a
// budget per block-row at each level. The pieces specific to three levels:
//
//  * pool_up_kernel: the scale-s0 means Q~0, K~0, V~0 as means of r
//    consecutive scale-b means (eq. recursive_pooling applied further up);
//  * mask_kernel: after the s0-level selection T0_X (per s0-block-row X),
//    b-block-row x may only refine b-blocks inside its parent row's refined
//    s0-blocks: every other entry of its row of S~ is set to -inf, so the
//    per-row top-m selection of select.hip picks among the candidates only
//    (the budget m2 never exceeds their number m1*r);
//  * coarse_term_ml_kernel: the low-resolution part of block-row x, relative
//    to its largest coarse logit M: s0 e^{S~0[X,Y] - M} V~0_Y over the s0-blocks
//    X did not refine plus b e^{S~[x,y] - M} V~_y over the candidate b-blocks x
//    did not refine (each coarse block counts the columns it spans), in the
//    (M, c, L) form the tile pass merges.
//
// The coarse logits at both scales, the two selections and the tile pass are
// the kernels of the two-level path.
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

// One wave per b-block-row: S[x, y] = -inf unless y / r is in idx1[x / r].
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
// Per-wave LDS: refined bitmaps (s0 level, b level), the s0-level weights,
// the candidate list and its weights.
__global__ __launch_bounds__(kMlWaves * kWave) void coarse_term_ml_kernel(
    const float* __restrict__ S0, const int32_t* __restrict__ idx1, const float* __restrict__ S,
    const int32_t* __restrict__ idx2, const float* __restrict__ vp0,
    const float* __restrict__ vp, float* __restrict__ cmax, float* __restrict__ csum,
    float* __restrict__ cvec, int nb, int nb0, int r, int m1, int m2, long long rows, int d,
    int waves) {
  extern __shared__ __attribute__((aligned(16))) uint32_t ml_smem[];
  const int nw0 = (nb0 + 31) / 32, nw1 = (nb + 31) / 32, nc = m1 * r;
  const int per_wave = nw0 + nw1 + nb0 + 2 * nc;
  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id();
  const long long g = (long long)blockIdx.x * waves + w;
  if (g >= rows) return;
  uint32_t* bm0 = ml_smem + w * per_wave;
  uint32_t* bm1 = bm0 + nw0;
  float* w0 = reinterpret_cast<float*>(bm1 + nw1);
  int32_t* cy = reinterpret_cast<int32_t*>(w0 + nb0);
  float* w1 = reinterpret_cast<float*>(cy + nc);
  const long long bh = g / nb;
  const int x = (int)(g - bh * nb);
  const long long G0 = bh * nb0 + x / r;

  for (int i = lane; i < nw0 + nw1; i += kWave) bm0[i] = 0u;
  wave_lds_sync();
  for (int i = lane; i < m1; i += kWave) {
    const int Y = idx1[G0 * m1 + i];
    if (Y >= 0 && Y < nb0) atomicOr(&bm0[Y >> 5], 1u << (Y & 31));
  }
  for (int i = lane; i < m2; i += kWave) {
    const int y = idx2[g * m2 + i];
    if (y >= 0 && y < nb) atomicOr(&bm1[y >> 5], 1u << (y & 31));
  }
  wave_lds_sync();
  // candidate b-blocks in idx1 order (ascending Y, then t)
  for (int c = lane; c < nc; c += kWave) cy[c] = idx1[G0 * m1 + c / r] * r + c % r;
  wave_lds_sync();

  const float* s0row = S0 + G0 * nb0;
  const float* srow = S + g * nb;
  float M = -INFINITY;
  for (int Y = lane; Y < nb0; Y += kWave)
    if (!((bm0[Y >> 5] >> (Y & 31)) & 1u)) M = fmaxf(M, s0row[Y]);
  for (int c = lane; c < nc; c += kWave) {
    const int y = cy[c];
    if (!((bm1[y >> 5] >> (y & 31)) & 1u)) M = fmaxf(M, srow[y]);
  }
  M = wave_max(M);
  const bool any = M != -INFINITY;
  const float wide = (float)(r * kBlock);
  float sum = 0.0f;
  for (int Y = lane; Y < nb0; Y += kWave) {
    const bool use = any && !((bm0[Y >> 5] >> (Y & 31)) & 1u);
    const float wt = use ? wide * expf(s0row[Y] - M) : 0.0f;
    w0[Y] = wt;
    sum += wt;
  }
  for (int c = lane; c < nc; c += kWave) {
    const int y = cy[c];
    const bool use = any && !((bm1[y >> 5] >> (y & 31)) & 1u);
    const float wt = use ? (float)kBlock * expf(srow[y] - M) : 0.0f;
    w1[c] = wt;
    sum += wt;
  }
  sum = wave_sum(sum);
  wave_lds_sync();
  if (lane == 0) {
    cmax[g] = M;
    csum[g] = sum;
  }
  const float* v0 = vp0 + bh * (long long)nb0 * d;
  const float* v1 = vp + bh * (long long)nb * d;
  for (int dd = lane; dd < d; dd += kWave) {
    float acc = 0.0f;
    for (int Y = 0; Y < nb0; ++Y) acc = fmaf(w0[Y], v0[(long long)Y * d + dd], acc);
    for (int c = 0; c < nc; ++c) acc = fmaf(w1[c], v1[(long long)cy[c] * d + dd], acc);
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

static size_t coarse_term_ml_wave_bytes(int nb, int nb0, int r, int m1) {
  return ((size_t)(nb0 + 31) / 32 + (nb + 31) / 32 + nb0 + 2 * (size_t)m1 * r) * sizeof(uint32_t);
}

hipError_t launch_coarse_term_ml(const float* S0, const int32_t* idx1, const float* S,
                                 const int32_t* idx2, const float* vp0, const float* vp,
                                 float* cmax, float* csum, float* cvec, long long bh, int nb,
                                 int nb0, int r, int m1, int m2, int d, hipStream_t stream) {
  const long long rows = bh * nb;
  // four waves per workgroup while their lists fit 64 KB of LDS, else one
  // (at most 21 KB: nb <= 2048, nb0 <= 1024)
  const size_t per_wave = coarse_term_ml_wave_bytes(nb, nb0, r, m1);
  const int waves = per_wave * kMlWaves <= 65536 ? kMlWaves : 1;
  const unsigned blocks = (unsigned)((rows + waves - 1) / waves);
  coarse_term_ml_kernel<<<blocks, waves * kWave, per_wave * waves, stream>>>(
      S0, idx1, S, idx2, vp0, vp, cmax, csum, cvec, nb, nb0, r, m1, m2, rows, d, waves);
  return hipGetLastError();
}

}  // namespace mra
