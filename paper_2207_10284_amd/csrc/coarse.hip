// Coarse logits S~ = Q~ K~^T / sqrt(d) of MRA-2 (Sec. 4.1, eq. exp_of_average:
// the exponential of the block mean of the fine logits factors into one dot
// product of pooled rows).
//
// Accumulated in float64 and rounded once to float32, so the ranking that the
// selection takes from these scores agrees with an exact computation except
// for scores within a few float32 ulps of each other.
//
// One workgroup computes a 64 x 64 tile of S~ for one head; the pooled rows are
// staged through LDS in 32-column slices (padded rows: the 16 column-rows a
// wave reads at once fall into distinct banks); every thread accumulates a
// 4 x 4 register tile.
#include "common.h"
#include "kernels.h"

namespace mra {

constexpr int kCT = 64;    // output tile edge
constexpr int kCK = 32;    // contraction slice

__global__ __launch_bounds__(256) void coarse_kernel(const float* __restrict__ qp,
                                                      const float* __restrict__ kp,
                                                      float* __restrict__ S, int nb, int d,
                                                      double scale) {
  __shared__ float qs[kCT][kCK + 1];
  __shared__ float ks[kCT][kCK + 1];
  // flattened grid: (head, tile row, tile column), column fastest
  const int nt = (nb + kCT - 1) / kCT;
  const long long bh = blockIdx.x / (nt * nt);
  const int tile = (int)(blockIdx.x - bh * nt * nt);
  const int x0 = (tile / nt) * kCT, y0 = (tile % nt) * kCT;
  const float* qh = qp + bh * nb * d;
  const float* kh = kp + bh * nb * d;
  const int t = threadIdx.x, ty = t / 16, tx = t % 16;

  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;

  for (int k0 = 0; k0 < d; k0 += kCK) {
    // 64 rows x 32 columns per operand = 2048 floats: 8 per thread.
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int li = t + 256 * e, r = li / kCK, c = li % kCK;
      qs[r][c] = (x0 + r < nb) ? qh[(long long)(x0 + r) * d + k0 + c] : 0.0f;
      ks[r][c] = (y0 + r < nb) ? kh[(long long)(y0 + r) * d + k0 + c] : 0.0f;
    }
    __syncthreads();
#pragma unroll 4
    for (int c = 0; c < kCK; ++c) {
      double a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = (double)qs[ty + 16 * i][c];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = (double)ks[tx + 16 * j][c];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fma(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  float* Sh = S + bh * nb * nb;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int x = x0 + ty + 16 * i;
    if (x >= nb) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int y = y0 + tx + 16 * j;
      if (y < nb) Sh[(long long)x * nb + y] = (float)(acc[i][j] * scale);
    }
  }
}

hipError_t launch_coarse(const float* qp, const float* kp, float* S, long long bh, int nb, int d,
                         hipStream_t stream) {
  const double scale = 1.0 / sqrt((double)d);
  const long long nt = (nb + kCT - 1) / kCT;
  coarse_kernel<<<dim3((unsigned)(bh * nt * nt)), 256, 0, stream>>>(qp, kp, S, nb, d, scale);
  return hipGetLastError();
}

}  // namespace mra
