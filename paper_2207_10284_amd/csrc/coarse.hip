// Coarse logits S~ = Q~ K~^T / sqrt(d) of MRA-2 (Sec. 4.1, eq. exp_of_average:
// the exponential of the block mean of the fine logits factors into one dot
// product of pooled rows).
//
// Accumulated in float64 on the matrix cores and rounded once to float32, so
// the ranking that the selection takes from these scores agrees with an exact
// computation except for scores within a few float32 ulps of each other.
//
// One workgroup (4 waves) computes a 64 x 64 block of S~ for one head; the
// pooled rows are staged through LDS in 32-column slices (Q~ converted to
// float64 once), and wave w owns the four 16 x 16 tiles of rows 16w..16w+15.
#include "coarse_tile.h"
#include "kernels.h"

namespace mra {

constexpr int kCT = 64;    // output block edge
constexpr int kCK = 32;    // contraction slice

__global__ __launch_bounds__(256) void coarse_kernel(const float* __restrict__ qp,
                                                      const float* __restrict__ kp,
                                                      float* __restrict__ S, int nb, int d,
                                                      double scale) {
  __shared__ double qs[kCT][kCK + 1];
  __shared__ float ks[kCT][kCK + 1];
  // flattened grid: (head, block row, block column), column fastest
  const int nt = (nb + kCT - 1) / kCT;
  const long long bh = blockIdx.x / (nt * nt);
  const int tile = (int)(blockIdx.x - bh * nt * nt);
  const int x0 = (tile / nt) * kCT, y0 = (tile % nt) * kCT;
  const float* qh = qp + bh * nb * d;
  const float* kh = kp + bh * nb * d;
  const int t = threadIdx.x, w = wave_uniform(t / kWave), lane = lane_id();

  f64x4 acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = f64x4{0.0, 0.0, 0.0, 0.0};

  for (int k0 = 0; k0 < d; k0 += kCK) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {              // 64 x 32 per operand, 8 per thread
      const int li = t + 256 * e, r = li / kCK, c = li % kCK;
      qs[r][c] = (x0 + r < nb) ? (double)qh[(long long)(x0 + r) * d + k0 + c] : 0.0;
      ks[r][c] = (y0 + r < nb) ? kh[(long long)(y0 + r) * d + k0 + c] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 4; ++c)
      coarse_tile_f64(acc[c], &qs[16 * w][0], kCK + 1, &ks[16 * c][0], kCK + 1, kCK);
    __syncthreads();
  }
  float* Sh = S + bh * nb * nb;
  const int col = lane & 15;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int y = y0 + 16 * c + col;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int x = x0 + 16 * w + coarse_tile_row(lane, e);
      if (x < nb && y < nb) Sh[(long long)x * nb + y] = coarse_round(acc[c][e], scale);
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
