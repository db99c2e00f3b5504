// Coarse logits S~ = Q~ K~^T / sqrt(d) of MRA-2 (Sec. 4.1, eq. exp_of_average:
// the exponential of the block mean of the fine logits factors into one dot
// product of pooled rows).
//
// Accumulated in float64 on the matrix cores and rounded once to float32, so
// the ranking that the selection takes from these scores agrees with an exact
// computation except for scores within a few float32 ulps of each other.
//
// One workgroup (4 waves) computes a 64 x 64 block of S~ for one head; wave w
// owns the four 16 x 16 tiles of rows 16w..16w+15 and loads its operands into
// registers straight from the pooled rows (the tile routine's layout).
#include "coarse_tile.h"
#include "kernels.h"

namespace mra {

constexpr int kCT = 64;    // output block edge

template <int D>
__global__ __launch_bounds__(256) void coarse_kernel(const float* __restrict__ qp,
                                                      const float* __restrict__ kp,
                                                      float* __restrict__ S, int nb, double scale) {
  // flattened grid: (head, block row, block column), column fastest
  const int nt = (nb + kCT - 1) / kCT;
  const long long bh = blockIdx.x / (nt * nt);
  const int tile = (int)(blockIdx.x - bh * nt * nt);
  const int x0 = (tile / nt) * kCT, y0 = (tile % nt) * kCT;
  const float* qh = qp + bh * nb * D;
  const float* kh = kp + bh * nb * D;
  const int w = wave_uniform(threadIdx.x / kWave), lane = lane_id(), r = lane & 15;

  f32x4 qv[D / 16];
  const int xr = x0 + 16 * w + r;
  coarse_load<D>(qh + (long long)min(xr, nb - 1) * D, qv);
  float* Sh = S + bh * nb * nb;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    f32x4 kv[D / 16];
    const int yr = y0 + 16 * c + r;
    coarse_load<D>(kh + (long long)min(yr, nb - 1) * D, kv);
    const f64x4 acc = coarse_tile_f64<D>(qv, kv);
    const int y = y0 + 16 * c + r;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int x = x0 + 16 * w + coarse_tile_row(lane, e);
      if (x < nb && y < nb) Sh[(long long)x * nb + y] = coarse_round(acc[e], scale);
    }
  }
}

hipError_t launch_coarse(const float* qp, const float* kp, float* S, long long bh, int nb, int d,
                         hipStream_t stream) {
  const double scale = 1.0 / sqrt((double)d);
  const long long nt = (nb + kCT - 1) / kCT;
  const dim3 grid((unsigned)(bh * nt * nt));
  if (d == 32) coarse_kernel<32><<<grid, 256, 0, stream>>>(qp, kp, S, nb, scale);
  else if (d == 64) coarse_kernel<64><<<grid, 256, 0, stream>>>(qp, kp, S, nb, scale);
  else coarse_kernel<128><<<grid, 256, 0, stream>>>(qp, kp, S, nb, scale);
  return hipGetLastError();
}

}  // namespace mra
