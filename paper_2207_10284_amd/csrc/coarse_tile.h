// One 16 x 16 tile of the coarse logits on the float64 matrix cores, shared by
// the coarse-logit kernel and the fused selection kernel so that both produce
// the same bits (same operands, same instruction sequence).
#pragma once

#include "common.h"

namespace mra {

typedef double f64x4 __attribute__((ext_vector_type(4)));

// Operands of a tile in registers. Lane l = 16g + r holds row r of the tile
// (a query row of Q~ or a key row of K~) at columns 16s + 4g .. 16s + 4g + 3
// for s < d/16, one float4 per s, loaded straight from the row-major pooled
// rows (the 16 lanes of a group read 16 rows, the four groups 64 contiguous
// bytes of each). Callers clamp rows past the end to a valid row and ignore
// the results in those rows and columns.
template <int D>
__device__ __forceinline__ void coarse_load(const float* __restrict__ row, f32x4 (&v)[D / 16]) {
  const int g = lane_id() >> 4;
#pragma unroll
  for (int s = 0; s < D / 16; ++s) v[s] = *reinterpret_cast<const f32x4*>(row + 16 * s + 4 * g);
}

// acc = sum over the d columns of q[i][k] * kf[j][k] (tile rows i = queries,
// columns j = keys), one v_mfma_f64_16x16x4_f64 per step. Step 4s + e takes
// column 16s + 4g + e in lane group g (the instruction's contraction index is
// the lane group), so the d columns are each used once, in this fixed order;
// the float32 values convert exactly to float64. Two chains (s even, s odd)
// keep two products in flight; their sums are added at the end. Result
// register e of lane l is row coarse_tile_row(l, e) of column l%16 (the
// float64 16x16x4 instruction interleaves rows across the four lane groups,
// unlike its float32 counterpart).
template <int D>
__device__ __forceinline__ f64x4 coarse_tile_f64(const f32x4 (&q)[D / 16], const f32x4 (&kf)[D / 16]) {
  f64x4 acc[2] = {{0.0, 0.0, 0.0, 0.0}, {0.0, 0.0, 0.0, 0.0}};
#pragma unroll
  for (int s = 0; s < D / 16; ++s)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      acc[s & 1] = __builtin_amdgcn_mfma_f64_16x16x4f64((double)q[s][e], (double)kf[s][e], acc[s & 1], 0, 0, 0);
  return acc[0] + acc[1];
}

// The same products and order with the query operands already in float64:
// qrow points at this lane's row of a float64 copy of the tile's query rows
// (16-byte aligned) whose column c is stored at c ^ x (x even and below 32),
// c0 = 4g is the lane's first column, so the results are the same bits.
typedef double f64x2 __attribute__((ext_vector_type(2)));
template <int D>
__device__ __forceinline__ f64x4 coarse_tile_f64_qd(const double* qrow, int c0, int x,
                                                   const f32x4 (&kf)[D / 16]) {
  f64x4 acc[2] = {{0.0, 0.0, 0.0, 0.0}, {0.0, 0.0, 0.0, 0.0}};
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    const int c = (c0 + 16 * s) ^ x;
    const f64x2 q01 = *reinterpret_cast<const f64x2*>(qrow + c);
    const f64x2 q23 = *reinterpret_cast<const f64x2*>(qrow + (c ^ 2));
    acc[s & 1] = __builtin_amdgcn_mfma_f64_16x16x4f64(q01[0], (double)kf[s][0], acc[s & 1], 0, 0, 0);
    acc[s & 1] = __builtin_amdgcn_mfma_f64_16x16x4f64(q01[1], (double)kf[s][1], acc[s & 1], 0, 0, 0);
    acc[s & 1] = __builtin_amdgcn_mfma_f64_16x16x4f64(q23[0], (double)kf[s][2], acc[s & 1], 0, 0, 0);
    acc[s & 1] = __builtin_amdgcn_mfma_f64_16x16x4f64(q23[1], (double)kf[s][3], acc[s & 1], 0, 0, 0);
  }
  return acc[0] + acc[1];
}

__device__ __forceinline__ int coarse_tile_row(int lane, int e) { return 4 * e + (lane >> 4); }

// Final rounding of a coarse logit: scale by 1/sqrt(d) in float64, round once.
__device__ __forceinline__ float coarse_round(double acc, double scale) {
  return (float)(acc * scale);
}

}  // namespace mra
