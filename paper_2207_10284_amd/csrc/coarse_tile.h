// One 16 x 16 tile of the coarse logits on the float64 matrix cores, shared by
// the coarse-logit kernel and the fused selection kernel so that both produce
// the same bits (same operands, same instruction sequence, k ascending).
#pragma once

#include "common.h"

namespace mra {

typedef double f64x4 __attribute__((ext_vector_type(4)));

// acc += sum_{k < klen} qd[i][k] * kf[j][k] for the tile rows i (queries) and
// columns j (keys), k in steps of four, one v_mfma_f64_16x16x4_f64 per step.
// qd: float64 rows in LDS (row stride ldq); kf: float32 rows in LDS (row
// stride ldk), converted exactly to float64. Lane l supplies A[l%16][l/16]
// and B[l/16][l%16]; result register e of lane l is row coarse_tile_row(l, e)
// of column l%16 (the float64 16x16x4 instruction interleaves rows across the
// four lane groups, unlike its float32 counterpart).
__device__ __forceinline__ void coarse_tile_f64(f64x4& acc, const double* qd, int ldq,
                                                const float* kf, int ldk, int klen) {
  const int lane = lane_id(), r = lane & 15, kq = lane >> 4;
  const double* qa = qd + r * ldq + kq;
  const float* kb = kf + r * ldk + kq;
#pragma unroll 4
  for (int k0 = 0; k0 < klen; k0 += 4)
    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[k0], (double)kb[k0], acc, 0, 0, 0);
}

__device__ __forceinline__ int coarse_tile_row(int lane, int e) { return 4 * e + (lane >> 4); }

// Final rounding of a coarse logit: scale by 1/sqrt(d) in float64, round once.
__device__ __forceinline__ float coarse_round(double acc, double scale) {
  return (float)(acc * scale);
}

}  // namespace mra
