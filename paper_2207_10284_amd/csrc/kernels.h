// Launchers of the MRA-2 kernels (internal; the public interface is mra.h).
// Every launcher only enqueues on `stream` and returns hipGetLastError().
// Arguments are assumed validated by the caller (api.cpp).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mra {

// Packed K/V (written by the pooling pass, read by the tile pass): for every
// head and 32-key block y, the tile's matrix-core operands in lane order, 16
// bytes per lane and instruction, 32*d elements per block. The K part (all
// blocks) comes first, then the V part.
//  K, chunk s*64 + 32h + j: K[j][(d/2)h + e*s .. +e-1], e = 8 (bf16) or 4 (f32)
//  V bf16, chunk (u*NT + t)*64 + 32h + j, NT = d/32: the 8 values
//        V[16u + 8(s/4) + 4h + s%4][32t + j], s = 0..7 (u = 0, 1)
//  V f32, chunk (t*4 + a)*64 + 32h + j: V[8a + 4h + kk][32t + j], kk = 0..3
// Block-means of q/k/v ([bh, n, d], dtype) into qp/kp/vp ([bh, n/32, d] f32);
// a NULL output skips that tensor. If kvpacked is not NULL (k, v, kp, vp
// given), the packed copies of k and v are written too.
hipError_t launch_pool(const void* q, const void* k, const void* v, float* qp, float* kp,
                       float* vp, void* kvpacked, long long bh, int n, int d, int dtype,
                       hipStream_t stream);

// S = qp kp^T / sqrt(d) per head, float64 accumulation, [bh, nb, nb] f32.
hipError_t launch_coarse(const float* qp, const float* kp, float* S, long long bh, int nb, int d,
                         hipStream_t stream);

// Top-m column blocks per row of S, ascending, into idx [bh, nb, m].
hipError_t launch_select(const float* S, int32_t* idx, long long bh, int nb, int m,
                         hipStream_t stream);

// Low-resolution term (cmax, csum, cvec) of the blocks not listed in idx.
hipError_t launch_coarse_term(const float* S, const int32_t* idx, const float* vp, float* cmax,
                              float* csum, float* cvec, long long bh, int nb, int d, int m,
                              hipStream_t stream);

// Head-wide selection (one budget per head over all nb x nb blocks, optional
// diagonal priors) into idx [bh, nb, nb]: ascending rows padded with -1.
hipError_t launch_select_global(const float* S, int32_t* idx, long long bh, int nb, int budget,
                                int prior_diagonal, hipStream_t stream);

// Coarse logits and selection in one pass (the logits kept in LDS), for the
// sparse-only variant; same arithmetic and order as the two calls above.
hipError_t launch_select_fused(const float* qp, const float* kp, int32_t* idx, long long bh,
                               int nb, int d, int m, hipStream_t stream);

// Coarse logits, selection and low-resolution term in one pass, the logits
// kept in LDS (same arithmetic and order as the three calls above).
hipError_t launch_select_term_fused(const float* qp, const float* kp, int32_t* idx,
                                    const float* vp, float* cmax, float* csum, float* cvec,
                                    long long bh, int nb, int d, int m, hipStream_t stream);

// Selected 32x32 tiles, merge with the low-resolution term (or none if cmax is
// NULL) and normalise into out [bh, n, d] of dtype. K and V are read from
// kvpacked when it is not NULL, else from the row-major k and v.
hipError_t launch_tile(const void* q, const void* k, const void* v, const void* kvpacked,
                       const int32_t* idx, const float* cmax, const float* csum,
                       const float* cvec, void* out, long long bh, int n, int d, int m, int dtype,
                       hipStream_t stream);

}  // namespace mra
