// Launchers of the MRA-2 kernels (internal; the public interface is mra.h).
// Every launcher only enqueues on `stream` and returns hipGetLastError().
// Arguments are assumed validated by the caller (api.cpp).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "mra.h"

namespace mra {

// The forward's host-side half, shared by mra_attention_forward and the entry
// point without a workspace argument (api.cpp). forward_check runs every
// argument check of mra_attention_forward except those of the workspace,
// makes no HIP call, and on MRA_OK sets *need to the workspace bytes and
// *empty when there is nothing to compute. forward_enqueue enqueues the three
// launches of the forward with the given workspace (at least *need bytes,
// 16-byte aligned) for arguments that passed forward_check.
mra_status_t forward_check(const void* q, const void* k, const void* v, const void* out,
                           const int32_t* idx_out, const float* lse_out, int B, int H, int n,
                           int d, int block, int budget, mra_dtype_t dtype, size_t* need,
                           bool* empty);
mra_status_t forward_enqueue(const void* q, const void* k, const void* v, void* out,
                             int32_t* idx_out, float* lse_out, void* workspace, int B, int H,
                             int n, int d, int budget, mra_dtype_t dtype, void* stream);
// MRA_OK for hipSuccess; otherwise records e as the calling thread's last HIP
// error (mra_last_hip_error) and returns MRA_ERR_HIP.
mra_status_t hip_error_status(hipError_t e);

// Packed K/V (written by the pooling pass, read by the tile pass): for every
// head and 32-key block y, the tile's matrix-core operands in lane order, 16
// bytes per lane and instruction, 32*d elements per block. The K part (all
// blocks) comes first, then the V part.
//  K, chunk s*64 + 32h + j: K[j][(d/2)h + e*s .. +e-1], e = 8 (bf16) or 4 (f32)
//  V bf16, chunk (u*NT + t)*64 + 32h + j, NT = d/32: the 8 values
//        V[16u + 8(s/4) + 4h + s%4][32t + j], s = 0..7 (u = 0, 1)
//  V f32, chunk (t*4 + a)*64 + 32h + j: V[8a + 4h + kk][32t + j], kk = 0..3

// One tensor of a packing launch: src [bh, n, d] of dtype; each output may be
// NULL: pooled (block means, [bh, n/32, d] f32), row_layout (the K part's
// layout above) and t_layout (the V part's layout above), each bh*n*d
// elements of dtype.
struct PackJob {
  const void* src;
  float* pooled;
  void* row_layout;
  void* t_layout;
};
struct PackJobs {
  PackJob job[4];
};

// Up to four packing jobs in one launch (jobs with src NULL do nothing).
hipError_t launch_pack(const PackJob* jobs, int njobs, long long bh, int n, int d, int dtype,
                       hipStream_t stream);

// Block-means of q/k/v ([bh, n, d], dtype) into qp/kp/vp ([bh, n/32, d] f32);
// a NULL output skips that tensor. If kvpacked is not NULL (k, v, kp, vp
// given), the packed copies of k and v are written too.
hipError_t launch_pool(const void* q, const void* k, const void* v, float* qp, float* kp,
                       float* vp, void* kvpacked, long long bh, int n, int d, int dtype,
                       hipStream_t stream);

// S = qp kp^T / sqrt(d) per head, float64 accumulation, [bh, nb, nb] f32.
hipError_t launch_coarse(const float* qp, const float* kp, float* S, long long bh, int nb, int d,
                         hipStream_t stream);

// Debug aid: every 32-bit word of p[0 .. bytes/4) set to `pattern`.
hipError_t launch_fill(void* p, size_t bytes, uint32_t pattern, hipStream_t stream);

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
// NULL) and normalise into out [bh, n, d] of dtype; if lse is not NULL, each
// query's natural log normaliser into lse [bh, n] f32. K and V are read from
// kvpacked when it is not NULL, else from the row-major k and v.
hipError_t launch_tile(const void* q, const void* k, const void* v, const void* kvpacked,
                       const int32_t* idx, const float* cmax, const float* csum,
                       const float* cvec, void* out, float* lse, long long bh, int n, int d,
                       int m, int dtype, hipStream_t stream);

// Gradient pass (bwd.hip) of one MRA-2 forward with the selection held fixed.
// Inputs q, k, v, out (Z), dout (G) [bh, n, d] of dtype; lse [bh, n] f32 (the
// forward's natural log normalisers); idx [bh, n/32, m] (entries outside
// [0, n/32) ignored, the others distinct); coarse = false for the
// sparse-only variant. Outputs dq, dk, dv [bh, n, d] of dtype. The remaining
// pointers are workspace: pooled rows (coarse only) [bh, nb, d] f32; packed
// operand copies (row / transposed layout above) of bh*n*d elements of
// dtype (float32 only: the bfloat16 passes read raw tiles); ld [bh*nb, 64] f32 (per block-row: 32 log normalisers in log2 units,
// then 32 deltas); bias [bh*n] x 16 bytes (bfloat16 only, else
// NULL: per query the bfloat16 triples hi + mid + lo of -L_i/c and of
// -delta_i, the A operand that adds both to the column pass's products);
// bits [bh*nb, ceil(nb/32)] u32; gh, dqp, dkp, dvp [bh, nb, d] f32 and W, dS
// [bh, nb, nb] f32 (coarse only).
struct BwdArgs {
  const void *q, *k, *v, *out, *dout;
  const float* lse;
  const int32_t* idx;
  void *dq, *dk, *dv;
  long long bh;
  int n, d, m, dtype;
  bool coarse;
  bool pooled_in;                 // qp, kp, vp hold the block means already
  float *qp, *kp, *vp;
  void *q_row, *q_t, *k_row, *k_t, *v_row, *g_row, *g_t;
  float* ld;
  uint32_t* bias;
  uint32_t* bits;
  float *gh, *W, *dS, *dqp, *dkp, *dvp;
};
hipError_t launch_bwd(const BwdArgs& args, hipStream_t stream);

// More resolutions R = {s_0 > ... > s_{L-1} = 32, 1} (multilevel.hip).
// Scale-32r means [bh, nb/r, d] of the scale-32 means [bh, nb, d] (f32; a NULL
// pair is skipped); rows_out = bh * nb / r.
hipError_t launch_pool_up(const float* qp, const float* kp, const float* vp, float* qp0,
                          float* kp0, float* vp0, long long rows_out, int d, int r,
                          hipStream_t stream);
// S [bh, nb, nb] of one level in place: -inf outside the children of the
// parent level's kept blocks idx1 [bh, nb0, m1] (nb0 = nb / r <= 1024) of each
// row's parent row.
hipError_t launch_mask_candidates(float* S, const int32_t* idx1, long long bh, int nb, int nb0,
                                  int r, int m1, hipStream_t stream);
// The levels of R = {s_0 > ... > s_{L-1} = 32, 1}: per level l the coarse
// logits S [bh, nb_l, nb_l], the kept blocks idx [bh, nb_l, m_l] (entries
// outside [0, nb_l) ignored), the pooled values vp [bh, nb_l, d] and
// r_l = s_l / 32.
constexpr int kMaxLevels = 8;
struct LevelTerm {
  const float* S[kMaxLevels];
  const int32_t* idx[kMaxLevels];
  const float* vp[kMaxLevels];
  int nb[kMaxLevels], m[kMaxLevels], r[kMaxLevels];
  int levels;
};
// Low-resolution term (cmax, csum, cvec) of every 32-block-row: at every
// level, the candidate blocks its ancestor did not keep.
hipError_t launch_coarse_term_levels(const LevelTerm& T, float* cmax, float* csum, float* cvec,
                                     long long bh, int d, hipStream_t stream);

}  // namespace mra
