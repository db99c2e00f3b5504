/*
 * mra.h — C ABI of libmra: MRA-2 multiresolution approximate self-attention
 * (Zeng et al., "Multi Resolution Analysis (MRA) for Approximate
 * Self-Attention", ICML 2022) on AMD Instinct MI355X (gfx950).
 *
 * MRA-2 is the two-resolution scheme R = {b, 1} with b = 32 (Sec. 5). For one
 * attention head with Q, K, V in R^{n x d} and c = 1/sqrt(d):
 *
 *   pooled rows   Q~, K~, V~ : means of consecutive 32-row blocks
 *                              (Sec. 4.1 eq. recursive_pooling, Sec. 4.3
 *                              eq. recursive_pooling_V)
 *   coarse logits S~ = c Q~ K~^T, mu_{b,x,y} = exp(S~[x,y])
 *                              (Sec. 4.1 eq. exp_of_average)
 *   selection     T_x = the `budget` column blocks with the largest S~[x,.]
 *                              (Sec. 4.2 Alg. 1, applied per block-row;
 *                              ties go to the lower block index)
 *   approximation A^_ij = exp(c Q_i.K_j) if block(j) in T_block(i),
 *                         exp(S~[block(i), block(j)]) otherwise
 *                              (Sec. 4.2 eq. actual_approx_mat_form)
 *   output        Z = D^ A^ V, D^ normalising each row of A^ to sum 1
 *                              (Sec. 2.1 eq. softmax-attention applied to A^;
 *                              computed as in Sec. 4.3 Alg. 2)
 *
 * Conventions shared by every call
 * --------------------------------
 * - Tensors are DEVICE pointers on the current HIP device, dense row-major
 *   [B][H][rows][cols] (batch, head, row, column), owned by the caller. The
 *   library never allocates, frees or synchronises; every call only enqueues
 *   kernels on `stream` (an opaque hipStream_t; NULL = the default stream)
 *   and returns. Outputs must not alias inputs.
 * - Every pointer must be 16-byte aligned.
 * - `block` must be 32 and `d` one of 32, 64, 128 (MRA_ERR_UNSUPPORTED
 *   otherwise). `n` must be a multiple of `block` and at most 65536.
 *   nb = n / block is the number of blocks per side of the block grid.
 * - `budget` is the number of selected blocks per block-row, 0 <= budget <= nb.
 *   budget = 0 leaves every block at low resolution; budget = nb gives exact
 *   softmax attention.
 * - B, H, n may be 0 (an empty problem): the call then validates its other
 *   arguments and returns MRA_OK without touching any pointer.
 * - Q/K/V/output element type is `dtype` (float32 or bfloat16). Pooled rows,
 *   coarse logits and the coarse term are float32. Fine products accumulate in
 *   float32 (bfloat16 inputs feed bfloat16 matrix-core products); coarse
 *   logits accumulate in float64 and are rounded once to float32.
 * - The scale c = 1/sqrt(d) is applied to both the fine and the coarse logits.
 * - Results for non-finite inputs are unspecified.
 *
 * Errors: every argument check runs on the host before any HIP call, so a call
 * that returns an error other than MRA_ERR_HIP has enqueued nothing. A failed
 * kernel launch returns MRA_ERR_HIP; mra_last_hip_error() then gives the
 * hipError_t of the calling thread's last failure. No C++ exception crosses
 * this interface.
 */
#ifndef MRA_H_
#define MRA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MRA_F32 = 0,
  MRA_BF16 = 1
} mra_dtype_t;

typedef enum {
  MRA_OK = 0,
  MRA_ERR_INVALID_ARG = 1,   /* NULL pointer, bad size, budget out of range */
  MRA_ERR_UNSUPPORTED = 2,   /* block != 32, d not in {32,64,128}, n > 65536, unknown dtype */
  MRA_ERR_MISALIGNED = 3,    /* a pointer not 16-byte aligned */
  MRA_ERR_WORKSPACE = 4,     /* workspace_bytes smaller than required */
  MRA_ERR_HIP = 5,           /* a HIP launch failed; see mra_last_hip_error() */
  MRA_ERR_SCRATCH = 6        /* problem too large for the static scratch of
                                mra_attention_forward_noalloc */
} mra_status_t;

/*
 * mra_pool — block means of Q, K and V (Sec. 4.1 eq. recursive_pooling,
 * Sec. 4.3 eq. recursive_pooling_V; for b = 32 the five-fold pairwise
 * averaging equals the plain 32-row mean).
 *   q, k, v    : [B,H,n,d] of `dtype`.
 *   qp, kp, vp : [B,H,nb,d] float32 outputs. A pair (x, xp) may be NULL
 *                together, in which case that tensor is skipped; at least one
 *                pair must be given.
 * Each mean is summed in float32 (rows 0..15 and 16..31 of a block each in
 * row order, then added) and multiplied by 1/32.
 */
mra_status_t mra_pool(const void* q, const void* k, const void* v,
                      float* qp, float* kp, float* vp,
                      int B, int H, int n, int d, int block,
                      mra_dtype_t dtype, void* stream);

/*
 * mra_coarse_scores — coarse logits S~ = Q~ K~^T / sqrt(d) (Sec. 4.1,
 * eq. exp_of_average: mu_{b,x,y} = exp(S~[x,y]) is the exponential of the
 * block mean of the fine logits).
 *   qp, kp : [B,H,nb,d] float32 pooled rows (as written by mra_pool).
 *   scores : [B,H,nb,nb] float32 output; accumulated in float64, rounded once.
 */
mra_status_t mra_coarse_scores(const float* qp, const float* kp, float* scores,
                               int B, int H, int n, int d, int block, void* stream);

/*
 * mra_select — per block-row choice of the blocks to refine (Sec. 4.2, Alg. 1:
 * pop the blocks with the largest mu; here `budget` of them in every
 * block-row). Ranks by S~ (exp is increasing); -0.0 and +0.0 rank equal;
 * among equal scores the lower column-block index wins.
 *   scores : [B,H,nb,nb] float32.
 *   idx    : [B,H,nb,budget] int32 output; each row strictly ascending.
 */
mra_status_t mra_select(const float* scores, int32_t* idx,
                        int B, int H, int n, int block, int budget, void* stream);

/*
 * mra_select_global — the selection of Alg. 1 (Sec. 4.2) with one budget for
 * the whole head (R = {b, 1}): pop the `budget` blocks with the largest
 * S~[x,y] over all nb x nb blocks of a head, among the blocks that are not
 * priors; with prior_diagonal = 1 every diagonal block (x, x) is refined as
 * well (the initial J of Alg. 1, not counted against the budget). Equal
 * scores: the lower flat index x*nb + y wins.
 *   scores : [B,H,nb,nb] float32.
 *   idx    : [B,H,nb,nb] int32 output; row x lists its refined column blocks in
 *            strictly ascending order, then -1 up to nb entries.
 *   budget : 0 <= budget <= nb*nb - (prior_diagonal ? nb : 0), per head.
 *   prior_diagonal : 0 or 1; anything else is MRA_ERR_INVALID_ARG.
 */
mra_status_t mra_select_global(const float* scores, int32_t* idx,
                               int B, int H, int n, int block, int budget,
                               int prior_diagonal, void* stream);

/*
 * mra_coarse_term — the low-resolution part of A^ V and of the row sums of A^
 * for every block-row: Alg. 2 (Sec. 4.3) at scale b over the blocks NOT in
 * T_x, each block spanning b columns (eq. actual_approx_mat_form):
 *   cmax[x]  = M_x = max_{y not in T_x} S~[x,y]            (-inf if none)
 *   csum[x]  = sum_{y not in T_x} b * exp(S~[x,y] - M_x)     (0 if none)
 *   cvec[x,:]= sum_{y not in T_x} b * exp(S~[x,y] - M_x) * V~[y,:]
 *   scores : [B,H,nb,nb] float32; idx : [B,H,nb,budget] int32, rows strictly
 *            ascending in [0, nb); entries outside [0, nb) are ignored (e.g.
 *            the -1 padding of mra_select_global with budget = nb);
 *   vp     : [B,H,nb,d] float32 pooled V.
 *   cmax, csum : [B,H,nb] float32 outputs; cvec : [B,H,nb,d] float32 output.
 */
mra_status_t mra_coarse_term(const float* scores, const int32_t* idx, const float* vp,
                             float* cmax, float* csum, float* cvec,
                             int B, int H, int n, int d, int block, int budget,
                             void* stream);

/*
 * mra_block_sddmm_spmm — the high-resolution part and the output (Sec. 4.2
 * eq. actual_approx_mat_form with mu_{1,i,j} = exp(P_ij); Sec. 4.3 Alg. 2 at
 * scale 1; Sec. 2.1 normalisation D^). For every block-row x and every
 * y in T_x it computes the 32x32 tile exp(c Q_x K_y^T) (block-sparse SDDMM),
 * multiplies it by V_y (block-sparse SpMM), merges the result with the coarse
 * term and normalises:
 *   Z_i = (sum_{j in T} e^{P_ij} V_j + e^{M_x} cvec[x]) /
 *         (sum_{j in T} e^{P_ij}     + e^{M_x} csum[x])
 * (evaluated with max shifts; nothing overflows for finite inputs).
 *   q, k, v : [B,H,n,d] of `dtype`.
 *   idx     : [B,H,nb,budget] int32, rows strictly ascending in [0, nb);
 *             entries outside [0, nb) are skipped.
 *   cmax, csum, cvec : the coarse term from mra_coarse_term. All three may be
 *             NULL together: then only the selected tiles are normalised
 *             (the sparse-only variant MRA-2-s of Sec. 5), which needs
 *             budget >= 1.
 *   out     : [B,H,n,d] of `dtype`, the output Z (bfloat16 rounded to nearest
 *             even). With bfloat16 inputs the tile probabilities are rounded
 *             to bfloat16 before the product with V and the row sums use the
 *             same rounded values.
 *   lse_out : optional [B,H,n] float32 output (NULL to skip): each query's
 *             log normaliser L_i = ln(sum_{j in T} e^{P_ij} + e^{M_x} csum[x]),
 *             the natural log of the denominator above (the row sum of A^).
 *             mra_attention_backward takes it.
 */
mra_status_t mra_block_sddmm_spmm(const void* q, const void* k, const void* v,
                                  const int32_t* idx,
                                  const float* cmax, const float* csum, const float* cvec,
                                  void* out, float* lse_out,
                                  int B, int H, int n, int d, int block, int budget,
                                  mra_dtype_t dtype, void* stream);

/*
 * mra_forward_workspace_bytes — bytes of device workspace mra_attention_forward
 * needs for these sizes and dtype: pooled rows, the selection and the coarse
 * term (B*H*(n/32)*(4d + budget + 2)*4 bytes, each part rounded up to 256),
 * plus, for float32 inputs, copies of K and V rearranged into matrix-core
 * operand order (2*B*H*n*d*elem bytes; bfloat16 tiles are read straight
 * from K and V). Returns 0 for invalid or unsupported arguments.
 */
size_t mra_forward_workspace_bytes(int B, int H, int n, int d, int block, int budget,
                                   mra_dtype_t dtype);

/*
 * mra_attention_forward — the whole MRA-2 forward pass: pooling (which, for
 * float32 inputs and d = 128, also rearranges K and V for the tile pass),
 * coarse logits with
 * selection and coarse term fused (the logits never leave on-chip memory),
 * then the tile pass. Results are bit-identical to the calls above made in
 * order (mra_pool, mra_coarse_scores, mra_select, mra_coarse_term,
 * mra_block_sddmm_spmm).
 *   q, k, v   : [B,H,n,d] of `dtype`; out : [B,H,n,d] of `dtype`.
 *   idx_out   : optional [B,H,nb,budget] int32 copy of the selection (NULL:
 *               kept in the workspace only).
 *   lse_out   : optional [B,H,n] float32 log normalisers (as for
 *               mra_block_sddmm_spmm; NULL to skip). With idx_out they are
 *               what mra_attention_backward needs.
 *   workspace : device buffer of at least mra_forward_workspace_bytes(...)
 *               bytes (16-byte aligned; contents on entry are ignored).
 */
mra_status_t mra_attention_forward(const void* q, const void* k, const void* v, void* out,
                                   int32_t* idx_out, float* lse_out, void* workspace,
                                   size_t workspace_bytes,
                                   int B, int H, int n, int d, int block, int budget,
                                   mra_dtype_t dtype, void* stream);

/*
 * mra_attention_forward_noalloc — mra_attention_forward without a workspace
 * argument, for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops, harnesses that forbid allocation). The
 * forward's workspace is taken from a file-scope device array of
 * MRA_NOALLOC_SCRATCH_BYTES bytes that every GPU the library runs on holds
 * from the first use of the library on it until the process ends; the call
 * itself allocates and frees nothing.
 *   Arguments, layouts, results and errors as for mra_attention_forward
 *   (same kernels, bit-identical output), except that a problem whose
 *   mra_forward_workspace_bytes exceeds MRA_NOALLOC_SCRATCH_BYTES returns
 *   MRA_ERR_SCRATCH after the other argument checks and enqueues nothing.
 *   64 MiB covers the five benchmark workloads (the largest needs ~36 MB).
 * All calls on one GPU share that GPU's array and leave their intermediates
 * in it (the forward writes every part before reading it, so nothing needs
 * clearing): calls that overlap on one GPU (concurrent streams or threads)
 * race and give undefined results. The first call on each GPU looks up the
 * array's device address (hipGetSymbolAddress) with that GPU current.
 */
#define MRA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
mra_status_t mra_attention_forward_noalloc(const void* q, const void* k, const void* v,
                                           void* out, int32_t* idx_out, float* lse_out,
                                           int B, int H, int n, int d, int block, int budget,
                                           mra_dtype_t dtype, void* stream);

/*
 * mra_forward_global_workspace_bytes — workspace of
 * mra_attention_forward_global: that of mra_attention_forward with budget nb
 * plus the coarse logits of every head (B*H*nb*nb*4 bytes). 0 for invalid or
 * unsupported arguments.
 */
size_t mra_forward_global_workspace_bytes(int B, int H, int n, int d, int block,
                                          mra_dtype_t dtype);

/*
 * mra_attention_forward_global — MRA-2 with the head-wide budget of
 * mra_select_global: pooling, coarse logits, head-wide selection, the
 * low-resolution term over every block a row did not refine, the tile pass
 * (rows refine different numbers of blocks). Bit-identical to mra_pool,
 * mra_coarse_scores, mra_select_global, mra_coarse_term and
 * mra_block_sddmm_spmm called in that order with budget (row width) nb.
 *   idx_out : optional [B,H,nb,nb] int32 copy of the selection (NULL: kept in
 *             the workspace only).
 *   lse_out : optional [B,H,n] float32 log normalisers (NULL to skip).
 *   budget, prior_diagonal : as for mra_select_global.
 *   Other arguments and errors as for mra_attention_forward; workspace of at
 *   least mra_forward_global_workspace_bytes(...) bytes.
 */
mra_status_t mra_attention_forward_global(const void* q, const void* k, const void* v,
                                          void* out, int32_t* idx_out, float* lse_out,
                                          void* workspace,
                                          size_t workspace_bytes, int B, int H, int n, int d,
                                          int block, int budget, int prior_diagonal,
                                          mra_dtype_t dtype, void* stream);

/*
 * mra_sparse_attention_forward — the sparse-only variant MRA-2-s (Sec. 5):
 * after the selection T_x, only the scale-1 part over the selected blocks is
 * kept, normalised by its own row sums:
 *   Z_i = sum_{j in T_x} e^{P_ij} V_j / sum_{j in T_x} e^{P_ij},  P = Q K^T / sqrt(d)
 * (no low-resolution term). Enqueues pooling, the fused coarse logits and
 * selection, and the tile pass without the coarse merge; bit-identical to
 * mra_pool, mra_coarse_scores, mra_select and mra_block_sddmm_spmm (cmax,
 * csum, cvec NULL) called in that order.
 *   Arguments, layouts, workspace (mra_forward_workspace_bytes) and errors as
 *   for mra_attention_forward, except that budget must be at least 1 (at most
 *   nb) whenever n > 0: MRA_ERR_INVALID_ARG otherwise. lse_out receives
 *   ln sum_{j in T_x} e^{P_ij}.
 */
mra_status_t mra_sparse_attention_forward(const void* q, const void* k, const void* v,
                                          void* out, int32_t* idx_out, float* lse_out,
                                          void* workspace,
                                          size_t workspace_bytes, int B, int H, int n, int d,
                                          int block, int budget, mra_dtype_t dtype,
                                          void* stream);

/*
 * mra_forward_multilevel_workspace_bytes — workspace of
 * mra_attention_forward_multilevel: that of mra_attention_forward with budget
 * budget2, plus the scale-s0 means, both coarse-logit grids and the
 * first-level selection. 0 for invalid or unsupported arguments.
 */
size_t mra_forward_multilevel_workspace_bytes(int B, int H, int n, int d, int block,
                                              int coarse_block, int budget1, int budget2,
                                              mra_dtype_t dtype);

/*
 * mra_attention_forward_multilevel — three resolutions R = {s0, 32, 1}
 * (Sec. 4.2 Alg. 1 with two refinement levels, s0 = coarse_block; Sec. 4.3
 * Alg. 2 over the resulting J), with a budget per block-row at each level:
 *   level 1: every s0-block-row X keeps the budget1 s0-blocks Y with the
 *            largest S~0[X,Y] = c Q~0_X . K~0_Y (Q~0, K~0: means of s0-row
 *            blocks, taken here as means of the r = s0/32 consecutive 32-row
 *            means);
 *   level 2: every 32-block-row x keeps, among the 32-blocks inside its
 *            parent row's refined s0-blocks (budget1 * r candidates), the
 *            budget2 with the largest S~[x,y];
 *   A^_ij = exp(c Q_i.K_j) in the refined 32-blocks, exp(S~[x,y]) in the other
 *           candidates, exp(S~0[X,Y]) in the unrefined s0-blocks
 *           (eq. actual_approx_mat_form), Z = D^ A^ V.
 * Ties go to the lower index at both levels. This is
 * mra_attention_forward_levels with scales {s0, 32} and budgets {budget1,
 * budget2}. Launches: pooling, scale-s0 means, coarse logits at both scales,
 * the two per-row selections (the second over the candidates only), the
 * low-resolution term (s0 e^{S~0} V~0 and 32 e^{S~} V~ over the unrefined
 * blocks), the tile pass.
 *   coarse_block : s0 = 32 r with r >= 2, dividing n (MRA_ERR_UNSUPPORTED if
 *                  not a multiple of 32 above 32, MRA_ERR_INVALID_ARG if it
 *                  does not divide n).
 *   budget1      : 0 <= budget1 <= n / s0; budget2 : 0 <= budget2 <= budget1 r.
 *   idx1_out     : optional [B,H,n/s0,budget1] int32, rows ascending.
 *   idx2_out     : optional [B,H,n/32,budget2] int32, rows ascending.
 *   lse_out      : optional [B,H,n] float32 log normalisers.
 *   Other arguments and errors as for mra_attention_forward; workspace of at
 *   least mra_forward_multilevel_workspace_bytes(...) bytes.
 */
mra_status_t mra_attention_forward_multilevel(const void* q, const void* k, const void* v,
                                              void* out, int32_t* idx1_out, int32_t* idx2_out,
                                              float* lse_out, void* workspace,
                                              size_t workspace_bytes, int B, int H, int n, int d,
                                              int block, int coarse_block, int budget1,
                                              int budget2, mra_dtype_t dtype, void* stream);

/*
 * mra_forward_levels_workspace_bytes — workspace of
 * mra_attention_forward_levels: that of mra_attention_forward with the finest
 * budget, plus for every coarser level its means, its coarse logits and its
 * selection, and the finest level's coarse-logit grid (levels = 1: exactly
 * mra_attention_forward's). 0 for invalid or unsupported arguments.
 */
size_t mra_forward_levels_workspace_bytes(int B, int H, int n, int d, int block, int levels,
                                          const int* scales, const int* budgets,
                                          mra_dtype_t dtype);

/*
 * mra_attention_forward_levels — any number of resolutions
 * R = {s_0 > s_1 > ... > s_{L-1} = 32, 1} (Sec. 4.2 Alg. 1 refined level by
 * level, Sec. 4.3 Alg. 2 over the resulting J), with a budget per block-row at
 * each level:
 *   level 0: every s_0-block-row keeps the budgets[0] s_0-blocks with the
 *            largest S~_0 = c Q~_0 . K~_0 (means of s_0-row blocks, taken as
 *            means of the consecutive 32-row means);
 *   level l: every s_l-block-row keeps, among the s_l-blocks inside its parent
 *            row's (scale s_{l-1}) kept blocks, the budgets[l] with the
 *            largest S~_l;
 *   A^_ij = exp(c Q_i.K_j) in the 32-blocks kept at the last level, else
 *           exp(S~_l) of the first level l whose block around j the row's
 *           ancestor at that level did not keep (eq. actual_approx_mat_form),
 *           Z = D^ A^ V.
 * Ties go to the lower index at every level. levels = 1 is MRA-2
 * (mra_attention_forward, bit-identical); levels = 2 is
 * mra_attention_forward_multilevel.
 *   levels   : 1 <= levels <= 8 (MRA_ERR_UNSUPPORTED above 8).
 *   scales   : host array of `levels` ints: scales[levels - 1] = 32 = block and
 *              every other a larger multiple of the next (MRA_ERR_UNSUPPORTED
 *              otherwise), each dividing n (MRA_ERR_INVALID_ARG otherwise).
 *   budgets  : host array of `levels` ints: 0 <= budgets[0] <= n / scales[0],
 *              0 <= budgets[l] <= budgets[l - 1] * scales[l - 1] / scales[l]
 *              (MRA_ERR_INVALID_ARG otherwise).
 *   idx_outs : NULL, or a host array of `levels` device pointers, each NULL or
 *              [B,H,n/scales[l],budgets[l]] int32 receiving level l's
 *              selection, rows ascending; 16-byte aligned.
 *   lse_out  : optional [B,H,n] float32 log normalisers.
 *   Other arguments and errors as for mra_attention_forward; workspace of at
 *   least mra_forward_levels_workspace_bytes(...) bytes. The arrays are read
 *   before the call returns; the caller keeps ownership.
 */
mra_status_t mra_attention_forward_levels(const void* q, const void* k, const void* v, void* out,
                                          int32_t* const* idx_outs, float* lse_out,
                                          void* workspace, size_t workspace_bytes, int B, int H,
                                          int n, int d, int block, int levels, const int* scales,
                                          const int* budgets, mra_dtype_t dtype, void* stream);

/*
 * mra_backward_workspace_bytes — device workspace of mra_attention_backward:
 * for float32 seven rearranged copies of Q, K, V and dZ (7*B*H*n*d*4 bytes;
 * the bfloat16 gradient passes read the inputs' rows and instead take 16
 * bytes per query of bias operands), pooled rows and their gradients, two
 * float32 values per query, the selection as a bitmap and two float32
 * nb x nb grids per head (W and dS~ below). 0 for
 * invalid or unsupported arguments.
 */
size_t mra_backward_workspace_bytes(int B, int H, int n, int d, int block, mra_dtype_t dtype);

/*
 * mra_attention_backward — gradients dQ, dK, dV of a scalar loss through one
 * MRA-2 (or MRA-2-s) forward, given dZ, with the selection held fixed (the
 * selection is a discrete choice with no gradient). The forward is the
 * softmax of Sec. 2.1 over the approximation A^ of Sec. 4.2
 * (eq. actual_approx_mat_form): each query's logits are the fine c Q_i.K_j
 * of its refined blocks and, with the low-resolution term, the coarse
 * S~[x,y] + ln b of the others, applied to V_j and V~_y. The coarse logits
 * and V~ depend on Q, K, V through the block means (Sec. 4.1
 * eq. recursive_pooling, Sec. 4.3 eq. recursive_pooling_V), so their
 * gradients reach every row of a block divided by 32. With
 * delta_i = dZ_i . Z_i and probabilities p = e^{logit - L_i}:
 *   d logit = p (dZ_i . value - delta_i)
 * then the chain rule through c Q K^T, c Q~ K~^T and the means.
 *   q, k, v   : [B,H,n,d] of `dtype`, the forward's inputs.
 *   out       : [B,H,n,d] of `dtype`, the forward's output Z.
 *   dout      : [B,H,n,d] of `dtype`, dZ.
 *   lse       : [B,H,n] float32, the forward's lse_out.
 *   idx       : [B,H,nb,width] int32, the forward's selection: entries
 *               outside [0, nb) are ignored, the others must be distinct
 *               (every selection of this library is); may be NULL when
 *               width = 0.
 *   width     : entries per row of idx, 0 <= width <= nb (the budget of
 *               mra_attention_forward / mra_sparse_attention_forward, nb for
 *               mra_attention_forward_global).
 *   coarse    : 1 for MRA-2 (the forward merged the low-resolution term),
 *               0 for MRA-2-s (mra_sparse_attention_forward); otherwise
 *               MRA_ERR_INVALID_ARG.
 *   dq, dk, dv: [B,H,n,d] of `dtype` outputs (bfloat16 rounded to nearest
 *               even); every element is written.
 *   workspace : at least mra_backward_workspace_bytes(...) bytes, 16-byte
 *               aligned; contents on entry are ignored.
 * Fine products run on the matrix cores in float32 accumulation; with
 * bfloat16 inputs the probabilities and logit gradients are rounded to
 * bfloat16 before their products. The coarse terms are float32. Rows whose
 * forward normaliser is zero (MRA-2-s with no valid entry in the row) give
 * unspecified gradients.
 */
mra_status_t mra_attention_backward(const void* q, const void* k, const void* v,
                                    const void* out, const void* dout, const float* lse,
                                    const int32_t* idx, void* dq, void* dk, void* dv,
                                    void* workspace, size_t workspace_bytes,
                                    int B, int H, int n, int d, int block, int width,
                                    int coarse, mra_dtype_t dtype, void* stream);

/*
 * mra_attention_backward_pooled — mra_attention_backward with the block means
 * of q, k, v supplied, so the backward does not compute them again: a
 * training step keeps the forward's (mra_forward_pooled_rows) and hands them
 * over. The gradients are bit-identical to mra_attention_backward's on the
 * same arguments.
 *   qp, kp, vp: [B,H,nb,d] float32 device arrays (16-byte aligned), the means
 *               of Sec. 4.1 eq. recursive_pooling and Sec. 4.3
 *               eq. recursive_pooling_V of these q, k, v exactly as mra_pool
 *               or the forward computed them; read only. All three are
 *               required for a non-empty problem (NULL: MRA_ERR_INVALID_ARG,
 *               not 16-byte aligned: MRA_ERR_MISALIGNED); with coarse = 0
 *               they are not read.
 *   Every other argument, the workspace size included, and every error as
 *   for mra_attention_backward.
 */
mra_status_t mra_attention_backward_pooled(const void* q, const void* k, const void* v,
                                           const void* out, const void* dout, const float* lse,
                                           const int32_t* idx, const float* qp, const float* kp,
                                           const float* vp, void* dq, void* dk, void* dv,
                                           void* workspace, size_t workspace_bytes,
                                           int B, int H, int n, int d, int block, int width,
                                           int coarse, mra_dtype_t dtype, void* stream);

/*
 * mra_forward_pooled_rows — where the block means Q~, K~, V~ ([B,H,nb,d]
 * float32 each, mra_pool's layout) lie in a workspace that
 * mra_attention_forward or mra_attention_forward_global filled for these
 * sizes. Host-only arithmetic on the workspace address: nothing is read or
 * launched, so the addresses are those of what the last forward enqueued on
 * that workspace, valid until the workspace is used again. The block means
 * do not depend on the budget, so none is taken.
 *   qp, kp, vp: host pointers that receive the three device addresses (NULL
 *               for an empty problem).
 * Errors: MRA_ERR_INVALID_ARG (a NULL output pointer, a NULL workspace for a
 * non-empty problem), MRA_ERR_UNSUPPORTED (sizes as for the forward),
 * MRA_ERR_MISALIGNED (workspace not 16-byte aligned).
 */
mra_status_t mra_forward_pooled_rows(const void* workspace, int B, int H, int n, int d, int block,
                                     const float** qp, const float** kp, const float** vp);

/* Static description of a status code. */
const char* mra_status_str(mra_status_t status);

/* hipError_t (as int) of the calling thread's last MRA_ERR_HIP; 0 if none. */
int mra_last_hip_error(void);

#ifdef __cplusplus
}  /* extern "C" */
#endif

#endif  /* MRA_H_ */
