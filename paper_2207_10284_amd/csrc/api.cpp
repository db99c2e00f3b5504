// C ABI of libmra (declared in mra.h): argument validation, workspace layout
// and kernel dispatch. Every check runs before the first HIP call, so a
// rejected call has enqueued nothing.
#include "mra.h"

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdlib>

#include "kernels.h"

namespace {

thread_local int g_last_hip_error = 0;

constexpr int kBlockSize = 32;
constexpr int kMaxN = 65536;
constexpr long long kMaxGrid = 2147483647LL;   // workgroups per launch

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Shape {
  long long bh = 0;
  int nb = 0;
  bool empty = true;
};

// B, H, n, block (and d when d_needed) checks shared by every call.
mra_status_t check_shape(int B, int H, int n, int d, int block, bool d_needed, Shape* s) {
  if (B < 0 || H < 0 || n < 0 || block <= 0) return MRA_ERR_INVALID_ARG;
  if (d_needed && d <= 0) return MRA_ERR_INVALID_ARG;
  if (block != kBlockSize) return MRA_ERR_UNSUPPORTED;
  if (n % block != 0) return MRA_ERR_INVALID_ARG;
  if (n > kMaxN) return MRA_ERR_UNSUPPORTED;
  if (d_needed && d != 32 && d != 64 && d != 128) return MRA_ERR_UNSUPPORTED;
  s->bh = (long long)B * (long long)H;
  s->nb = n / block;
  s->empty = (s->bh == 0 || n == 0);
  if (!s->empty) {
    const long long rows = s->bh * s->nb;
    const long long nt = (s->nb + 63) / 64;
    // pool: one thread per 16 bytes of a block (at most 32 x 128 / 4 per block-row)
    if (rows * 32 > kMaxGrid) return MRA_ERR_UNSUPPORTED;
    if (s->bh * nt * nt > kMaxGrid) return MRA_ERR_UNSUPPORTED;
  }
  return MRA_OK;
}

mra_status_t check_dtype(mra_dtype_t dt) {
  return (dt == MRA_F32 || dt == MRA_BF16) ? MRA_OK : MRA_ERR_UNSUPPORTED;
}

mra_status_t check_ptr(const void* p) {
  if (p == nullptr) return MRA_ERR_INVALID_ARG;
  return aligned16(p) ? MRA_OK : MRA_ERR_MISALIGNED;
}

mra_status_t hip_status(hipError_t e) {
  if (e == hipSuccess) return MRA_OK;
  g_last_hip_error = (int)e;
  return MRA_ERR_HIP;
}

// Debug aid: with MRA_DEBUG_NANFILL=1 in the environment, every call that
// computes fills its outputs and the part of the workspace it uses with quiet
// NaN before its kernels run (bfloat16 outputs with bfloat16 NaNs; index
// outputs with the same bits, an id outside every block range). An element
// the call fails to write then stays NaN (or an invalid id), and a value read
// before the call wrote it turns the results that depend on it into NaN.
bool nanfill_enabled() {
  const char* e = std::getenv("MRA_DEBUG_NANFILL");
  return e != nullptr && e[0] == '1';
}

constexpr uint32_t kNanF32 = 0x7FC00000u;        // float32 quiet NaN
constexpr uint32_t kNanBf16x2 = 0x7FC07FC0u;     // two bfloat16 quiet NaNs

uint32_t nan_pattern(mra_dtype_t dt) { return dt == MRA_BF16 ? kNanBf16x2 : kNanF32; }

#define MRA_TRY(expr)                 \
  do {                                \
    const mra_status_t st_ = (expr);  \
    if (st_ != MRA_OK) return st_;    \
  } while (0)

// Fills the (pointer, bytes, pattern) buffers when the debug flag is set.
struct Fill {
  void* p;
  size_t bytes;
  uint32_t pattern;
};
template <int N>
mra_status_t debug_fill(const Fill (&f)[N], void* stream) {
  if (!nanfill_enabled()) return MRA_OK;
  for (const Fill& x : f)
    MRA_TRY(hip_status(mra::launch_fill(x.p, x.bytes, x.pattern, static_cast<hipStream_t>(stream))));
  return MRA_OK;
}

struct WsLayout {
  size_t qp, kp, vp, kvpacked, idx, cmax, csum, cvec, total;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// The forward's tile pass reads K/V tiles straight from their rows (bfloat16,
// and float32 with d <= 64); float32 tiles of d = 128 need the copy in
// matrix-core operand order that the pooling pass writes.
bool raw_tiles(int d, mra_dtype_t dtype) { return dtype == MRA_BF16 || d <= 64; }

WsLayout ws_layout(long long bh, int nb, int d, int m, mra_dtype_t dtype) {
  WsLayout L{};
  size_t off = 0;
  const size_t pooled = align256((size_t)bh * nb * d * sizeof(float));
  const size_t elem = dtype == MRA_BF16 ? 2 : 4;
  L.qp = off; off += pooled;
  L.kp = off; off += pooled;
  L.vp = off; off += pooled;
  L.kvpacked = off;
  if (!raw_tiles(d, dtype)) off += align256((size_t)2 * bh * nb * kBlockSize * d * elem);
  L.idx = off; off += align256((size_t)bh * nb * m * sizeof(int32_t));
  L.cmax = off; off += align256((size_t)bh * nb * sizeof(float));
  L.csum = off; off += align256((size_t)bh * nb * sizeof(float));
  L.cvec = off; off += align256((size_t)bh * nb * d * sizeof(float));
  L.total = off;
  return L;
}

// The head-wide-budget forward: the forward's layout with nb-wide selection
// rows, plus the coarse logits of every head (the selection needs all of them).
struct WsGlobal {
  WsLayout base;
  size_t scores, total;
};

WsGlobal ws_global(long long bh, int nb, int d, mra_dtype_t dtype) {
  WsGlobal G{};
  G.base = ws_layout(bh, nb, d, nb, dtype);
  G.scores = G.base.total;
  G.total = G.scores + align256((size_t)bh * nb * nb * sizeof(float));
  return G;
}

mra_status_t check_global_budget(const Shape& s, int budget, int prior_diagonal) {
  if (prior_diagonal != 0 && prior_diagonal != 1) return MRA_ERR_INVALID_ARG;
  const long long nfree = (long long)s.nb * s.nb - (prior_diagonal ? s.nb : 0);
  if (budget < 0 || budget > nfree) return MRA_ERR_INVALID_ARG;
  return MRA_OK;
}

// Workspace of the gradient pass (pointer roles in kernels.h, BwdArgs).
struct WsBwd {
  size_t qp, kp, vp, q_row, q_t, k_row, k_t, v_row, g_row, g_t, ld, bias, bits, gh, W, dS, dqp,
      dkp, dvp, total;
};

WsBwd ws_bwd(long long bh, int nb, int d, mra_dtype_t dtype) {
  WsBwd L{};
  size_t off = 0;
  const size_t pooled = align256((size_t)bh * nb * d * sizeof(float));
  // packed operand copies: float32 only (bfloat16 passes read raw tiles)
  const bool raw = dtype == MRA_BF16;
  const size_t packed = raw ? 0 : align256((size_t)bh * nb * kBlockSize * d * (dtype == MRA_BF16 ? 2 : 4));
  const size_t grid = align256((size_t)bh * nb * nb * sizeof(float));
  L.qp = off; off += pooled;
  L.kp = off; off += pooled;
  L.vp = off; off += pooled;
  L.q_row = off; off += packed;
  L.q_t = off; off += packed;
  L.k_row = off; off += packed;
  L.k_t = off; off += packed;
  L.v_row = off; off += packed;
  L.g_row = off; off += packed;
  L.g_t = off; off += packed;
  L.ld = off; off += align256((size_t)bh * nb * 64 * sizeof(float));
  L.bias = off; off += raw ? align256((size_t)bh * nb * kBlockSize * 16) : 0;
  L.bits = off; off += align256((size_t)bh * nb * ((nb + 31) / 32) * sizeof(uint32_t));
  L.gh = off; off += pooled;
  L.W = off; off += grid;
  L.dS = off; off += grid;
  L.dqp = off; off += pooled;
  L.dkp = off; off += pooled;
  L.dvp = off; off += pooled;
  L.total = off;
  return L;
}

// The forward over levels R = {s_0 > ... > s_{L-1} = 32, 1}: the forward's
// layout with the finest selection as its rows, plus for every coarser level
// l < L - 1 its means, its coarse logits and its selection, and the finest
// level's coarse-logit grid.
struct WsLevels {
  WsLayout base;
  size_t qp[mra::kMaxLevels], kp[mra::kMaxLevels], vp[mra::kMaxLevels], S[mra::kMaxLevels],
      idx[mra::kMaxLevels];
  size_t S_fine, total;
};

WsLevels ws_levels(long long bh, int n, int d, int levels, const int* scales, const int* budgets,
                   mra_dtype_t dtype) {
  WsLevels W{};
  const int nb = n / kBlockSize;
  W.base = ws_layout(bh, nb, d, budgets[levels - 1], dtype);
  size_t off = W.base.total;
  for (int l = 0; l + 1 < levels; ++l) {
    const long long nbl = n / scales[l];
    const size_t pooled = align256((size_t)bh * nbl * d * sizeof(float));
    W.qp[l] = off; off += pooled;
    W.kp[l] = off; off += pooled;
    W.vp[l] = off; off += pooled;
    W.S[l] = off; off += align256((size_t)bh * nbl * nbl * sizeof(float));
    W.idx[l] = off; off += align256((size_t)bh * nbl * budgets[l] * sizeof(int32_t));
  }
  W.S_fine = off; off += align256((size_t)bh * nb * nb * sizeof(float));
  W.total = off;
  return W;
}

// 1 <= levels <= kMaxLevels; scales[levels - 1] = 32 and every coarser scale a
// larger multiple of the next one (else unsupported) dividing n (else
// invalid); 0 <= budgets[0] <= n / scales[0] and
// 0 <= budgets[l] <= budgets[l - 1] * scales[l - 1] / scales[l].
mra_status_t check_levels(int n, int levels, const int* scales, const int* budgets) {
  if (levels < 1 || scales == nullptr || budgets == nullptr) return MRA_ERR_INVALID_ARG;
  if (levels > mra::kMaxLevels) return MRA_ERR_UNSUPPORTED;
  if (scales[levels - 1] != kBlockSize) return MRA_ERR_UNSUPPORTED;
  for (int l = 0; l + 1 < levels; ++l)
    if (scales[l] <= scales[l + 1] || scales[l] % scales[l + 1] != 0) return MRA_ERR_UNSUPPORTED;
  for (int l = 0; l + 1 < levels; ++l)
    if (n % scales[l] != 0) return MRA_ERR_INVALID_ARG;
  if (budgets[0] < 0 || budgets[0] > n / scales[0]) return MRA_ERR_INVALID_ARG;
  for (int l = 1; l < levels; ++l)
    if (budgets[l] < 0 || (long long)budgets[l] > (long long)budgets[l - 1] * (scales[l - 1] / scales[l]))
      return MRA_ERR_INVALID_ARG;
  return MRA_OK;
}

size_t levels_workspace_bytes(int B, int H, int n, int d, int block, int levels, const int* scales,
                              const int* budgets, mra_dtype_t dtype) {
  Shape s;
  if (check_shape(B, H, n, d, block, true, &s) != MRA_OK) return 0;
  if (check_dtype(dtype) != MRA_OK) return 0;
  if (check_levels(n, levels, scales, budgets) != MRA_OK) return 0;
  if (levels == 1) return ws_layout(s.bh, s.nb, d, budgets[0], dtype).total;
  return ws_levels(s.bh, n, d, levels, scales, budgets, dtype).total;
}

// idx_outs: NULL, or `levels` optional device pointers (level l's selection
// [B, H, n / scales[l], budgets[l]]).
mra_status_t levels_forward(const void* q, const void* k, const void* v, void* out,
                            int32_t* const* idx_outs, float* lse_out, void* workspace,
                            size_t workspace_bytes, int B, int H, int n, int d, int block,
                            int levels, const int* scales, const int* budgets, mra_dtype_t dtype,
                            void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  MRA_TRY(check_dtype(dtype));
  MRA_TRY(check_levels(n, levels, scales, budgets));
  if (s.empty) return MRA_OK;
  MRA_TRY(check_ptr(q));
  MRA_TRY(check_ptr(k));
  MRA_TRY(check_ptr(v));
  MRA_TRY(check_ptr(out));
  int32_t* outs[mra::kMaxLevels] = {};
  for (int l = 0; l < levels && idx_outs != nullptr; ++l) outs[l] = idx_outs[l];
  for (int l = 0; l < levels; ++l)
    if (outs[l] != nullptr && !aligned16(outs[l])) return MRA_ERR_MISALIGNED;
  if (lse_out != nullptr && !aligned16(lse_out)) return MRA_ERR_MISALIGNED;
  MRA_TRY(check_ptr(workspace));
  if (workspace_bytes < levels_workspace_bytes(B, H, n, d, block, levels, scales, budgets, dtype))
    return MRA_ERR_WORKSPACE;
  if (levels == 1)                                          // R = {32, 1}: the two-level forward
    return mra::forward_enqueue(q, k, v, out, outs[0], lse_out, workspace, B, H, n, d, budgets[0],
                                dtype, stream);

  const WsLevels W = ws_levels(s.bh, n, d, levels, scales, budgets, dtype);
  char* ws = static_cast<char*>(workspace);
  const WsLayout& L = W.base;
  auto f32 = [&](size_t off) { return reinterpret_cast<float*>(ws + off); };
  const int nb = s.nb, fin = levels - 1;
  float *qp = f32(L.qp), *kp = f32(L.kp), *vp = f32(L.vp), *S = f32(W.S_fine);
  void* kvpacked = raw_tiles(d, dtype) ? nullptr : ws + L.kvpacked;
  float *cmax = f32(L.cmax), *csum = f32(L.csum), *cvec = f32(L.cvec);
  hipStream_t st = static_cast<hipStream_t>(stream);
  mra::LevelTerm T{};
  T.levels = levels;
  for (int l = 0; l < levels; ++l) {
    T.nb[l] = n / scales[l];
    T.m[l] = budgets[l];
    T.r[l] = scales[l] / kBlockSize;
  }
  int32_t* idx[mra::kMaxLevels];
  for (int l = 0; l < fin; ++l) {
    idx[l] = outs[l] ? outs[l] : reinterpret_cast<int32_t*>(ws + W.idx[l]);
    T.S[l] = f32(W.S[l]);
    T.vp[l] = f32(W.vp[l]);
  }
  idx[fin] = outs[fin] ? outs[fin] : reinterpret_cast<int32_t*>(ws + L.idx);
  T.S[fin] = S;
  T.vp[fin] = vp;
  for (int l = 0; l < levels; ++l) T.idx[l] = idx[l];

  Fill fills[mra::kMaxLevels + 3] = {{out, (size_t)s.bh * n * d * (dtype == MRA_BF16 ? 2 : 4), nan_pattern(dtype)},
                                     {lse_out, (size_t)s.bh * n * 4, kNanF32},
                                     {workspace, W.total, kNanF32}};
  for (int l = 0; l < levels; ++l) fills[3 + l] = {outs[l], (size_t)s.bh * T.nb[l] * budgets[l] * 4, kNanF32};
  MRA_TRY(debug_fill(fills, stream));

  MRA_TRY(hip_status(mra::launch_pool(q, k, v, qp, kp, vp, kvpacked, s.bh, n, d, (int)dtype, st)));
  for (int l = 0; l <= fin; ++l) {
    float* Sl = const_cast<float*>(T.S[l]);
    if (l < fin) {
      float *ql = f32(W.qp[l]), *kl = f32(W.kp[l]);
      MRA_TRY(hip_status(mra::launch_pool_up(qp, kp, vp, ql, kl, f32(W.vp[l]), s.bh * T.nb[l], d, T.r[l], st)));
      MRA_TRY(hip_status(mra::launch_coarse(ql, kl, Sl, s.bh, T.nb[l], d, st)));
    } else {
      MRA_TRY(hip_status(mra::launch_coarse(qp, kp, Sl, s.bh, nb, d, st)));
    }
    if (l > 0)
      MRA_TRY(hip_status(mra::launch_mask_candidates(Sl, idx[l - 1], s.bh, T.nb[l], T.nb[l - 1],
                                                     T.r[l - 1] / T.r[l], budgets[l - 1], st)));
    if (budgets[l] > 0) MRA_TRY(hip_status(mra::launch_select(Sl, idx[l], s.bh, T.nb[l], budgets[l], st)));
  }
  MRA_TRY(hip_status(mra::launch_coarse_term_levels(T, cmax, csum, cvec, s.bh, d, st)));
  return hip_status(mra::launch_tile(q, k, v, kvpacked, idx[fin], cmax, csum, cvec, out, lse_out, s.bh,
                                     n, d, budgets[fin], (int)dtype, st));
}

}  // namespace

namespace mra {

mra_status_t hip_error_status(hipError_t e) { return hip_status(e); }

mra_status_t forward_check(const void* q, const void* k, const void* v, const void* out,
                           const int32_t* idx_out, const float* lse_out, int B, int H, int n,
                           int d, int block, int budget, mra_dtype_t dtype, size_t* need,
                           bool* empty) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  MRA_TRY(check_dtype(dtype));
  if (budget < 0 || budget > s.nb) return MRA_ERR_INVALID_ARG;
  *empty = s.empty;
  *need = 0;
  if (s.empty) return MRA_OK;
  MRA_TRY(check_ptr(q));
  MRA_TRY(check_ptr(k));
  MRA_TRY(check_ptr(v));
  MRA_TRY(check_ptr(out));
  if (idx_out != nullptr && !aligned16(idx_out)) return MRA_ERR_MISALIGNED;
  if (lse_out != nullptr && !aligned16(lse_out)) return MRA_ERR_MISALIGNED;
  *need = ws_layout(s.bh, s.nb, d, budget, dtype).total;
  return MRA_OK;
}

mra_status_t forward_enqueue(const void* q, const void* k, const void* v, void* out,
                             int32_t* idx_out, float* lse_out, void* workspace, int B, int H,
                             int n, int d, int budget, mra_dtype_t dtype, void* stream) {
  const long long bh = (long long)B * H;
  const int nb = n / kBlockSize;
  const WsLayout L = ws_layout(bh, nb, d, budget, dtype);
  char* ws = static_cast<char*>(workspace);
  float* qp = reinterpret_cast<float*>(ws + L.qp);
  float* kp = reinterpret_cast<float*>(ws + L.kp);
  float* vp = reinterpret_cast<float*>(ws + L.vp);
  void* kvpacked = raw_tiles(d, dtype) ? nullptr : ws + L.kvpacked;
  int32_t* idx = idx_out ? idx_out : reinterpret_cast<int32_t*>(ws + L.idx);
  float* cmax = reinterpret_cast<float*>(ws + L.cmax);
  float* csum = reinterpret_cast<float*>(ws + L.csum);
  float* cvec = reinterpret_cast<float*>(ws + L.cvec);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t elem = dtype == MRA_BF16 ? 2 : 4;
  const Fill fills[4] = {{out, (size_t)bh * n * d * elem, nan_pattern(dtype)},
                         {idx_out, (size_t)bh * nb * budget * 4, kNanF32},
                         {lse_out, (size_t)bh * n * 4, kNanF32},
                         {workspace, L.total, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));

  MRA_TRY(hip_status(launch_pool(q, k, v, qp, kp, vp, kvpacked, bh, n, d, (int)dtype, st)));
  MRA_TRY(hip_status(launch_select_term_fused(qp, kp, idx, vp, cmax, csum, cvec, bh, nb, d, budget,
                                              st)));
  return hip_status(launch_tile(q, k, v, kvpacked, idx, cmax, csum, cvec, out, lse_out, bh, n, d,
                                budget, (int)dtype, st));
}

}  // namespace mra

extern "C" {

mra_status_t mra_pool(const void* q, const void* k, const void* v, float* qp, float* kp,
                      float* vp, int B, int H, int n, int d, int block, mra_dtype_t dtype,
                      void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  MRA_TRY(check_dtype(dtype));
  if ((q == nullptr) != (qp == nullptr) || (k == nullptr) != (kp == nullptr) ||
      (v == nullptr) != (vp == nullptr))
    return MRA_ERR_INVALID_ARG;
  if (q == nullptr && k == nullptr && v == nullptr) return MRA_ERR_INVALID_ARG;
  if (s.empty) return MRA_OK;
  const void* ptrs[6] = {q, k, v, qp, kp, vp};
  for (const void* p : ptrs)
    if (p != nullptr && !aligned16(p)) return MRA_ERR_MISALIGNED;
  const size_t pooled = (size_t)s.bh * s.nb * d * 4;
  const Fill fills[3] = {{qp, pooled, kNanF32}, {kp, pooled, kNanF32}, {vp, pooled, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));
  return hip_status(mra::launch_pool(q, k, v, qp, kp, vp, nullptr, s.bh, n, d, (int)dtype,
                                     static_cast<hipStream_t>(stream)));
}

mra_status_t mra_coarse_scores(const float* qp, const float* kp, float* scores, int B, int H,
                               int n, int d, int block, void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  if (s.empty) return MRA_OK;
  MRA_TRY(check_ptr(qp));
  MRA_TRY(check_ptr(kp));
  MRA_TRY(check_ptr(scores));
  const Fill fills[1] = {{scores, (size_t)s.bh * s.nb * s.nb * 4, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));
  return hip_status(mra::launch_coarse(qp, kp, scores, s.bh, s.nb, d,
                                       static_cast<hipStream_t>(stream)));
}

mra_status_t mra_select(const float* scores, int32_t* idx, int B, int H, int n, int block,
                        int budget, void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, 0, block, false, &s));
  if (budget < 0 || budget > s.nb) return MRA_ERR_INVALID_ARG;
  if (s.empty || budget == 0) return MRA_OK;
  MRA_TRY(check_ptr(scores));
  MRA_TRY(check_ptr(idx));
  const Fill fills[1] = {{idx, (size_t)s.bh * s.nb * budget * 4, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));
  return hip_status(mra::launch_select(scores, idx, s.bh, s.nb, budget,
                                       static_cast<hipStream_t>(stream)));
}

mra_status_t mra_coarse_term(const float* scores, const int32_t* idx, const float* vp,
                             float* cmax, float* csum, float* cvec, int B, int H, int n, int d,
                             int block, int budget, void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  if (budget < 0 || budget > s.nb) return MRA_ERR_INVALID_ARG;
  if (s.empty) return MRA_OK;
  MRA_TRY(check_ptr(scores));
  if (budget > 0) MRA_TRY(check_ptr(idx));
  MRA_TRY(check_ptr(vp));
  MRA_TRY(check_ptr(cmax));
  MRA_TRY(check_ptr(csum));
  MRA_TRY(check_ptr(cvec));
  const Fill fills[3] = {{cmax, (size_t)s.bh * s.nb * 4, kNanF32},
                         {csum, (size_t)s.bh * s.nb * 4, kNanF32},
                         {cvec, (size_t)s.bh * s.nb * d * 4, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));
  return hip_status(mra::launch_coarse_term(scores, idx, vp, cmax, csum, cvec, s.bh, s.nb, d,
                                            budget, static_cast<hipStream_t>(stream)));
}

mra_status_t mra_block_sddmm_spmm(const void* q, const void* k, const void* v,
                                  const int32_t* idx, const float* cmax, const float* csum,
                                  const float* cvec, void* out, float* lse_out, int B, int H,
                                  int n, int d, int block, int budget, mra_dtype_t dtype,
                                  void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  MRA_TRY(check_dtype(dtype));
  if (budget < 0 || budget > s.nb) return MRA_ERR_INVALID_ARG;
  const int given = (cmax != nullptr) + (csum != nullptr) + (cvec != nullptr);
  if (given != 0 && given != 3) return MRA_ERR_INVALID_ARG;
  if (given == 0 && budget == 0) return MRA_ERR_INVALID_ARG;   // nothing to normalise
  if (s.empty) return MRA_OK;
  MRA_TRY(check_ptr(q));
  MRA_TRY(check_ptr(k));
  MRA_TRY(check_ptr(v));
  MRA_TRY(check_ptr(out));
  if (lse_out != nullptr && !aligned16(lse_out)) return MRA_ERR_MISALIGNED;
  if (budget > 0) MRA_TRY(check_ptr(idx));
  if (given) {
    MRA_TRY(check_ptr(cmax));
    MRA_TRY(check_ptr(csum));
    MRA_TRY(check_ptr(cvec));
  }
  const Fill fills[2] = {{out, (size_t)s.bh * n * d * (dtype == MRA_BF16 ? 2 : 4), nan_pattern(dtype)},
                         {lse_out, (size_t)s.bh * n * 4, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));
  return hip_status(mra::launch_tile(q, k, v, nullptr, idx, cmax, csum, cvec, out, lse_out, s.bh,
                                     n, d, budget, (int)dtype, static_cast<hipStream_t>(stream)));
}

size_t mra_forward_workspace_bytes(int B, int H, int n, int d, int block, int budget,
                                   mra_dtype_t dtype) {
  Shape s;
  if (check_shape(B, H, n, d, block, true, &s) != MRA_OK) return 0;
  if (check_dtype(dtype) != MRA_OK) return 0;
  if (budget < 0 || budget > s.nb) return 0;
  return ws_layout(s.bh, s.nb, d, budget, dtype).total;
}

mra_status_t mra_attention_forward(const void* q, const void* k, const void* v, void* out,
                                   int32_t* idx_out, float* lse_out, void* workspace,
                                   size_t workspace_bytes,
                                   int B, int H, int n, int d, int block, int budget,
                                   mra_dtype_t dtype, void* stream) {
  size_t need = 0;
  bool empty = true;
  MRA_TRY(mra::forward_check(q, k, v, out, idx_out, lse_out, B, H, n, d, block, budget, dtype, &need,
                             &empty));
  if (empty) return MRA_OK;
  MRA_TRY(check_ptr(workspace));
  if (workspace_bytes < need) return MRA_ERR_WORKSPACE;
  return mra::forward_enqueue(q, k, v, out, idx_out, lse_out, workspace, B, H, n, d, budget, dtype,
                              stream);
}

mra_status_t mra_sparse_attention_forward(const void* q, const void* k, const void* v,
                                          void* out, int32_t* idx_out, float* lse_out,
                                          void* workspace,
                                          size_t workspace_bytes, int B, int H, int n, int d,
                                          int block, int budget, mra_dtype_t dtype,
                                          void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  MRA_TRY(check_dtype(dtype));
  // at least one selected block per row (n = 0 leaves no block to select)
  if (budget < 0 || budget > s.nb || (s.nb > 0 && budget < 1)) return MRA_ERR_INVALID_ARG;
  if (s.empty) return MRA_OK;
  MRA_TRY(check_ptr(q));
  MRA_TRY(check_ptr(k));
  MRA_TRY(check_ptr(v));
  MRA_TRY(check_ptr(out));
  if (idx_out != nullptr && !aligned16(idx_out)) return MRA_ERR_MISALIGNED;
  if (lse_out != nullptr && !aligned16(lse_out)) return MRA_ERR_MISALIGNED;
  MRA_TRY(check_ptr(workspace));
  const WsLayout L = ws_layout(s.bh, s.nb, d, budget, dtype);
  if (workspace_bytes < L.total) return MRA_ERR_WORKSPACE;

  char* ws = static_cast<char*>(workspace);
  float* qp = reinterpret_cast<float*>(ws + L.qp);
  float* kp = reinterpret_cast<float*>(ws + L.kp);
  float* vp = reinterpret_cast<float*>(ws + L.vp);
  void* kvpacked = raw_tiles(d, dtype) ? nullptr : ws + L.kvpacked;
  int32_t* idx = idx_out ? idx_out : reinterpret_cast<int32_t*>(ws + L.idx);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const Fill fills[4] = {{out, (size_t)s.bh * n * d * (dtype == MRA_BF16 ? 2 : 4), nan_pattern(dtype)},
                         {idx_out, (size_t)s.bh * s.nb * budget * 4, kNanF32},
                         {lse_out, (size_t)s.bh * n * 4, kNanF32},
                         {workspace, L.total, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));

  MRA_TRY(hip_status(mra::launch_pool(q, k, v, qp, kp, vp, kvpacked, s.bh, n, d, (int)dtype, st)));
  MRA_TRY(hip_status(mra::launch_select_fused(qp, kp, idx, s.bh, s.nb, d, budget, st)));
  return hip_status(mra::launch_tile(q, k, v, kvpacked, idx, nullptr, nullptr, nullptr, out,
                                     lse_out, s.bh, n, d, budget, (int)dtype, st));
}

mra_status_t mra_select_global(const float* scores, int32_t* idx, int B, int H, int n,
                               int block, int budget, int prior_diagonal, void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, 0, block, false, &s));
  MRA_TRY(check_global_budget(s, budget, prior_diagonal));
  if (s.empty) return MRA_OK;
  MRA_TRY(check_ptr(scores));
  MRA_TRY(check_ptr(idx));
  const Fill fills[1] = {{idx, (size_t)s.bh * s.nb * s.nb * 4, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));
  return hip_status(mra::launch_select_global(scores, idx, s.bh, s.nb, budget, prior_diagonal,
                                              static_cast<hipStream_t>(stream)));
}

size_t mra_forward_global_workspace_bytes(int B, int H, int n, int d, int block,
                                          mra_dtype_t dtype) {
  Shape s;
  if (check_shape(B, H, n, d, block, true, &s) != MRA_OK) return 0;
  if (check_dtype(dtype) != MRA_OK) return 0;
  return ws_global(s.bh, s.nb, d, dtype).total;
}

mra_status_t mra_attention_forward_global(const void* q, const void* k, const void* v,
                                          void* out, int32_t* idx_out, float* lse_out,
                                          void* workspace,
                                          size_t workspace_bytes, int B, int H, int n, int d,
                                          int block, int budget, int prior_diagonal,
                                          mra_dtype_t dtype, void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  MRA_TRY(check_dtype(dtype));
  MRA_TRY(check_global_budget(s, budget, prior_diagonal));
  if (s.empty) return MRA_OK;
  MRA_TRY(check_ptr(q));
  MRA_TRY(check_ptr(k));
  MRA_TRY(check_ptr(v));
  MRA_TRY(check_ptr(out));
  if (idx_out != nullptr && !aligned16(idx_out)) return MRA_ERR_MISALIGNED;
  if (lse_out != nullptr && !aligned16(lse_out)) return MRA_ERR_MISALIGNED;
  MRA_TRY(check_ptr(workspace));
  const WsGlobal G = ws_global(s.bh, s.nb, d, dtype);
  if (workspace_bytes < G.total) return MRA_ERR_WORKSPACE;

  char* ws = static_cast<char*>(workspace);
  const WsLayout& L = G.base;
  float* qp = reinterpret_cast<float*>(ws + L.qp);
  float* kp = reinterpret_cast<float*>(ws + L.kp);
  float* vp = reinterpret_cast<float*>(ws + L.vp);
  void* kvpacked = raw_tiles(d, dtype) ? nullptr : ws + L.kvpacked;
  int32_t* idx = idx_out ? idx_out : reinterpret_cast<int32_t*>(ws + L.idx);
  float* cmax = reinterpret_cast<float*>(ws + L.cmax);
  float* csum = reinterpret_cast<float*>(ws + L.csum);
  float* cvec = reinterpret_cast<float*>(ws + L.cvec);
  float* S = reinterpret_cast<float*>(ws + G.scores);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int nb = s.nb;
  const Fill fills[4] = {{out, (size_t)s.bh * n * d * (dtype == MRA_BF16 ? 2 : 4), nan_pattern(dtype)},
                         {idx_out, (size_t)s.bh * nb * nb * 4, kNanF32},
                         {lse_out, (size_t)s.bh * n * 4, kNanF32},
                         {workspace, G.total, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));

  MRA_TRY(hip_status(mra::launch_pool(q, k, v, qp, kp, vp, kvpacked, s.bh, n, d, (int)dtype, st)));
  MRA_TRY(hip_status(mra::launch_coarse(qp, kp, S, s.bh, nb, d, st)));
  MRA_TRY(hip_status(mra::launch_select_global(S, idx, s.bh, nb, budget, prior_diagonal, st)));
  MRA_TRY(hip_status(mra::launch_coarse_term(S, idx, vp, cmax, csum, cvec, s.bh, nb, d, nb, st)));
  return hip_status(mra::launch_tile(q, k, v, kvpacked, idx, cmax, csum, cvec, out, lse_out, s.bh,
                                     n, d, nb, (int)dtype, st));
}

size_t mra_backward_workspace_bytes(int B, int H, int n, int d, int block, mra_dtype_t dtype) {
  Shape s;
  if (check_shape(B, H, n, d, block, true, &s) != MRA_OK) return 0;
  if (check_dtype(dtype) != MRA_OK) return 0;
  return ws_bwd(s.bh, s.nb, d, dtype).total;
}

// The backward of mra_attention_backward(_pooled): with `given`, pq, pk, pv
// are the block means of q, k, v, supplied by the caller. (Internal linkage:
// only the mra_ entry points are exported.)
static mra_status_t backward(const void* q, const void* k, const void* v, const void* out,
                      const void* dout, const float* lse, const int32_t* idx, bool given,
                      const float* pq, const float* pk, const float* pv, void* dq, void* dk,
                      void* dv, void* workspace, size_t workspace_bytes, int B, int H, int n,
                      int d, int block, int width, int coarse, mra_dtype_t dtype, void* stream) {
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  MRA_TRY(check_dtype(dtype));
  if (width < 0 || width > s.nb) return MRA_ERR_INVALID_ARG;
  if (coarse != 0 && coarse != 1) return MRA_ERR_INVALID_ARG;
  if (s.empty) return MRA_OK;
  const void* in[7] = {q, k, v, out, dout, lse, workspace};
  for (const void* p : in) MRA_TRY(check_ptr(p));
  if (width > 0) MRA_TRY(check_ptr(idx));
  MRA_TRY(check_ptr(dq));
  MRA_TRY(check_ptr(dk));
  MRA_TRY(check_ptr(dv));
  if (given) {
    MRA_TRY(check_ptr(pq));
    MRA_TRY(check_ptr(pk));
    MRA_TRY(check_ptr(pv));
  }
  const WsBwd L = ws_bwd(s.bh, s.nb, d, dtype);
  if (workspace_bytes < L.total) return MRA_ERR_WORKSPACE;

  char* ws = static_cast<char*>(workspace);
  auto f32 = [&](size_t off) { return reinterpret_cast<float*>(ws + off); };
  mra::BwdArgs A{};
  A.q = q; A.k = k; A.v = v; A.out = out; A.dout = dout;
  A.lse = lse; A.idx = idx;
  A.dq = dq; A.dk = dk; A.dv = dv;
  A.bh = s.bh; A.n = n; A.d = d; A.m = width; A.dtype = (int)dtype; A.coarse = coarse != 0;
  A.qp = f32(L.qp); A.kp = f32(L.kp); A.vp = f32(L.vp);
  A.pooled_in = given && coarse != 0;
  if (A.pooled_in) {                                        // read only by the kernels
    A.qp = const_cast<float*>(pq);
    A.kp = const_cast<float*>(pk);
    A.vp = const_cast<float*>(pv);
  }
  A.q_row = ws + L.q_row; A.q_t = ws + L.q_t; A.k_row = ws + L.k_row; A.k_t = ws + L.k_t;
  A.v_row = ws + L.v_row; A.g_row = ws + L.g_row; A.g_t = ws + L.g_t;
  A.ld = f32(L.ld);
  A.bias = dtype == MRA_BF16 ? reinterpret_cast<uint32_t*>(ws + L.bias) : nullptr;
  A.bits = reinterpret_cast<uint32_t*>(ws + L.bits);
  A.gh = f32(L.gh); A.W = f32(L.W); A.dS = f32(L.dS);
  A.dqp = f32(L.dqp); A.dkp = f32(L.dkp); A.dvp = f32(L.dvp);
  const size_t gbytes = (size_t)s.bh * n * d * (dtype == MRA_BF16 ? 2 : 4);
  const Fill fills[4] = {{dq, gbytes, nan_pattern(dtype)}, {dk, gbytes, nan_pattern(dtype)},
                         {dv, gbytes, nan_pattern(dtype)}, {workspace, L.total, kNanF32}};
  MRA_TRY(debug_fill(fills, stream));
  return hip_status(mra::launch_bwd(A, static_cast<hipStream_t>(stream)));
}

mra_status_t mra_attention_backward(const void* q, const void* k, const void* v, const void* out,
                                    const void* dout, const float* lse, const int32_t* idx,
                                    void* dq, void* dk, void* dv, void* workspace,
                                    size_t workspace_bytes, int B, int H, int n, int d, int block,
                                    int width, int coarse, mra_dtype_t dtype, void* stream) {
  return backward(q, k, v, out, dout, lse, idx, false, nullptr, nullptr, nullptr, dq, dk, dv,
                  workspace, workspace_bytes, B, H, n, d, block, width, coarse, dtype, stream);
}

mra_status_t mra_attention_backward_pooled(const void* q, const void* k, const void* v,
                                           const void* out, const void* dout, const float* lse,
                                           const int32_t* idx, const float* qp, const float* kp,
                                           const float* vp, void* dq, void* dk, void* dv,
                                           void* workspace, size_t workspace_bytes, int B, int H,
                                           int n, int d, int block, int width, int coarse,
                                           mra_dtype_t dtype, void* stream) {
  return backward(q, k, v, out, dout, lse, idx, true, qp, kp, vp, dq, dk, dv, workspace,
                  workspace_bytes, B, H, n, d, block, width, coarse, dtype, stream);
}

mra_status_t mra_forward_pooled_rows(const void* workspace, int B, int H, int n, int d, int block,
                                     const float** qp, const float** kp, const float** vp) {
  if (qp == nullptr || kp == nullptr || vp == nullptr) return MRA_ERR_INVALID_ARG;
  *qp = *kp = *vp = nullptr;
  Shape s;
  MRA_TRY(check_shape(B, H, n, d, block, true, &s));
  if (s.empty) return MRA_OK;
  MRA_TRY(check_ptr(workspace));
  // Q~, K~, V~ lead the forward's layout (and the head-wide-budget forward's,
  // which extends it); their offsets depend on neither budget nor dtype
  const WsLayout L = ws_layout(s.bh, s.nb, d, 0, MRA_BF16);
  const char* ws = static_cast<const char*>(workspace);
  *qp = reinterpret_cast<const float*>(ws + L.qp);
  *kp = reinterpret_cast<const float*>(ws + L.kp);
  *vp = reinterpret_cast<const float*>(ws + L.vp);
  return MRA_OK;
}

size_t mra_forward_multilevel_workspace_bytes(int B, int H, int n, int d, int block,
                                              int coarse_block, int budget1, int budget2,
                                              mra_dtype_t dtype) {
  const int scales[2] = {coarse_block, kBlockSize}, budgets[2] = {budget1, budget2};
  return levels_workspace_bytes(B, H, n, d, block, 2, scales, budgets, dtype);
}

mra_status_t mra_attention_forward_multilevel(const void* q, const void* k, const void* v,
                                              void* out, int32_t* idx1_out, int32_t* idx2_out,
                                              float* lse_out, void* workspace,
                                              size_t workspace_bytes, int B, int H, int n, int d,
                                              int block, int coarse_block, int budget1,
                                              int budget2, mra_dtype_t dtype, void* stream) {
  const int scales[2] = {coarse_block, kBlockSize}, budgets[2] = {budget1, budget2};
  int32_t* const outs[2] = {idx1_out, idx2_out};
  return levels_forward(q, k, v, out, outs, lse_out, workspace, workspace_bytes, B, H, n, d, block,
                        2, scales, budgets, dtype, stream);
}

size_t mra_forward_levels_workspace_bytes(int B, int H, int n, int d, int block, int levels,
                                          const int* scales, const int* budgets,
                                          mra_dtype_t dtype) {
  return levels_workspace_bytes(B, H, n, d, block, levels, scales, budgets, dtype);
}

mra_status_t mra_attention_forward_levels(const void* q, const void* k, const void* v, void* out,
                                          int32_t* const* idx_outs, float* lse_out,
                                          void* workspace, size_t workspace_bytes, int B, int H,
                                          int n, int d, int block, int levels, const int* scales,
                                          const int* budgets, mra_dtype_t dtype, void* stream) {
  return levels_forward(q, k, v, out, idx_outs, lse_out, workspace, workspace_bytes, B, H, n, d,
                        block, levels, scales, budgets, dtype, stream);
}

const char* mra_status_str(mra_status_t status) {
  switch (status) {
    case MRA_OK: return "MRA_OK";
    case MRA_ERR_INVALID_ARG: return "MRA_ERR_INVALID_ARG: invalid argument";
    case MRA_ERR_UNSUPPORTED: return "MRA_ERR_UNSUPPORTED: unsupported block, head dim, length or dtype";
    case MRA_ERR_MISALIGNED: return "MRA_ERR_MISALIGNED: pointer not 16-byte aligned";
    case MRA_ERR_WORKSPACE: return "MRA_ERR_WORKSPACE: workspace too small";
    case MRA_ERR_HIP: return "MRA_ERR_HIP: HIP launch failed";
    case MRA_ERR_SCRATCH: return "MRA_ERR_SCRATCH: problem needs more than the static scratch of mra_attention_forward_noalloc";
  }
  return "unknown mra_status_t";
}

int mra_last_hip_error(void) { return g_last_hip_error; }

}  // extern "C"
