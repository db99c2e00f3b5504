// High-resolution part of MRA-2 and the output (Sec. 4.2 eq.
// actual_approx_mat_form with mu_{1,i,j} = exp(P_ij); Sec. 4.3 Alg. 2 at
// scale 1; Sec. 3.1 row normalisation D^).
//
// One wave owns one block-row x (32 queries). For every selected column block
// y it computes the 32x32 tile S = c Q_x K_y^T on the matrix cores
// (block-sparse SDDMM), folds it into a running max / row sum (online
// softmax), and accumulates P V_y (block-sparse SpMM). At the end the result
// is merged with the block-row's low-resolution term (M_x, c_x, L_x) and
// normalised.
//
// Matrix-core layout (v_mfma_f32_32x32x16_bf16; 32x32x2_f32 for float32):
//  * S is formed transposed, S^T = K_y Q_x^T, so lane l holds query l%32 and
//    16 of its 32 key scores (keys 8(r/4) + 4(l/32) + r%4 in register r).
//    That is already the B-operand layout of O^T += V_y^T P^T up to a fixed
//    permutation of the key index, so P never moves between lanes; only the
//    row max crosses the two half-waves.
//  * The contraction index over d is permuted too: lane half h = l/32 takes
//    the contiguous half [h*d/2, (h+1)*d/2) of each Q and K row, so every lane
//    streams d bytes (bf16) of one row with 16-byte loads.
//  * With the packed copies of K and V written by the pooling pass, every
//    operand load (K_y, and V_y^T, the A operand of the second product) is
//    one 16-byte chunk per lane, 1 KB contiguous per wave: no LDS, no
//    shuffles. For raw K/V, K_y rows are read directly and V_y goes through a
//    wave-private LDS tile stored transposed with the key permutation applied.
// With packed K/V the next tile's loads are in flight while the current one is
// computed. O is rescaled only when some query's running max grew a lot.
// Workgroups of 4 waves take 4 consecutive block-rows; the workgroup order is
// remapped so each XCD processes a contiguous range of heads and keeps their
// K/V tiles in its L2.
#include "common.h"
#include "kernels.h"

namespace mra {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <int DT, int D>
struct TileCfg {
  static constexpr int kWaves = (DT == F32 && D == 128) ? 2 : 4;
  static constexpr int kPitch = DT == BF16 ? 40 : 36;           // LDS row pitch, elements
  static constexpr int kNT = D / 32;                            // output tiles over d
  // 16-byte V operand chunks per lane per tile
  static constexpr int kVChunks = DT == BF16 ? 2 * kNT : 4 * kNT;
  static constexpr int kKChunks = DT == BF16 ? D / 16 : D / 8;  // 16-byte K chunks per lane
  using elem = typename std::conditional<DT == BF16, uint16_t, float>::type;
};

// Running max of the scores (log2 units) for the online softmax. The max is
// refreshed, and O and the row sums rescaled, only when some query's tile max
// exceeds the current one by more than kLazy (log2 units): in between, the
// weights exp2(s - mrun) stay below 2^kLazy, far inside float32 and bfloat16
// range, and the final normalisation uses the same mrun, so the result is the
// same softmax. Lanes l and l^32 share a query.
constexpr float kLazy = 8.0f;

template <int NT>
__device__ __forceinline__ void rescale_if_grown(float mx, float sl2, float& mrun, float& lrun,
                                                 f32x16 (&o)[NT]) {
  mx = halves_max(mx);
  const float cand = mx * sl2;
  if (__ballot(cand > mrun + kLazy)) {             // wave-uniform, rarely taken
    // keeps the compiler from turning this branch into an unconditional
    // multiply of every accumulator by a selected factor
    asm volatile("; mra rescale" ::: "memory");
    const float mnew = __builtin_elementwise_maximum(mrun, cand);
    const float alpha = __builtin_amdgcn_exp2f(mrun - mnew);   // 0 at the first tile
    lrun *= alpha;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
    mrun = mnew;
  }
}

__device__ __forceinline__ float tile_max(const f32x16& s) {
  float a = s[0];
#pragma unroll
  for (int r = 1; r < 16; ++r) a = __builtin_elementwise_maximum(a, s[r]);
  return a;
}

template <int DT, int D, bool COARSE, bool PACKED>
__global__ __launch_bounds__((TileCfg<DT, D>::kWaves * kWave)) void tile_kernel(
    const void* __restrict__ qv, const void* __restrict__ kv, const void* __restrict__ vv,
    const int32_t* __restrict__ idx, const float* __restrict__ cmax,
    const float* __restrict__ csum, const float* __restrict__ cvec, void* __restrict__ outv,
    int n, int nb, int m, long long rows, float scale_log2) {
  using Cfg = TileCfg<DT, D>;
  using elem = typename Cfg::elem;
  constexpr int W = Cfg::kWaves, PITCH = Cfg::kPitch, NT = Cfg::kNT;
  constexpr int VC = Cfg::kVChunks, KC = Cfg::kKChunks;
  __shared__ __attribute__((aligned(16))) elem vt_all[PACKED ? 1 : W][PACKED ? 8 : D * PITCH];

  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id();
  const int jq = lane & 31, h = lane >> 5;
  const long long wg = xcd_remap(blockIdx.x, gridDim.x);
  const long long g = wg * W + w;                    // global block-row
  if (g >= rows) return;                             // no workgroup barriers below
  const long long bh = g / nb;
  const int x = (int)(g - bh * nb);
  const long long hoff = bh * (long long)n * D;
  const elem* Q = reinterpret_cast<const elem*>(qv) + hoff;
  const elem* K = reinterpret_cast<const elem*>(kv) + hoff;
  elem* Out = reinterpret_cast<elem*>(outv) + hoff;
  const float sl2 = scale_log2;
  // The row's selection, staged once in LDS: reading block ids from LDS keeps
  // them off the vector-memory counter, so prefetched K/V loads stay in flight.
  extern __shared__ int32_t sidx_all[];
  int32_t* myidx = sidx_all + w * m;
  for (int i = lane; i < m; i += kWave) myidx[i] = idx[g * m + i];
  wave_lds_sync();

  f32x16 o[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  float mrun = -INFINITY, lrun = 0.0f;

  // Q_x as the B operand, K_y as the A operand: lane reads d/2 contiguous
  // elements of one row, 16 bytes at a time.
  u32x4 qf[KC];
  {
    const u32x4* qrow = reinterpret_cast<const u32x4*>(Q + (long long)(x * 32 + jq) * D + (D / 2) * h);
#pragma unroll
    for (int s = 0; s < KC; ++s) qf[s] = qrow[s];
  }
  auto load_k = [&](int y, u32x4 (&kf)[KC]) {
    const u32x4* krow = reinterpret_cast<const u32x4*>(K + (long long)(y * 32 + jq) * D + (D / 2) * h);
#pragma unroll
    for (int s = 0; s < KC; ++s) kf[s] = krow[s];
  };
  // packed K/V (see kernels.h): every operand load is 1 KB contiguous per wave
  auto load_kpacked = [&](int y, u32x4 (&kf)[KC]) {
    const u32x4* kt = reinterpret_cast<const u32x4*>(kv) + ((bh * nb + y) * KC) * 64 + lane;
#pragma unroll
    for (int c = 0; c < KC; ++c) kf[c] = kt[c * 64];
  };
  auto load_vpacked = [&](int y, u32x4 (&vf)[VC]) {
    const u32x4* vt = reinterpret_cast<const u32x4*>(vv) + ((bh * nb + y) * VC) * 64 + lane;
#pragma unroll
    for (int c = 0; c < VC; ++c) vf[c] = vt[c * 64];
  };
  // S^T = K_y Q_x^T
  auto scores = [&](const u32x4 (&kf)[KC]) {
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.0f;
    if constexpr (DT == BF16) {
#pragma unroll
      for (int k = 0; k < KC; ++k)
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf[k]),
                                                    __builtin_bit_cast(bf16x8, qf[k]), s, 0, 0, 0);
    } else {
#pragma unroll
      for (int k = 0; k < KC; ++k)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          s = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(kf[k][e]), __uint_as_float(qf[k][e]), s, 0, 0, 0);
    }
    return s;
  };
  // Softmax weights of one tile and O^T += V_y^T P^T. `va(c)` yields the
  // 16-byte A-operand chunk c of V_y^T for this lane. The matrix-core
  // instructions always run (they consume the tile's loads on every path, which
  // keeps the compiler's load-counter waits tight); a skipped block only
  // zeroes P, inside a branch that holds no memory operations.
  auto accumulate = [&](const f32x16& s, bool use, auto va) {
    if constexpr (DT == BF16) {
      uint32_t pk[8];
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) pk[rr] = 0u;
      if (use) {
        rescale_if_grown<NT>(tile_max(s), sl2, mrun, lrun, o);
        const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
        for (int rr = 0; rr < 8; ++rr) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(s[2 * rr], sl2, -mrun));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(s[2 * rr + 1], sl2, -mrun));
          bf16x2 pb;
          pb[0] = (__bf16)p0;
          pb[1] = (__bf16)p1;
          lrun = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, lrun, false);   // sum of the rounded P
          pk[rr] = __builtin_bit_cast(uint32_t, pb);
        }
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const u32x4 pw = {pk[4 * u], pk[4 * u + 1], pk[4 * u + 2], pk[4 * u + 3]};
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
        for (int t = 0; t < NT; ++t)
          o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, va(u * NT + t)), pb, o[t], 0, 0, 0);
      }
    } else {
      float p[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) p[r] = 0.0f;
      if (use) {
        rescale_if_grown<NT>(tile_max(s), sl2, mrun, lrun, o);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          p[r] = __builtin_amdgcn_exp2f(fmaf(s[r], sl2, -mrun));
          lrun += p[r];
        }
      }
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const u32x4 v4 = va(t * 4 + a);
#pragma unroll
          for (int e = 0; e < 4; ++e)
            o[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(v4[e]), p[4 * a + e], o[t], 0, 0, 0);
        }
    }
  };
  auto clampy = [&](int y) { return (y < 0 || y >= nb) ? 0 : y; };

  if constexpr (PACKED) {
    // Two register buffers: tile i+1 loads while tile i is computed. Loads
    // are issued unconditionally (past the last tile they re-read the last
    // tile, a cache hit) so every path leaves the same loads in flight.
    u32x4 kA[KC], vA[VC], kB[KC], vB[VC];
    auto valid = [&](int y) { return y >= 0 && y < nb; };
    if (m > 0) {
      const int y0 = clampy(wave_uniform(myidx[0]));
      load_kpacked(y0, kA);
      load_vpacked(y0, vA);
    }
    for (int i = 0; i < m; i += 2) {
      const int ya = wave_uniform(myidx[i]);
      const int yb = wave_uniform(myidx[min(i + 1, m - 1)]);
      load_kpacked(clampy(yb), kB);
      load_vpacked(clampy(yb), vB);
      accumulate(scores(kA), valid(ya), [&](int c) { return vA[c]; });
      if (i + 1 >= m) break;
      const int yc = clampy(wave_uniform(myidx[min(i + 2, m - 1)]));
      load_kpacked(yc, kA);
      load_vpacked(yc, vA);
      accumulate(scores(kB), valid(yb), [&](int c) { return vB[c]; });
    }
  } else {
    elem* vt = vt_all[w];
    const elem* V = reinterpret_cast<const elem*>(vv) + hoff;
    for (int i = 0; i < m; ++i) {
      const int y = wave_uniform(myidx[i]);
      if (y < 0 || y >= nb) continue;
      u32x4 kc[KC];
      load_k(y, kc);
      // V_y -> LDS transposed, keys in the operand order of the packed layout
      if constexpr (DT == BF16) {
        // key 16u + 8a + 4hh + kk goes to position 16u + 8hh + 4a + kk
#pragma unroll
        for (int gi = lane; gi < D; gi += kWave) {
          const int c = gi % (D / 8), kg = gi / (D / 8);
          const elem* vsrc = V + (long long)(y * 32 + 4 * kg) * D + 8 * c;
          const u32x4 r0 = *reinterpret_cast<const u32x4*>(vsrc);
          const u32x4 r1 = *reinterpret_cast<const u32x4*>(vsrc + D);
          const u32x4 r2 = *reinterpret_cast<const u32x4*>(vsrc + 2 * D);
          const u32x4 r3 = *reinterpret_cast<const u32x4*>(vsrc + 3 * D);
          const int pos0 = 16 * (kg >> 2) + 8 * (kg & 1) + 4 * ((kg >> 1) & 1);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int sh = (e & 1) * 16;
            u32x2 pr;
            pr[0] = ((r0[e >> 1] >> sh) & 0xFFFFu) | (((r1[e >> 1] >> sh) & 0xFFFFu) << 16);
            pr[1] = ((r2[e >> 1] >> sh) & 0xFFFFu) | (((r3[e >> 1] >> sh) & 0xFFFFu) << 16);
            *reinterpret_cast<u32x2*>(vt + (8 * c + e) * PITCH + pos0) = pr;
          }
        }
      } else {
        // key 8a + 4hh + kk goes to position 16hh + 4a + kk
#pragma unroll
        for (int gi = lane; gi < 2 * D; gi += kWave) {
          const int c = gi % (D / 4), kg = gi / (D / 4);
          const float* vsrc = V + (long long)(y * 32 + 4 * kg) * D + 4 * c;
          const f32x4 r0 = *reinterpret_cast<const f32x4*>(vsrc);
          const f32x4 r1 = *reinterpret_cast<const f32x4*>(vsrc + D);
          const f32x4 r2 = *reinterpret_cast<const f32x4*>(vsrc + 2 * D);
          const f32x4 r3 = *reinterpret_cast<const f32x4*>(vsrc + 3 * D);
          const int pos0 = 16 * (kg & 1) + 4 * (kg >> 1);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const f32x4 col = {r0[e], r1[e], r2[e], r3[e]};
            *reinterpret_cast<f32x4*>(vt + (4 * c + e) * PITCH + pos0) = col;
          }
        }
      }
      const f32x16 s = scores(kc);
      wave_lds_sync();
      if constexpr (DT == BF16) {
        accumulate(s, true, [&](int c) {
          const int u = c / NT, t = c % NT;
          return *reinterpret_cast<const u32x4*>(vt + (32 * t + jq) * PITCH + 16 * u + 8 * h);
        });
      } else {
        accumulate(s, true, [&](int c) {
          const int t = c / 4, a = c % 4;
          return *reinterpret_cast<const u32x4*>(vt + (32 * t + jq) * PITCH + 16 * h + 4 * a);
        });
      }
      wave_lds_sync();                               // reads done before the next overwrite
    }
  }

  // ---- merge with the low-resolution term and normalise
  const float ltot = halves_sum(lrun);
  float af = 1.0f, bc = 0.0f, den = ltot;
  if constexpr (COARSE) {
    const float Mx = cmax[g] * kLog2e;
    const float Mt = fmaxf(mrun, Mx);
    af = exp2f(mrun - Mt);
    bc = exp2f(Mx - Mt);
    den = ltot * af + csum[g] * bc;
  }
  const float inv = 1.0f / den;
  elem* orow = Out + (long long)(x * 32 + jq) * D;
  const float* cv = COARSE ? cvec + g * D : nullptr;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int d0 = 32 * t + 8 * rg + 4 * h;
      float z[4];
      f32x4 c4 = {0.0f, 0.0f, 0.0f, 0.0f};
      if constexpr (COARSE) c4 = *reinterpret_cast<const f32x4*>(cv + d0);
#pragma unroll
      for (int e = 0; e < 4; ++e) z[e] = (o[t][4 * rg + e] * af + c4[e] * bc) * inv;
      if constexpr (DT == BF16) {
        bf16x2 lo, hi;
        lo[0] = (__bf16)z[0]; lo[1] = (__bf16)z[1];
        hi[0] = (__bf16)z[2]; hi[1] = (__bf16)z[3];
        const u32x2 pr = {__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
        *reinterpret_cast<u32x2*>(orow + d0) = pr;
      } else {
        const f32x4 st = {z[0], z[1], z[2], z[3]};
        *reinterpret_cast<f32x4*>(orow + d0) = st;
      }
    }
  }
}

template <int DT, int D, bool PACKED>
static void launch_tile_t(const void* q, const void* k, const void* v, const int32_t* idx,
                          const float* cmax, const float* csum, const float* cvec, void* out,
                          long long bh, int n, int m, hipStream_t stream) {
  constexpr int W = TileCfg<DT, D>::kWaves;
  const int nb = n / kBlock;
  const long long rows = bh * nb;
  const unsigned blocks = (unsigned)((rows + W - 1) / W);
  const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
  const size_t smem = (size_t)W * m * sizeof(int32_t);     // per-wave selection lists
  if (cmax)
    tile_kernel<DT, D, true, PACKED><<<blocks, W * kWave, smem, stream>>>(q, k, v, idx, cmax, csum, cvec, out, n, nb, m, rows, scale_log2);
  else
    tile_kernel<DT, D, false, PACKED><<<blocks, W * kWave, smem, stream>>>(q, k, v, idx, cmax, csum, cvec, out, n, nb, m, rows, scale_log2);
}

template <bool PACKED>
static void launch_tile_p(const void* q, const void* k, const void* v, const int32_t* idx,
                          const float* cmax, const float* csum, const float* cvec, void* out,
                          long long bh, int n, int d, int m, int dtype, hipStream_t stream) {
  if (dtype == BF16) {
    if (d == 32) launch_tile_t<BF16, 32, PACKED>(q, k, v, idx, cmax, csum, cvec, out, bh, n, m, stream);
    else if (d == 64) launch_tile_t<BF16, 64, PACKED>(q, k, v, idx, cmax, csum, cvec, out, bh, n, m, stream);
    else launch_tile_t<BF16, 128, PACKED>(q, k, v, idx, cmax, csum, cvec, out, bh, n, m, stream);
  } else {
    if (d == 32) launch_tile_t<F32, 32, PACKED>(q, k, v, idx, cmax, csum, cvec, out, bh, n, m, stream);
    else if (d == 64) launch_tile_t<F32, 64, PACKED>(q, k, v, idx, cmax, csum, cvec, out, bh, n, m, stream);
    else launch_tile_t<F32, 128, PACKED>(q, k, v, idx, cmax, csum, cvec, out, bh, n, m, stream);
  }
}

hipError_t launch_tile(const void* q, const void* k, const void* v, const void* kvpacked,
                       const int32_t* idx, const float* cmax, const float* csum,
                       const float* cvec, void* out, long long bh, int n, int d, int m, int dtype,
                       hipStream_t stream) {
  if (kvpacked) {
    const size_t half = (size_t)bh * n * d * (dtype == BF16 ? 2 : 4);
    const void* kpk = kvpacked;
    const void* vpk = static_cast<const char*>(kvpacked) + half;
    launch_tile_p<true>(q, kpk, vpk, idx, cmax, csum, cvec, out, bh, n, d, m, dtype, stream);
  } else {
    launch_tile_p<false>(q, k, v, idx, cmax, csum, cvec, out, bh, n, d, m, dtype, stream);
  }
  return hipGetLastError();
}

}  // namespace mra
