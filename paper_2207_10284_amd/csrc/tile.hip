// High-resolution part of MRA-2 and the output (Sec. 4.2 eq.
// actual_approx_mat_form with mu_{1,i,j} = exp(P_ij); Sec. 4.3 Alg. 2 at
// scale 1; Sec. 2.1 row normalisation D^).
//
// One wave owns one block-row x (32 queries). For every selected column block
// y, in ascending order, it computes the 32x32 tile S = c Q_x K_y^T on the
// matrix cores (block-sparse SDDMM), turns it into softmax weights and row sums
// (online softmax), and accumulates P V_y (block-sparse SpMM). At the end the
// result is merged with the block-row's low-resolution term (M_x, c_x, L_x)
// and normalised.
//
// Matrix-core layout (v_mfma_f32_32x32x16_bf16; 32x32x2_f32 for float32):
//  * S is formed transposed, S^T = K_y Q_x^T, so lane l holds query l%32 and
//    16 of its 32 key scores (keys 8(r/4) + 4(l/32) + r%4 in register r).
//    That is already the B-operand layout of O^T += V_y^T P^T up to a fixed
//    permutation of the key index, so P never moves between lanes; only the
//    row max crosses the two half-waves.
//  * The contraction index over d is permuted too: lane half h = l/32 takes
//    the contiguous half [h*d/2, (h+1)*d/2) of each Q and K row.
//  * In the packed copies of K and V written by the pooling pass (layout in
//    kernels.h) every operand of a tile (K_y, and V_y^T, the A operand of the
//    second product) is one 16-byte chunk per lane, 1 KB contiguous per wave.
//
// Two kernels share that per-row arithmetic (struct TileRow), so their results
// are bit-identical:
//  * tile_stream_kernel (raw K/V rows: bfloat16, and float32 with d <= 64;
//    packed K/V, tiles up to 8 KB): the next selected tile is copied HBM/L2 ->
//    a wave-private LDS slot with direct-to-LDS loads while the current one is
//    computed from registers.
//  * tile_kernel: raw float32 K/V with d = 128 (K rows read directly, V_y
//    through a wave-private LDS tile stored transposed with the key
//    permutation applied), and packed K/V with larger tiles (next tile's loads
//    in flight in registers).
// The softmax reference is set once per row (restart on overflow). Workgroup order
// is remapped so each XCD processes a contiguous range of heads and keeps
// their K/V tiles in its L2.
#include "common.h"
#include "kernels.h"
#include "tile_ops.h"

namespace mra {

// Reference point of the online softmax (log2 units). The weights of a tile
// are exp2(s * c * log2(e) - mrun) for the row's reference mrun, which need
// not be the running max: any reference works as long as weights and
// accumulators stay finite, because the final normalisation uses the same
// reference. mrun is set to the exact max of the row's first tile plus
// kRefMargin; later tiles only check that their weights sum to at most
// 2^kWeightCap per lane (far inside float32 and bfloat16 range, 2^128, even
// summed over 65536 keys). If a tile exceeds it, the row is computed again with
// the exact max over all its tiles as the reference, where no weight exceeds 1.
// The loop body thus has no 16-way max, no cross-lane exchange and no branch
// that rescales O. The margin makes that restart rare: a later logit must
// exceed the first tile's max by 96 (log2 units, 66.5 nats) to trigger it,
// while the row's largest weight stays at least 2^-32, far above the float32
// and bfloat16 underflow threshold 2^-126 (and bfloat16 rounding is relative,
// so the precision of the weights does not change).
constexpr float kWeightCap = 0x1p64f;
constexpr float kRefMargin = 32.0f;

__device__ __forceinline__ float tile_max(const f32x16& s) {
  float a = s[0];
#pragma unroll
  for (int r = 1; r < 16; ++r) a = __builtin_elementwise_maximum(a, s[r]);
  return a;
}

// Accumulator state and arithmetic of one block-row (32 queries) in one wave.
template <int DT, int D, bool COARSE>
struct TileRow {
  using Cfg = TileCfg<DT, D>;
  using elem = typename Cfg::elem;
  static constexpr int NT = Cfg::kNT, KC = Cfg::kKChunks;
  f32x16 o[NT];
  float mrun, lrun, sl2;
  bool first;                                      // no reference yet
  u32x4 qf[KC];

  // Q_x as the B operand: each lane reads d/2 contiguous elements of one row.
  __device__ __forceinline__ void init(const elem* Q, int x, float scale_log2) {
    const int lane = lane_id(), jq = lane & 31, h = lane >> 5;
    const u32x4* qrow = reinterpret_cast<const u32x4*>(Q + (long long)(x * 32 + jq) * D + (D / 2) * h);
#pragma unroll
    for (int s = 0; s < KC; ++s) qf[s] = qrow[s];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
    mrun = -INFINITY;                              // no fine block: no weight
    lrun = 0.0f;
    sl2 = scale_log2;
    first = true;
  }

  // S^T = K_y Q_x^T
  __device__ __forceinline__ f32x16 scores(const u32x4 (&kf)[KC]) const {
    return mfma_abt<DT, KC>(kf, qf);
  }

  // Max of this tile's scores for this lane's query, in log2 units (lanes l
  // and l^32 share a query).
  __device__ __forceinline__ float tile_ref(const f32x16& s) const {
    return halves_max(tile_max(s)) * sl2;
  }

  // Start the row again with a fixed reference (no weight above 1).
  __device__ __forceinline__ void restart(float ref) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
    lrun = 0.0f;
    mrun = ref;
    first = false;
  }

  // bfloat16 weights of one tile into pk (two per register, the operand
  // order of the second product); returns their sum in float32.
  __device__ __forceinline__ float weights_bf16(const f32x16& s, uint32_t (&pk)[8]) const {
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    float t = 0.0f;
#pragma unroll
    for (int rr = 0; rr < 8; ++rr) {
      const float p0 = __builtin_amdgcn_exp2f(fmaf(s[2 * rr], sl2, -mrun));
      const float p1 = __builtin_amdgcn_exp2f(fmaf(s[2 * rr + 1], sl2, -mrun));
      bf16x2 pb;
      pb[0] = (__bf16)p0;
      pb[1] = (__bf16)p1;
      t = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, t, false);   // sum of the rounded weights
      pk[rr] = __builtin_bit_cast(uint32_t, pb);
    }
    return t;
  }

  __device__ __forceinline__ float weights_f32(const f32x16& s, float (&p)[16]) const {
    float t = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      p[r] = __builtin_amdgcn_exp2f(fmaf(s[r], sl2, -mrun));
      t += p[r];
    }
    return t;
  }

  // Softmax weights of one tile and O^T += V_y^T P^T. `va(c)` yields the
  // 16-byte A-operand chunk c of V_y^T for this lane. With use == false (a
  // block id outside [0, nb)) the weights are zero: the matrix-core
  // instructions still run, consuming the tile's operands on every path,
  // which keeps the compiler's load-counter waits tight. Returns false if
  // some weight of the row may have exceeded the cap (the caller then restarts
  // the row); with check == false the caller guarantees it cannot.
  template <class VA>
  __device__ __forceinline__ bool accumulate(const f32x16& s, bool use, bool check, VA va) {
    if (first && use) {                              // wave-uniform: the row's first tile
      mrun = tile_ref(s) + kRefMargin;
      first = false;
    }
    float t;
    if constexpr (DT == BF16) {
      uint32_t pk[8];
      t = weights_bf16(s, pk);
      if (!use) {
#pragma unroll
        for (int rr = 0; rr < 8; ++rr) pk[rr] = 0u;
        t = 0.0f;
      }
      mfma_acc_bf16<NT>(o, pk, va);
    } else {
      float p[16];
      t = weights_f32(s, p);
      if (!use) {
#pragma unroll
        for (int r = 0; r < 16; ++r) p[r] = 0.0f;
        t = 0.0f;
      }
      mfma_acc_f32<NT>(o, p, va);
    }
    lrun += t;
    return !check || __ballot(!(t <= kWeightCap)) == 0;
  }

  // Merge with the low-resolution term, normalise and store the 32 x d block;
  // if lse is not NULL also each query's log normaliser, ln of the row sum of
  // A^ (natural units).
  // cmaxg, csumg, cv: the block-row's coarse-term maximum, sum and vector
  // (its D floats, in LDS or global memory)
  __device__ __forceinline__ void finish(elem* Out, float* lse, int x, long long g, float cmaxg,
                                         float csumg, const float* cv) {
    const int lane = lane_id(), jq = lane & 31, h = lane >> 5;
    const float ltot = halves_sum(lrun);
    float af = 1.0f, bc = 0.0f, den = ltot, Mt = mrun;
    if constexpr (COARSE) {
      const float Mx = cmaxg * kLog2e;
      Mt = fmaxf(mrun, Mx);
      af = exp2f(mrun - Mt);
      bc = exp2f(Mx - Mt);
      den = ltot * af + csumg * bc;
    }
    if (lse != nullptr && h == 0) lse[g * 32 + jq] = (log2f(den) + Mt) * kLn2;
    const float inv = 1.0f / den;
    const float ao = af * inv, bv = bc * inv;       // z = o * ao + cvec * bv
    elem* orow = Out + (long long)(x * 32 + jq) * D;
    u32x2 pend = {0u, 0u};                          // bf16: the even group's 4 values
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int d0 = 32 * t + 8 * rg + 4 * h;
        float z[4];
        f32x4 c4 = {0.0f, 0.0f, 0.0f, 0.0f};
        if constexpr (COARSE) c4 = *reinterpret_cast<const f32x4*>(cv + d0);
#pragma unroll
        for (int e = 0; e < 4; ++e) z[e] = COARSE ? fmaf(o[t][4 * rg + e], ao, c4[e] * bv) : o[t][4 * rg + e] * ao;
        if constexpr (DT == BF16) {
          bf16x2 lo, hi;
          lo[0] = (__bf16)z[0]; lo[1] = (__bf16)z[1];
          hi[0] = (__bf16)z[2]; hi[1] = (__bf16)z[3];
          const u32x2 pr = {__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
          // lanes l and l^32 hold dims 4h..4h+3 of groups rg (even, odd):
          // exchange so that lane h = 0 stores the even group's 8 dims and
          // lane h = 1 the odd group's, 16 contiguous bytes each
          if ((rg & 1) == 0) {
            pend = pr;
          } else {
            const u32x2 send = h ? pend : pr;          // h = 0 sends its odd group, h = 1 its even one
            u32x2 recv;
            recv[0] = (uint32_t)__shfl_xor((int)send[0], 32);
            recv[1] = (uint32_t)__shfl_xor((int)send[1], 32);
            const u32x4 st = h ? u32x4{recv[0], recv[1], pr[0], pr[1]} : u32x4{pend[0], pend[1], recv[0], recv[1]};
            *reinterpret_cast<u32x4*>(orow + 32 * t + 8 * (rg - 1) + 8 * h) = st;
          }
        } else {
          const f32x4 st = {z[0], z[1], z[2], z[3]};
          *reinterpret_cast<f32x4*>(orow + d0) = st;
        }
      }
    }
  }
};

// ---------------------------------------------------------------------------
// One wave per block-row.
template <int DT, int D, bool COARSE, bool PACKED>
__global__ __launch_bounds__((TileCfg<DT, D>::kWaves * kWave)) void tile_kernel(
    const void* __restrict__ qv, const void* __restrict__ kv, const void* __restrict__ vv,
    const int32_t* __restrict__ idx, const float* __restrict__ cmax,
    const float* __restrict__ csum, const float* __restrict__ cvec, void* __restrict__ outv,
    float* __restrict__ lse, int n, int nb, int m, long long rows, float scale_log2) {
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
  const elem* K = reinterpret_cast<const elem*>(kv) + hoff;
  extern __shared__ int32_t sidx_all[];
  int32_t* myidx = sidx_all + w * m;
  // Q_x's loads are issued first, so their latency overlaps the staging of
  // the selection list
  TileRow<DT, D, COARSE> row;
  row.init(reinterpret_cast<const elem*>(qv) + hoff, x, scale_log2);
  m = stage_selection(idx + g * m, m, nb, myidx);  // valid entries only, in order
  auto clampy = [&](int y) { return (y < 0 || y >= nb) ? 0 : y; };
  auto valid = [&](int y) { return y >= 0 && y < nb; };

  if constexpr (PACKED) {
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
    // Two register buffers: tile i+1 loads while tile i is computed. Loads
    // are issued unconditionally (past the last tile they re-read the last
    // tile, a cache hit) so every path leaves the same loads in flight.
    auto pass = [&](bool check) -> bool {
      u32x4 kA[KC], vA[VC], kB[KC], vB[VC];
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
        if (!row.accumulate(row.scores(kA), valid(ya), check, [&](int c) { return vA[c]; })) return false;
        if (i + 1 >= m) break;
        const int yc = clampy(wave_uniform(myidx[min(i + 2, m - 1)]));
        load_kpacked(yc, kA);
        load_vpacked(yc, vA);
        if (!row.accumulate(row.scores(kB), valid(yb), check, [&](int c) { return vB[c]; })) return false;
      }
      return true;
    };
    if (!pass(true)) {
      // some weight grew too large: again, relative to the row's exact max
      float mx = -INFINITY;
      for (int i = 0; i < m; ++i) {
        const int yy = wave_uniform(myidx[i]);
        if (!valid(yy)) continue;
        u32x4 kf[KC];
        load_kpacked(yy, kf);
        mx = __builtin_elementwise_maximum(mx, row.tile_ref(row.scores(kf)));
      }
      row.restart(mx);
      pass(false);
    }
  } else {
    elem* vt = vt_all[w];
    const elem* V = reinterpret_cast<const elem*>(vv) + hoff;
    auto load_k = [&](int y, u32x4 (&kc)[KC]) {
      const u32x4* krow = reinterpret_cast<const u32x4*>(K + (long long)(y * 32 + jq) * D + (D / 2) * h);
#pragma unroll
      for (int s = 0; s < KC; ++s) kc[s] = krow[s];
    };
    auto pass = [&](bool check) -> bool {
    for (int i = 0; i < m; ++i) {
      const int y = wave_uniform(myidx[i]);
      if (!valid(y)) continue;
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
      const f32x16 s = row.scores(kc);
      wave_lds_sync();
      bool ok;
      if constexpr (DT == BF16) {
        ok = row.accumulate(s, true, check, [&](int c) {
          const int u = c / NT, t = c % NT;
          return *reinterpret_cast<const u32x4*>(vt + (32 * t + jq) * PITCH + 16 * u + 8 * h);
        });
      } else {
        ok = row.accumulate(s, true, check, [&](int c) {
          const int t = c / 4, a = c % 4;
          return *reinterpret_cast<const u32x4*>(vt + (32 * t + jq) * PITCH + 16 * h + 4 * a);
        });
      }
      wave_lds_sync();                               // reads done before the next overwrite
      if (!ok) return false;
    }
    return true;
    };
    if (!pass(true)) {
      float mx = -INFINITY;
      for (int i = 0; i < m; ++i) {
        const int yy = wave_uniform(myidx[i]);
        if (!valid(yy)) continue;
        u32x4 kf[KC];
        load_k(yy, kf);
        mx = __builtin_elementwise_maximum(mx, row.tile_ref(row.scores(kf)));
      }
      row.restart(mx);
      pass(false);
    }
  }
  row.finish(reinterpret_cast<elem*>(outv) + hoff, lse, x, g, COARSE ? cmax[g] : 0.0f, COARSE ? csum[g] : 0.0f,
             COARSE ? cvec + g * D : nullptr);
}

// ---------------------------------------------------------------------------
// Raw K/V tiles in LDS (bfloat16, d <= 64). A 32-row tile of K (or V) is 4 KB
// (d = 64) of consecutive rows in HBM. It is copied with direct-to-LDS loads
// of whole rows (each 1 KB load covers 1024 / (2d) complete rows, so it
// touches as many cache lines as a contiguous copy), but each lane fetches
// the 16-byte block that belongs at its LDS position under an XOR swizzle of
// the blocks within a row: block b of row r sits at block b ^ f(r). With the
// swizzles below the matrix-core operand reads are free of bank conflicts
// (checked with a CPU model of the LDS banks):
//   K, row layout, ds_read_b128 (16 lanes = 16 rows per pass): lane (h, j)
//     reads row j, block (d/16) h + s;
//   V^T, transposed layout, ds_read_b64_tr_b16 (32 lanes per pass): within a
//     group of 16 lanes, lane 4k + g supplies 4 columns of row key0 + k and
//     lane i receives element i % 4 of lane (4k + i/4)'s 8 bytes as value k;
//     two reads (key0 = 16u + 4h and 16u + 8 + 4h) fill the 8 keys of a
//     chunk in the order the weights of the second product hold them.
template <int D>
__host__ __device__ constexpr int raw_swz_k(int r) {
  return D == 128 ? r & 15 : (D == 64 ? (r >> 1) & 7 : (r >> 2) & 3);
}
template <int D>
__host__ __device__ constexpr int raw_swz_v(int r) {
  return D == 128 ? 4 * (r & 3) : (D == 64 ? ((r >> 1) & 1) << 2 : 0);
}

// The 1 KB copies of a raw K tile and of a raw V tile (32 x d bfloat16: d/16
// copies each), buffer loads to LDS: the head's rows are one buffer resource,
// the tile's offset goes in the scalar offset and the lane's swizzled source
// offset in the vector offset, so a copy costs no vector instruction. Copy i
// moves source and destination by i KB; the swizzled lane offsets repeat with
// period 2 (K, d = 64: the swizzle of row r depends on r / 2), 4 (K, d = 128:
// r mod 16) or 1 in the copy index, so koff holds the offsets of copies
// i mod 4 and voff the V offset.
template <int I>
__device__ __forceinline__ void copy_raw_tiles_buf(i32x4 krs, i32x4 vrs, unsigned ktile, unsigned vtile,
                                                   const unsigned (&koff)[4], unsigned voff, lptr_t ks,
                                                   lptr_t vs) {
  if constexpr (I > 0) {
    copy_raw_tiles_buf<I - 1>(krs, vrs, ktile, vtile, koff, voff, ks, vs);
    constexpr int i = I - 1;
    buffer_load_lds16(krs, ks + i * 1024, koff[i & 3], ktile + i * 1024);
    buffer_load_lds16(vrs, vs + i * 1024, voff, vtile + i * 1024);
  }
}

// Transposed V chunks c = u NT + t (c < VC) of a raw tile: two transposing
// reads each, 8 rows apart, from this lane's column-tile address vt[t].
template <int D, int C, int VC>
struct RawTrChunks {
  static constexpr int NT = D / 32, RB = 2 * D;
  static __device__ __forceinline__ void run(const uint32_t* vt, u32x4* v) {
    if constexpr (C < VC) {
      constexpr int u = C / NT, t = C % NT;
      const u32x2 lo = lds_read_tr16<16 * u * RB>(vt[t]);
      const u32x2 hi = lds_read_tr16<(16 * u + 8) * RB>(vt[t]);
      v[C] = u32x4{lo[0], lo[1], hi[0], hi[1]};
      RawTrChunks<D, C + 1, VC>::run(vt, v);
    }
  }
};

// Raw float32 tiles (d <= 64). K: 4d-byte rows, the byte geometry of a
// bfloat16 tile of 2d columns, so its copies, swizzle and row-layout reads are
// those above with D2 = 2d (element (r, c) at raw_offset<D2>(r, 2c)). V is read
// transposed, four consecutive keys of one column per 16-byte operand chunk,
// with two ds_read2st64_b32 (keys 8a + 4h + e, e = 0, 1 and 2, 3, 256 bytes
// apart in LDS); rows are placed so that neither read has a bank conflict
// (CPU-modelled): d = 32 (128-byte rows): row r of each group of eight at
// slot 2 (r mod 4) + (r / 4 mod 2), so rows r and r + 4 fall in opposite bank
// halves; d = 64 (256-byte rows): the two 128-byte halves of rows with
// r / 4 odd swapped.
template <int D>
__host__ __device__ constexpr int f32v_slot(int r) {
  return D == 32 ? 8 * (r >> 3) + 2 * (r & 3) + ((r >> 2) & 1) : r;
}
template <int D>
__host__ __device__ constexpr int f32v_offset(int r, int c) {
  return f32v_slot<D>(r) * (4 * D) + 16 * ((c >> 2) ^ (D == 64 ? 8 * ((r >> 2) & 1) : 0)) + 4 * (c & 3);
}
// Source byte offset (within the V tile) of the 16 bytes lane `lane` copies to
// LDS byte i * 1024 + 16 lane.
template <int D>
__device__ __forceinline__ int f32v_copy_offset(int i, int lane) {
  const int rb = 4 * D, q = i * 1024 + 16 * lane, sl = q / rb, b = (q % rb) / 16;
  if (D == 32) return (8 * (sl >> 3) + 4 * (sl & 1) + ((sl >> 1) & 3)) * rb + 16 * b;
  return sl * rb + 16 * (b ^ (8 * ((sl >> 2) & 1)));
}

// The K copies (KPB-periodic lane offsets, as copy_raw_tiles_buf) and the V
// copies of a raw float32 tile (period 1 for d = 32, 2 for d = 64).
template <int I>
__device__ __forceinline__ void copy_raw_f32_buf(i32x4 krs, i32x4 vrs, unsigned ktile, unsigned vtile,
                                                 const unsigned (&koff)[4], const unsigned (&voff)[2], lptr_t ks,
                                                 lptr_t vs) {
  if constexpr (I > 0) {
    copy_raw_f32_buf<I - 1>(krs, vrs, ktile, vtile, koff, voff, ks, vs);
    constexpr int i = I - 1;
    buffer_load_lds16(krs, ks + i * 1024, koff[i & 3], ktile + i * 1024);
    buffer_load_lds16(vrs, vs + i * 1024, voff[i & 1], vtile + i * 1024);
  }
}

// Transposed V chunks c = 4 t + a (c < VC) of a raw float32 tile: keys
// 8a + 4h + e of column 32 t + i, from this lane's column-tile address vt[t].
template <int D, int C, int VC>
struct RawF32TrChunks {
  static constexpr int K64 = D == 32 ? 4 : 8;          // 256-byte units between key groups a
  static __device__ __forceinline__ void run(const uint32_t* vt, u32x4* v) {
    if constexpr (C < VC) {
      constexpr int t = C / 4, a = C % 4;
      const u32x2 lo = lds_read2st64<K64 * a, K64 * a + 1>(vt[t]);
      const u32x2 hi = lds_read2st64<K64 * a + 2, K64 * a + 3>(vt[t]);
      v[C] = u32x4{lo[0], lo[1], hi[0], hi[1]};
      RawF32TrChunks<D, C + 1, VC>::run(vt, v);
    }
  }
};

// ---------------------------------------------------------------------------
// One wave per block-row, K/V staged through a wave-private LDS slot:
// the next selected tile is copied HBM/L2 -> LDS with direct-to-LDS loads
// while the current one is computed from registers. Prefetching into LDS
// instead of registers leaves room for four waves per SIMD.
constexpr int kStreamWaves = 4;
constexpr int kStreamSlots = 1;

// Wait until at most `keep` tiles of CH loads each are still in flight (the
// load counter counts down in issue order, so the older tiles have landed).
template <int CH>
__device__ __forceinline__ void wait_tiles_in_flight(int keep) {
  if (keep <= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if (keep == 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CH) : "memory");
  else asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * CH) : "memory");
}

template <int DT, int D, bool COARSE, int WAVES, int SLOTS>
__global__ __launch_bounds__(WAVES * kWave) void tile_stream_kernel(
    const void* __restrict__ qv, const void* __restrict__ kv, const void* __restrict__ vv,
    const int32_t* __restrict__ idx, const float* __restrict__ cmax,
    const float* __restrict__ csum, const float* __restrict__ cvec, void* __restrict__ outv,
    float* __restrict__ lse, int n, int nb, int m, long long row0, long long rows, float scale_log2) {
  using Cfg = TileCfg<DT, D>;
  using elem = typename Cfg::elem;
  constexpr int KC = Cfg::kKChunks, VC = Cfg::kVChunks, CH = Cfg::kChunks;
  static_assert(CH <= 16, "operands of a tile are held in registers");
  static_assert(SLOTS >= 1 && SLOTS <= 3, "tiles in flight per wave");
  static_assert(DT == BF16 || D <= 64, "raw tiles: bfloat16, or float32 with d <= 64");
  constexpr bool F32RAW = DT == F32;
  constexpr int D2 = F32RAW ? 2 * D : D;             // the bfloat16 geometry of the K tile
  // the slots are their own LDS object, apart from the selection lists, so
  // reading a list does not wait for loads in flight into a slot
  __shared__ __attribute__((aligned(16))) u32x4 slot_all[WAVES][SLOTS][CH * 64];
  // Tiles of 8 KB per part (two waves per SIMD) fetch the coarse term's
  // vector into LDS while the tiles run (its maximum and sum are loaded then
  // too): with two waves per SIMD, reading it after the last tile exposed its
  // latency at every row's end; at four waves per SIMD the other waves hide
  // it, and the extra load at the row's start cost more than it saved.
  constexpr bool kTermAhead = COARSE && D2 >= 128;
  __shared__ __attribute__((aligned(16))) float cvl[WAVES][kTermAhead ? add_lds_floats(D) : 1];
  extern __shared__ int32_t sidx_all[];

  const int w = wave_uniform(threadIdx.x / kWave);
  const int lane = lane_id();
  const long long wg = xcd_remap(blockIdx.x, gridDim.x);
  const long long g = row0 + wg * WAVES + w;         // global block-row (rows row0 .. rows - 1)
  if (g >= rows) return;                             // no workgroup barriers below
  float cmaxg = 0.0f, csumg = 0.0f;
  if constexpr (kTermAhead) {
    prefetch_vec_lds<D>(cvec + g * D, (__attribute__((address_space(3))) char*)cvl[w]);
    cmaxg = cmax[g];
    csumg = csum[g];
  }
  const long long bh = g / nb;
  const int x = (int)(g - bh * nb);
  const long long hoff = bh * (long long)n * D;
  int32_t* myidx = sidx_all + w * m;
  // Q_x's loads are issued first, so their latency overlaps the staging of
  // the selection list
  TileRow<DT, D, COARSE> row;
  row.init(reinterpret_cast<const elem*>(qv) + hoff, x, scale_log2);
  m = stage_selection(idx + g * m, m, nb, myidx);  // valid entries only, in order
  // the head's K and V rows (tile y at byte y * 32 d e)
  const char* kslab = static_cast<const char*>(kv) + (size_t)bh * nb * KC * 1024;
  const char* vslab = static_cast<const char*>(vv) + (size_t)bh * nb * VC * 1024;
  // this lane's source offsets for the copies (see copy_raw_tiles_buf) and its
  // LDS read offsets (K chunk c; V^T column tile t)
  constexpr int NT = TileCfg<DT, D>::kNT;
  constexpr int KPB = D2 == 128 ? 4 : (D2 == 64 ? 2 : 1);  // period of the K copy offsets
  unsigned koffq[4];                                 // K source offsets of copies i mod 4
#pragma unroll
  for (int q = 0; q < 4; ++q) koffq[q] = raw_copy_offset<D2, raw_swz_k<D2>>(q % KPB, lane) - (q % KPB) * 1024;
  const i32x4 krs = buffer_rsrc(kslab, (unsigned)nb * KC * 1024u);
  const i32x4 vrs = buffer_rsrc(vslab, (unsigned)nb * VC * 1024u);
  const int h = lane >> 5, j = lane & 31, i16 = lane & 15;
  int kread[KC], vread[NT];
#pragma unroll
  for (int c = 0; c < KC; ++c) kread[c] = raw_offset<D2, raw_swz_k<D2>>(j, (D2 / 2) * h + 8 * c);
  unsigned voff0 = 0, voffq[2] = {0u, 0u};
  if constexpr (F32RAW) {
#pragma unroll
    for (int q = 0; q < 2; ++q) voffq[q] = f32v_copy_offset<D>(q, lane) - q * 1024;
#pragma unroll
    for (int t = 0; t < NT; ++t) vread[t] = KC * 1024 + f32v_offset<D>(4 * h, 32 * t + j);
  } else {
    voff0 = raw_copy_offset<D, raw_swz_v<D>>(0, lane);
#pragma unroll
    for (int t = 0; t < NT; ++t)
      vread[t] = KC * 1024 +
                 raw_offset<D, raw_swz_v<D>>(4 * h + i16 / 4, 32 * t + 16 * ((lane >> 4) & 1) + 4 * (i16 & 3));
  }
  auto issue = [&](int y, int sidx) {
    unsigned char* slot = reinterpret_cast<unsigned char*>(slot_all[w][sidx]);
    auto* ks = (__attribute__((address_space(3))) char*)slot;
    auto* vs = (__attribute__((address_space(3))) char*)(slot + KC * 1024);
    if constexpr (F32RAW)
      copy_raw_f32_buf<KC>(krs, vrs, (unsigned)y * KC * 1024u, (unsigned)y * VC * 1024u, koffq, voffq, ks, vs);
    else
      copy_raw_tiles_buf<KC>(krs, vrs, (unsigned)y * KC * 1024u, (unsigned)y * VC * 1024u, koffq, voff0, ks, vs);
  };
  // entries outside [0, nb) are skipped
  auto next_valid = [&](int j, int& y) {
    for (; j < m; ++j) {
      y = wave_uniform(myidx[j]);
      if (y >= 0 && y < nb) break;
    }
    return j;
  };
  // Tiles are numbered in the order they are used; tile t goes to slot
  // t % SLOTS, and up to SLOTS of them are in flight.
  auto pass = [&](bool check) -> bool {
    int yn = 0;
    int ni = next_valid(0, yn);                      // next list entry to load
    int issued = 0, used = 0;
#pragma unroll
    for (int t = 0; t < SLOTS; ++t)
      if (ni < m) {
        issue(yn, t);
        ++issued;
        ni = next_valid(ni + 1, yn);
      }
    while (used < issued) {
      wait_tiles_in_flight<CH>(issued - used - 1);   // tile `used` is in its slot
      u32x4 kf[KC], vf[VC];
      const uint32_t base = lds_addr(slot_all[w][used % SLOTS]);
#pragma unroll
      for (int c = 0; c < KC; ++c) kf[c] = lds_read16<0>(base + kread[c]);
      uint32_t va[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) va[t] = base + vread[t];
      if constexpr (F32RAW) RawF32TrChunks<D, 0, VC>::run(va, vf);
      else RawTrChunks<D, 0, VC>::run(va, vf);
      lds_done(kf);
      lds_done(vf);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // operands in registers
      ++used;
      if (ni < m) {                                  // refill the slot just read
        issue(yn, issued % SLOTS);
        ++issued;
        ni = next_valid(ni + 1, yn);
      }
      if (!row.accumulate(row.scores(kf), true, check, [&](int c) { return vf[c]; })) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the slots are idle again
        return false;
      }
    }
    return true;
  };
  if (!pass(true)) {
    // some weight grew too large: again, relative to the row's exact max
    float mx = -INFINITY;
    for (int i = 0; i < m; ++i) {
      const int yy = wave_uniform(myidx[i]);
      if (yy < 0 || yy >= nb) continue;
      u32x4 kf[KC];
      load_rows<DT, D>(reinterpret_cast<const elem*>(kslab + (size_t)yy * KC * 1024), kf);
      mx = __builtin_elementwise_maximum(mx, row.tile_ref(row.scores(kf)));
    }
    row.restart(mx);
    pass(false);
  }
  if constexpr (kTermAhead) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the coarse-term vector is in LDS
    row.finish(reinterpret_cast<elem*>(outv) + hoff, lse, x, g, cmaxg, csumg, cvl[w]);
  } else {
    row.finish(reinterpret_cast<elem*>(outv) + hoff, lse, x, g, COARSE ? cmax[g] : 0.0f,
               COARSE ? csum[g] : 0.0f, COARSE ? cvec + g * D : nullptr);
  }
}

// ---------------------------------------------------------------------------
// Raw K/V tiles of up to 8 KB (bfloat16; float32 with d <= 64) stream through
// LDS.
//
// Where a head's K and V exceed an XCD's L2 (4 MB), the pass is launched one
// occupancy round of block-rows at a time: every block-row of a launch starts
// together and walks its (ascending) selection in step with its neighbours,
// so the blocks the XCD's resident rows touch at any moment stay close
// together and more of them hit L2. Within one launch, later rows start as
// earlier ones finish and the rows drift apart over the head. Heads that fit
// L2 are launched whole (a launch per round costs more than it saves there).
template <int DT, int D, bool COARSE>
static void launch_stream_c(const void* q, const void* k, const void* v, const int32_t* idx,
                            const float* cmax, const float* csum, const float* cvec, void* out,
                            float* lse, long long bh, int n, int m, float scale_log2, hipStream_t stream) {
  const int nb = n / kBlock;
  const long long rows = bh * nb;
  const size_t smem = (size_t)kStreamWaves * m * sizeof(int32_t);  // per-wave selection lists
  auto kernel = tile_stream_kernel<DT, D, COARSE, kStreamWaves, kStreamSlots>;
  const size_t head_kv = (size_t)2 * n * D * (DT == BF16 ? 2 : 4);
  long long chunk = head_kv > kL2PerXcd ? resident_items(kernel, kStreamWaves * kWave, smem, kStreamWaves) : 0;
  if (chunk <= 0) chunk = rows;
  for (long long r0 = 0; r0 < rows; r0 += chunk) {
    const long long r1 = r0 + chunk < rows ? r0 + chunk : rows;
    const unsigned blocks = (unsigned)((r1 - r0 + kStreamWaves - 1) / kStreamWaves);
    kernel<<<blocks, kStreamWaves * kWave, smem, stream>>>(q, k, v, idx, cmax, csum, cvec, out, lse, n, nb,
                                                           m, r0, r1, scale_log2);
  }
}

template <int DT, int D>
static void launch_stream(const void* q, const void* k, const void* v, const int32_t* idx,
                          const float* cmax, const float* csum, const float* cvec, void* out,
                          float* lse, long long bh, int n, int m, float scale_log2, hipStream_t stream) {
  if (cmax)
    launch_stream_c<DT, D, true>(q, k, v, idx, cmax, csum, cvec, out, lse, bh, n, m, scale_log2, stream);
  else
    launch_stream_c<DT, D, false>(q, k, v, idx, cmax, csum, cvec, out, lse, bh, n, m, scale_log2, stream);
}

// float32 tiles of d = 128 (16 KB): the packed copy, or the raw rows
template <bool PACKED>
static void launch_tile_f32_128(const void* q, const void* k, const void* v, const int32_t* idx,
                                const float* cmax, const float* csum, const float* cvec, void* out,
                                float* lse, long long bh, int n, int m, float scale_log2, hipStream_t stream) {
  constexpr int W = TileCfg<F32, 128>::kWaves;
  const int nb = n / kBlock;
  const long long rows = bh * nb;
  const unsigned blocks = (unsigned)((rows + W - 1) / W);
  const size_t smem = (size_t)W * m * sizeof(int32_t);     // per-wave selection lists
  if (cmax)
    tile_kernel<F32, 128, true, PACKED><<<blocks, W * kWave, smem, stream>>>(q, k, v, idx, cmax, csum, cvec, out, lse, n, nb, m, rows, scale_log2);
  else
    tile_kernel<F32, 128, false, PACKED><<<blocks, W * kWave, smem, stream>>>(q, k, v, idx, cmax, csum, cvec, out, lse, n, nb, m, rows, scale_log2);
}

hipError_t launch_tile(const void* q, const void* k, const void* v, const void* kvpacked,
                       const int32_t* idx, const float* cmax, const float* csum,
                       const float* cvec, void* out, float* lse, long long bh, int n, int d,
                       int m, int dtype, hipStream_t stream) {
  const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)d));
  if (kvpacked) {
    // only float32 tiles of d = 128 are read from the packed copy
    if (dtype != F32 || d != 128) return hipErrorInvalidValue;
    const size_t half = (size_t)bh * n * d * 4;
    const void* kpk = kvpacked;
    const void* vpk = static_cast<const char*>(kvpacked) + half;
    launch_tile_f32_128<true>(q, kpk, vpk, idx, cmax, csum, cvec, out, lse, bh, n, m, scale_log2, stream);
    return hipGetLastError();
  }
  if (dtype == BF16) {
    if (d == 32) launch_stream<BF16, 32>(q, k, v, idx, cmax, csum, cvec, out, lse, bh, n, m, scale_log2, stream);
    else if (d == 64) launch_stream<BF16, 64>(q, k, v, idx, cmax, csum, cvec, out, lse, bh, n, m, scale_log2, stream);
    else launch_stream<BF16, 128>(q, k, v, idx, cmax, csum, cvec, out, lse, bh, n, m, scale_log2, stream);
  } else {
    if (d == 32) launch_stream<F32, 32>(q, k, v, idx, cmax, csum, cvec, out, lse, bh, n, m, scale_log2, stream);
    else if (d == 64) launch_stream<F32, 64>(q, k, v, idx, cmax, csum, cvec, out, lse, bh, n, m, scale_log2, stream);
    else launch_tile_f32_128<false>(q, k, v, idx, cmax, csum, cvec, out, lse, bh, n, m, scale_log2, stream);
  }
  return hipGetLastError();
}

}  // namespace mra
