// Block means of Q, K, V: the scale-32 rows Q~, K~, V~ of MRA-2
// (Sec. 4.1 eq. recursive_pooling, Sec. 4.3 eq. recursive_pooling_V; five
// pairwise halvings of a 32-row block equal its plain mean).
//
// HBM-bound: every input byte is read once, 1/32 of it is written back.
// One thread owns one 16-byte column chunk of one 32-row block and walks its
// 32 rows; a wave's load covers whole 128-byte row segments of consecutive
// blocks, so every HBM line fetched is fully used. No LDS, no barriers.
//
// Optionally K and V are also written in the tile kernel's matrix-core operand
// order ("packed K/V", layout in kernels.h), so every operand load of the tile
// pass is one contiguous 1 KB wave access; that configuration pools Q, K and V
// in one launch that stages blocks through LDS so the packed writes stay
// contiguous.
#include "common.h"
#include "kernels.h"

namespace mra {

template <int DT>
__global__ __launch_bounds__(256) void pool_kernel(const void* __restrict__ x0,
                                                    const void* __restrict__ x1,
                                                    const void* __restrict__ x2,
                                                    float* __restrict__ y0,
                                                    float* __restrict__ y1,
                                                    float* __restrict__ y2,
                                                    long long chunks, int d) {
  const int which = blockIdx.y;
  const void* x = which == 0 ? x0 : (which == 1 ? x1 : x2);
  float* y = which == 0 ? y0 : (which == 1 ? y1 : y2);
  if (y == nullptr) return;
  constexpr int kPer = DT == BF16 ? 8 : 4;        // elements per 16-byte chunk
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= chunks) return;
  const int cpr = d / kPer;                        // chunks per row
  const long long blk = t / cpr;
  const int c = (int)(t - blk * cpr);
  const long long row0 = blk * kBlock;             // first row of the block (all heads flattened)
  const u32x4* base = reinterpret_cast<const u32x4*>(x) + row0 * cpr + c;

  float acc[kPer];
#pragma unroll
  for (int e = 0; e < kPer; ++e) acc[e] = 0.0f;
#pragma unroll 8
  for (int r = 0; r < kBlock; ++r) {
    const u32x4 w = base[(long long)r * cpr];
    if constexpr (DT == BF16) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] += bf16_to_f32(w[e] & 0xFFFFu);
        acc[2 * e + 1] += bf16_to_f32(w[e] >> 16);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] += __uint_as_float(w[e]);
    }
  }
  constexpr float inv = 1.0f / kBlock;             // exact: power of two
  f32x4* out = reinterpret_cast<f32x4*>(y + blk * d + c * kPer);
#pragma unroll
  for (int v = 0; v < kPer / 4; ++v) {
    f32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = acc[4 * v + e] * inv;
    out[v] = o;
  }
}

// Q, K and V in one launch (blockIdx.y = 0: K, 1: V, 2: Q): block means
// (same row order as above, so the same bits) and, for K and V, the packed
// copies. Whole 32-row blocks are staged through LDS so that both the reads
// and the packed writes are contiguous 16-byte chunks across lanes.
template <int DT, int D>
__global__ __launch_bounds__(256) void pool_pack_kernel(const void* __restrict__ qin,
                                                         const void* __restrict__ kin,
                                                         const void* __restrict__ vin,
                                                         float* __restrict__ qp,
                                                         float* __restrict__ kp,
                                                         float* __restrict__ vp,
                                                         void* __restrict__ kvpacked,
                                                         long long nblocks) {
  using elem = typename std::conditional<DT == BF16, uint16_t, float>::type;
  constexpr int kPer = DT == BF16 ? 8 : 4;         // elements per chunk
  constexpr int CPR = D / kPer;                    // chunks per row
  constexpr int CPB = kBlock * CPR;                // chunks per block
  constexpr int NBLK = CPB >= 1024 ? 1 : 1024 / CPB; // blocks per workgroup pass (16 KB)
  constexpr int NT = D / 32;
  __shared__ __attribute__((aligned(16))) u32x4 tile[NBLK * CPB];
  const elem* te = reinterpret_cast<const elem*>(tile);
  const int which = blockIdx.y;
  const bool is_k = which == 0, pack = which < 2;
  const u32x4* src = reinterpret_cast<const u32x4*>(which == 0 ? kin : (which == 1 ? vin : qin));
  float* pooled = which == 0 ? kp : (which == 1 ? vp : qp);
  u32x4* dst = reinterpret_cast<u32x4*>(kvpacked) + (is_k ? 0 : nblocks * CPB);
  if (src == nullptr) return;                      // Q not requested (whole workgroup)
  const int tid = threadIdx.x;

  for (long long b0 = (long long)blockIdx.x * NBLK; b0 < nblocks; b0 += (long long)gridDim.x * NBLK) {
    const int nblk = (int)min((long long)NBLK, nblocks - b0);
#pragma unroll
    for (int ci = tid; ci < NBLK * CPB; ci += 256)
      if (ci < nblk * CPB) tile[ci] = src[b0 * CPB + ci];
    __syncthreads();
    // block means: one thread per (block, column chunk), rows in order
    for (int pc = tid; pc < nblk * CPR; pc += 256) {
      const int bl = pc / CPR, c = pc % CPR;
      float acc[kPer];
#pragma unroll
      for (int e = 0; e < kPer; ++e) acc[e] = 0.0f;
#pragma unroll 8
      for (int r = 0; r < kBlock; ++r) {
        const u32x4 w = tile[bl * CPB + r * CPR + c];
        if constexpr (DT == BF16) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[2 * e] += bf16_to_f32(w[e] & 0xFFFFu);
            acc[2 * e + 1] += bf16_to_f32(w[e] >> 16);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] += __uint_as_float(w[e]);
        }
      }
      constexpr float inv = 1.0f / kBlock;
      f32x4* out = reinterpret_cast<f32x4*>(pooled + (b0 + bl) * D + c * kPer);
#pragma unroll
      for (int q = 0; q < kPer / 4; ++q) {
        f32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = acc[4 * q + e] * inv;
        out[q] = o;
      }
    }
    // packed copy, one 16-byte output chunk per thread and pass
#pragma unroll
    for (int oc = tid; oc < NBLK * CPB; oc += 256) {
      if (!pack || oc >= nblk * CPB) continue;
      const int bl = oc / CPB, k = oc % CPB;
      const elem* tb = te + bl * kBlock * D;
      u32x4 o;
      if (is_k) {
        // chunk s*64 + 32h + j holds K[j][(d/2)h + kPer*s .. +kPer-1]
        const int sk = k / 64, h = (k % 64) / 32, j = k % 32;
        o = *reinterpret_cast<const u32x4*>(tb + j * D + (D / 2) * h + kPer * sk);
      } else if constexpr (DT == BF16) {
        // chunk (u*NT + t)*64 + 32h + j: V[16u + 8(s/4) + 4h + s%4][32t + j], s = 0..7
        const int u = k / (64 * NT), t = (k / 64) % NT, h = (k % 64) / 32, j = k % 32;
        const int dim = 32 * t + j;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
          const int key = 16 * u + 8 * (s2 >> 1) + 4 * h + 2 * (s2 & 1);
          o[s2] = (uint32_t)tb[key * D + dim] | ((uint32_t)tb[(key + 1) * D + dim] << 16);
        }
      } else {
        // chunk (t*4 + a)*64 + 32h + j: V[8a + 4h + kk][32t + j], kk = 0..3
        const int t = k / 256, a = (k / 64) % 4, h = (k % 64) / 32, j = k % 32;
        const int dim = 32 * t + j;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) o[kk] = __float_as_uint(tb[(8 * a + 4 * h + kk) * D + dim]);
      }
      dst[(b0 + bl) * CPB + k] = o;
    }
    __syncthreads();
  }
}

hipError_t launch_pool(const void* q, const void* k, const void* v, float* qp, float* kp,
                       float* vp, void* kvpacked, long long bh, int n, int d, int dtype,
                       hipStream_t stream) {
  const int threads = 256;
  if (kvpacked != nullptr) {
    // the forward's configuration: Q, K, V pooled and K, V packed in one launch
    const long long nblocks = bh * (n / kBlock);
    const int cpb = kBlock * d / (dtype == BF16 ? 8 : 4);
    const long long nblk = cpb >= 1024 ? 1 : 1024 / cpb;
    const long long wgs = (nblocks + nblk - 1) / nblk;
    const dim3 g((unsigned)(wgs < 65536 ? wgs : 65536), 3);
#define MRA_PACK(DT_, D_) pool_pack_kernel<DT_, D_><<<g, threads, 0, stream>>>(q, k, v, qp, kp, vp, kvpacked, nblocks)
    if (dtype == BF16) {
      if (d == 32) MRA_PACK(BF16, 32); else if (d == 64) MRA_PACK(BF16, 64); else MRA_PACK(BF16, 128);
    } else {
      if (d == 32) MRA_PACK(F32, 32); else if (d == 64) MRA_PACK(F32, 64); else MRA_PACK(F32, 128);
    }
#undef MRA_PACK
    return hipGetLastError();
  }
  const int per = dtype == BF16 ? 8 : 4;
  const long long chunks = bh * (n / kBlock) * (d / per);
  const long long blocks = (chunks + threads - 1) / threads;
  dim3 grid((unsigned)blocks, 3);
  if (dtype == BF16)
    pool_kernel<BF16><<<grid, threads, 0, stream>>>(q, k, v, qp, kp, vp, chunks, d);
  else
    pool_kernel<F32><<<grid, threads, 0, stream>>>(q, k, v, qp, kp, vp, chunks, d);
  return hipGetLastError();
}

}  // namespace mra
