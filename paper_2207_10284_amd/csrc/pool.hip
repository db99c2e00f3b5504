// Block means of Q, K, V: the scale-32 rows Q~, K~, V~ of MRA-2
// (Sec. 4.1 eq. recursive_pooling, Sec. 4.3 eq. recursive_pooling_V; five
// pairwise halvings of a 32-row block equal its plain mean).
//
// HBM-bound: every input byte is read once, 1/32 of it is written back.
// Two threads own one 16-byte column chunk of one 32-row block: one sums rows
// 0..15, the other rows 16..31 (each in row order, float32), and the mean is
// (first half + second half) / 32. A wave's load covers whole 128-byte row
// segments, so every HBM line fetched is fully used; two threads per chunk
// keep enough waves in flight to fill the GPU. No LDS, no barriers.
//
// For float32 passes that read packed operands (the forward at d = 128, the
// gradient passes) K and V (and Q, dZ) are also written in the tile kernels'
// matrix-core operand order ("packed", layout in kernels.h), so every operand
// load is one contiguous 1 KB wave access; that configuration pools in one
// launch that stages blocks through LDS so the packed writes stay contiguous.
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
  const int cpr = d / kPer;                        // chunks per row
  // thread t: block t / (2 cpr); within it, half (rows 16 half ..) and chunk
  const long long blk = t / (2 * cpr);
  const int i = (int)(t - blk * 2 * cpr), half = i / cpr, c = i - half * cpr;
  const bool active = t < 2 * chunks;              // whole (block, chunk) pairs: 2 cpr divides 64
  float acc[kPer];
#pragma unroll
  for (int e = 0; e < kPer; ++e) acc[e] = 0.0f;
  if (active) {
    const long long row0 = blk * kBlock + 16 * half;   // all heads flattened
    const u32x4* base = reinterpret_cast<const u32x4*>(x) + row0 * cpr + c;
#pragma unroll 8
    for (int r = 0; r < 16; ++r) {
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
  }
  // the second half's sums, from lane + cpr of the same wave
  float hi[kPer];
#pragma unroll
  for (int e = 0; e < kPer; ++e) hi[e] = __shfl_down(acc[e], cpr);
  if (!active || half != 0) return;
  constexpr float inv = 1.0f / kBlock;             // exact: power of two
  f32x4* out = reinterpret_cast<f32x4*>(y + blk * d + c * kPer);
#pragma unroll
  for (int v = 0; v < kPer / 4; ++v) {
    f32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = (acc[4 * v + e] + hi[4 * v + e]) * inv;
    out[v] = o;
  }
}

// Up to four tensors in one launch (blockIdx.y selects the job): for each,
// the block means (same row order as pool_kernel, so the same bits) and any of
// the two packed copies: the row layout (the "K" part of kvpacked) and the
// transposed layout (the "V" part), layouts in kernels.h. Whole 32-row blocks
// are staged through LDS so that both the reads and the packed writes are
// contiguous 16-byte chunks across lanes.
template <int DT, int D>
__global__ __launch_bounds__(256) void pool_pack_kernel(PackJobs jobs, long long nblocks) {
  using elem = typename std::conditional<DT == BF16, uint16_t, float>::type;
  constexpr int kPer = DT == BF16 ? 8 : 4;         // elements per chunk
  constexpr int CPR = D / kPer;                    // chunks per row
  constexpr int CPB = kBlock * CPR;                // chunks per block
  constexpr int NBLK = CPB >= 1024 ? 1 : 1024 / CPB; // blocks per workgroup pass (16 KB)
  constexpr int NT = D / 32;
  __shared__ __attribute__((aligned(16))) u32x4 tile[NBLK * CPB];
  const elem* te = reinterpret_cast<const elem*>(tile);
  const PackJob job = jobs.job[blockIdx.y];
  const u32x4* src = reinterpret_cast<const u32x4*>(job.src);
  float* pooled = job.pooled;
  u32x4* rowl = reinterpret_cast<u32x4*>(job.row_layout);
  u32x4* tl = reinterpret_cast<u32x4*>(job.t_layout);
  if (src == nullptr) return;                      // empty job (whole workgroup)
  const int tid = threadIdx.x;

  for (long long b0 = (long long)blockIdx.x * NBLK; b0 < nblocks; b0 += (long long)gridDim.x * NBLK) {
    const int nblk = (int)min((long long)NBLK, nblocks - b0);
#pragma unroll
    for (int ci = tid; ci < NBLK * CPB; ci += 256)
      if (ci < nblk * CPB) tile[ci] = src[b0 * CPB + ci];
    __syncthreads();
    // block means: one thread per (block, column chunk); rows 0..15 and
    // 16..31 summed in order, then added (pool_kernel's arithmetic)
    if (pooled != nullptr) {
      for (int pc = tid; pc < nblk * CPR; pc += 256) {
        const int bl = pc / CPR, c = pc % CPR;
        float acc[2][kPer];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int e = 0; e < kPer; ++e) acc[hh][e] = 0.0f;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll 8
          for (int r = 16 * hh; r < 16 * hh + 16; ++r) {
            const u32x4 w = tile[bl * CPB + r * CPR + c];
            if constexpr (DT == BF16) {
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                acc[hh][2 * e] += bf16_to_f32(w[e] & 0xFFFFu);
                acc[hh][2 * e + 1] += bf16_to_f32(w[e] >> 16);
              }
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e) acc[hh][e] += __uint_as_float(w[e]);
            }
          }
        constexpr float inv = 1.0f / kBlock;
        f32x4* out = reinterpret_cast<f32x4*>(pooled + (b0 + bl) * D + c * kPer);
#pragma unroll
        for (int q = 0; q < kPer / 4; ++q) {
          f32x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = (acc[0][4 * q + e] + acc[1][4 * q + e]) * inv;
          out[q] = o;
        }
      }
    }
    // row layout: chunk s*64 + 32h + j holds X[j][(d/2)h + kPer*s .. +kPer-1]
    if (rowl != nullptr) {
#pragma unroll
      for (int oc = tid; oc < NBLK * CPB; oc += 256) {
        if (oc >= nblk * CPB) continue;
        const int bl = oc / CPB, k = oc % CPB;
        const elem* tb = te + bl * kBlock * D;
        const int sk = k / 64, h = (k % 64) / 32, j = k % 32;
        rowl[(b0 + bl) * CPB + k] = *reinterpret_cast<const u32x4*>(tb + j * D + (D / 2) * h + kPer * sk);
      }
    }
    if (tl != nullptr) {
#pragma unroll
      for (int oc = tid; oc < NBLK * CPB; oc += 256) {
        if (oc >= nblk * CPB) continue;
        const int bl = oc / CPB, k = oc % CPB;
        const elem* tb = te + bl * kBlock * D;
        u32x4 o;
        if constexpr (DT == BF16) {
          // chunk (u*NT + t)*64 + 32h + j: X[16u + 8(s/4) + 4h + s%4][32t + j], s = 0..7
          const int u = k / (64 * NT), t = (k / 64) % NT, h = (k % 64) / 32, j = k % 32;
          const int dim = 32 * t + j;
#pragma unroll
          for (int s2 = 0; s2 < 4; ++s2) {
            const int key = 16 * u + 8 * (s2 >> 1) + 4 * h + 2 * (s2 & 1);
            o[s2] = (uint32_t)tb[key * D + dim] | ((uint32_t)tb[(key + 1) * D + dim] << 16);
          }
        } else {
          // chunk (t*4 + a)*64 + 32h + j: X[8a + 4h + kk][32t + j], kk = 0..3
          const int t = k / 256, a = (k / 64) % 4, h = (k % 64) / 32, j = k % 32;
          const int dim = 32 * t + j;
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) o[kk] = __float_as_uint(tb[(8 * a + 4 * h + kk) * D + dim]);
        }
        tl[(b0 + bl) * CPB + k] = o;
      }
    }
    __syncthreads();
  }
}

hipError_t launch_pack(const PackJob* jobs, int njobs, long long bh, int n, int d, int dtype,
                       hipStream_t stream) {
  PackJobs J{};
  for (int i = 0; i < njobs && i < 4; ++i) J.job[i] = jobs[i];
  const long long nblocks = bh * (n / kBlock);
  const int cpb = kBlock * d / (dtype == BF16 ? 8 : 4);
  const long long nblk = cpb >= 1024 ? 1 : 1024 / cpb;
  const long long wgs = (nblocks + nblk - 1) / nblk;
  const dim3 g((unsigned)(wgs < 65536 ? wgs : 65536), (unsigned)njobs);
  // only float32 passes read packed copies (bfloat16 tiles are read raw)
  if (dtype != F32) return hipErrorInvalidValue;
#define MRA_PACK(D_) pool_pack_kernel<F32, D_><<<g, 256, 0, stream>>>(J, nblocks)
  if (d == 32) MRA_PACK(32); else if (d == 64) MRA_PACK(64); else MRA_PACK(128);
#undef MRA_PACK
  return hipGetLastError();
}

hipError_t launch_pool(const void* q, const void* k, const void* v, float* qp, float* kp,
                       float* vp, void* kvpacked, long long bh, int n, int d, int dtype,
                       hipStream_t stream) {
  if (kvpacked != nullptr) {
    // the forward's configuration: Q, K, V pooled and K, V packed in one launch
    const size_t half = (size_t)bh * n * d * (dtype == BF16 ? 2 : 4);
    const PackJob jobs[3] = {{k, kp, kvpacked, nullptr},
                             {v, vp, nullptr, static_cast<char*>(kvpacked) + half},
                             {q, qp, nullptr, nullptr}};
    return launch_pack(jobs, 3, bh, n, d, dtype, stream);
  }
  const int per = dtype == BF16 ? 8 : 4;
  const long long chunks = bh * (n / kBlock) * (d / per);
  const int threads = 256;
  const long long blocks = (2 * chunks + threads - 1) / threads;   // two threads per chunk
  dim3 grid((unsigned)blocks, 3);
  if (dtype == BF16)
    pool_kernel<BF16><<<grid, threads, 0, stream>>>(q, k, v, qp, kp, vp, chunks, d);
  else
    pool_kernel<F32><<<grid, threads, 0, stream>>>(q, k, v, qp, kp, vp, chunks, d);
  return hipGetLastError();
}

// Debug aid (MRA_DEBUG_NANFILL, api.cpp): every 32-bit word of a buffer set to
// one pattern, grid-stride, plain vector stores.
__global__ void fill_u32_kernel(uint32_t* __restrict__ p, long long words, uint32_t pattern) {
  const long long stride = (long long)gridDim.x * blockDim.x;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < words; i += stride) p[i] = pattern;
}

hipError_t launch_fill(void* p, size_t bytes, uint32_t pattern, hipStream_t stream) {
  const long long words = (long long)(bytes / 4);
  if (p == nullptr || words == 0) return hipSuccess;
  const int threads = 256;
  long long blocks = (words + threads - 1) / threads;
  if (blocks > 65536) blocks = 65536;
  fill_u32_kernel<<<(unsigned)blocks, threads, 0, stream>>>(static_cast<uint32_t*>(p), words, pattern);
  return hipGetLastError();
}

}  // namespace mra
