// Head-wide selection of Alg. 1 (Sec. 4.2) for R = {b, 1}: pop the `budget`
// blocks with the largest coarse logit S~[x, y] over all nb x nb blocks of a
// head (equal scores: the lower flat index x*nb + y first), among the blocks
// that are not priors; the priors (optionally the diagonal blocks (x, x)) are
// refined in addition. Row x of the output lists its refined column blocks in
// ascending order, followed by -1 up to nb entries.
//
// One workgroup (16 waves) per head. The threshold key T (the budget-th
// largest order-preserving 32-bit key among the non-prior blocks) is found
// with four 8-bit radix passes over the head's scores, each building a
// 256-bin histogram in LDS of the keys that share the digits fixed so far.
// The keys equal to T are taken in flat-index order: per-row counts of such
// keys, an exclusive scan over rows, and a rank inside the row give every one
// its position. A last sweep, one wave per row, compacts the row's refined
// blocks with ballots.
#include "common.h"
#include "kernels.h"

namespace mra {

constexpr int kGWaves = 16;
constexpr int kGThreads = kGWaves * kWave;

__global__ __launch_bounds__(kGThreads) void select_global_kernel(const float* __restrict__ S,
                                                                   int32_t* __restrict__ idx,
                                                                   int nb, int budget,
                                                                   int prior_diagonal) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem);          // [256]
  int* ties = reinterpret_cast<int*>(hist + 256);              // [nb] keys == T per row, then exclusive scan
  int* shared_vals = ties + nb;                                // [4] broadcast slots
  const long long head = blockIdx.x;
  const float* Sh = S + head * (long long)nb * nb;
  int32_t* out = idx + head * (long long)nb * nb;
  const int tid = threadIdx.x;
  const int w = wave_uniform(tid / kWave);
  const int lane = lane_id();
  const long long N = (long long)nb * nb;
  const long long nfree = N - (prior_diagonal ? nb : 0);
  auto is_prior = [&](long long f) { return prior_diagonal && (f / nb) == (f % nb); };

  // ---- threshold: the budget-th largest key among the non-prior blocks
  uint32_t T = 0;
  int need = 0;                        // keys equal to T to take (flat order)
  const bool none = budget == 0, all = (long long)budget >= nfree;
  if (!none && !all) {
    uint32_t prefix = 0;
    int remaining = budget;
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += kGThreads) hist[i] = 0u;
      __syncthreads();
      const uint32_t hi_mask = shift == 24 ? 0u : ~((1u << (shift + 8)) - 1u);
      for (long long f = tid; f < N; f += kGThreads) {
        if (is_prior(f)) continue;
        const uint32_t key = ordered_key(Sh[f]);
        if ((key & hi_mask) == (prefix & hi_mask)) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (w == 0) {
        // lane l holds bins 255-4l .. 252-4l (descending); find the digit
        // where the count of larger-or-equal digits first reaches `remaining`
        uint32_t c[4];
        uint32_t mine = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          c[e] = hist[255 - 4 * lane - e];
          mine += c[e];
        }
        // inclusive prefix over lanes (descending digits)
        uint32_t incl = mine;
        for (int off = 1; off < kWave; off <<= 1) {
          const uint32_t other = __shfl_up(incl, off);
          if (lane >= off) incl += other;
        }
        const uint32_t excl = incl - mine;
        const bool here = excl < (uint32_t)remaining && incl >= (uint32_t)remaining;
        const uint64_t hm = __ballot(here);
        const int src = __builtin_ctzll(hm);                  // exactly one lane
        if (lane == src) {
          uint32_t acc = excl;
          int digit = 0, before = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (acc + c[e] >= (uint32_t)remaining) {
              digit = 255 - 4 * lane - e;
              before = (int)acc;
              break;
            }
            acc += c[e];
          }
          shared_vals[0] = digit;
          shared_vals[1] = before;
        }
      }
      __syncthreads();
      prefix |= (uint32_t)shared_vals[0] << shift;
      remaining -= shared_vals[1];
      __syncthreads();                                       // slots reused by the next pass
    }
    T = prefix;
    need = remaining;                                        // >= 1
    // keys equal to T per row, then their exclusive scan over rows
    for (int i = tid; i < nb; i += kGThreads) ties[i] = 0;
    __syncthreads();
    for (long long f = tid; f < N; f += kGThreads)
      if (!is_prior(f) && ordered_key(Sh[f]) == T) atomicAdd(&ties[f / nb], 1);
    __syncthreads();
    if (w == 0) {
      const int per = (nb + kWave - 1) / kWave;               // rows per lane, contiguous
      int mine = 0;
      for (int r = lane * per; r < min(nb, (lane + 1) * per); ++r) mine += ties[r];
      int incl = mine;
      for (int off = 1; off < kWave; off <<= 1) {
        const int other = __shfl_up(incl, off);
        if (lane >= off) incl += other;
      }
      int run = incl - mine;
      for (int r = lane * per; r < min(nb, (lane + 1) * per); ++r) {
        const int t = ties[r];
        ties[r] = run;
        run += t;
      }
    }
    __syncthreads();
  }

  // ---- rows: one wave per row, blocks in ascending order
  for (int x = w; x < nb; x += kGWaves) {
    const float* row = Sh + (long long)x * nb;
    int32_t* orow = out + (long long)x * nb;
    int written = 0, tie_seen = (!none && !all) ? ties[x] : 0;
    for (int y0 = 0; y0 < nb; y0 += kWave) {
      const int y = y0 + lane;
      const bool valid = y < nb;
      const bool prior = valid && prior_diagonal && y == x;
      const bool cand = valid && !prior && !none && !all;    // decided by the threshold
      const uint32_t key = cand ? ordered_key(row[y]) : 0u;
      const bool eq = cand && key == T;
      const uint64_t em = __ballot(eq);                      // whole wave: tie_seen stays uniform
      const int rank = tie_seen + __popcll(em & lanemask_lt());
      tie_seen += __popcll(em);
      const bool take = prior || (valid && !prior && all) || (cand && (key > T || (eq && rank < need)));
      const uint64_t tm = __ballot(take);
      if (take) orow[written + __popcll(tm & lanemask_lt())] = y;
      written += __popcll(tm);
    }
    for (int i = written + lane; i < nb; i += kWave) orow[i] = -1;
  }
}

hipError_t launch_select_global(const float* S, int32_t* idx, long long bh, int nb, int budget,
                                int prior_diagonal, hipStream_t stream) {
  const size_t smem = (256 + (size_t)nb + 4) * sizeof(int);
  select_global_kernel<<<(unsigned)bh, kGThreads, smem, stream>>>(S, idx, nb, budget,
                                                                   prior_diagonal);
  return hipGetLastError();
}

}  // namespace mra
