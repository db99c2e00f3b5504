// Head-wide selection of Alg. 1 (Sec. 4.2) for R = {b, 1}: pop the `budget`
// blocks with the largest coarse logit S~[x, y] over all nb x nb blocks of a
// head (equal scores: the lower flat index x*nb + y first), among the blocks
// that are not priors; the priors (optionally the diagonal blocks (x, x)) are
// refined in addition. Row x of the output lists its refined column blocks in
// ascending order, followed by -1 up to nb entries.
//
// One workgroup (16 waves) per head. The threshold key T (the budget-th
// largest order-preserving 32-bit key among the non-prior blocks) is found
// with radix passes over the head's scores, each building a histogram in LDS
// of the keys that share the digits fixed so far: heads of up to 256 x 256
// blocks keep their keys in registers, whole rows per wave (so the ties are
// counted and the rows compacted without reading S again), and take digits of
// 12, 10 and 10 bits; larger heads take four 8-bit digits over many
// workgroups.
// The keys equal to T are taken in flat-index order: per-row counts of such
// keys, an exclusive scan over rows, and a rank inside the row give every one
// its position. A last sweep, one wave per row, compacts the row's refined
// blocks with ballots.
#include "common.h"
#include "kernels.h"

namespace mra {

constexpr int kGWaves = 16;
constexpr int kGThreads = kGWaves * kWave;

// The digit of the `remaining`-th largest key from a 256-bin histogram (wave
// 0; lane l holds bins 255-4l .. 252-4l, descending) into shared_vals[0] and
// the count of larger digits into shared_vals[1].
__device__ __forceinline__ void pick_digit(const uint32_t* hist, int remaining, int lane, int* shared_vals) {
  uint32_t c[4];
  uint32_t mine = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    c[e] = hist[255 - 4 * lane - e];
    mine += c[e];
  }
  uint32_t incl = mine;                                      // inclusive prefix over lanes
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t other = __shfl_up(incl, off);
    if (lane >= off) incl += other;
  }
  const uint32_t excl = incl - mine;
  const bool here = excl < (uint32_t)remaining && incl >= (uint32_t)remaining;
  const uint64_t hm = __ballot(here);
  const int src = __builtin_ctzll(hm);                       // exactly one lane
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

// Exclusive scan of ties[0 .. nb) in place (wave 0; contiguous rows per lane).
__device__ __forceinline__ void scan_rows(int* ties, int nb, int lane) {
  const int per = (nb + kWave - 1) / kWave;
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

// Register tier: digits of 12, 10 and 10 bits (shifts 20, 10, 0). The top
// 8 bits of an order-preserving key are the sign and most of the exponent,
// which logits of one head share, so a histogram over them puts most keys of
// a wave into one or two bins and the LDS atomics serialize; 12 bits reach
// into the mantissa and spread the first pass over many bins.
constexpr int kGBins = 4096;

// The digit of the `remaining`-th largest key of the histogram hist[0 .. bins)
// (bins = 4096 or 1024; all threads of the workgroup): thread t sums bins
// bins-1-t*per .. bins-(t+1)*per (descending), a scan over threads finds the
// one holding the remaining-th key, which writes the digit to shared_vals[0]
// and the count of larger digits to shared_vals[1]. wave_tot: 16 ints.
__device__ __forceinline__ void pick_digit_block(const uint32_t* hist, int bins, int remaining, int tid, int w,
                                                 int lane, int* wave_tot, int* shared_vals) {
  const int per = bins / kGThreads;                            // 4 or 1
  const int top = bins - 1 - tid * per;
  uint32_t c[4] = {0u, 0u, 0u, 0u};
  uint32_t mine = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (e < per) {
      c[e] = hist[top - e];
      mine += c[e];
    }
  uint32_t incl = mine;                                        // inclusive prefix within the wave
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t other = __shfl_up(incl, off);
    if (lane >= off) incl += other;
  }
  if (lane == kWave - 1) wave_tot[w] = (int)incl;
  __syncthreads();
  uint32_t base = 0;
  for (int q = 0; q < w; ++q) base += (uint32_t)wave_tot[q];
  const uint32_t excl = base + incl - mine, incl_all = base + incl;
  if (excl < (uint32_t)remaining && incl_all >= (uint32_t)remaining) {   // exactly one thread
    uint32_t acc = excl;
    int digit = 0, before = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (e < per && acc + c[e] >= (uint32_t)remaining) {
        digit = top - e;
        before = (int)acc;
        break;
      }
      acc += c[e];
    }
    shared_vals[0] = digit;
    shared_vals[1] = before;
  }
  __syncthreads();
}

// Heads of up to 16 RW rows and 64 CW columns: wave w keeps the keys of rows
// x = w + 16 i (i < RW), columns y = lane + 64 c (c < CW) in registers, read
// from S once; the radix passes count them into one histogram, the rows' ties
// are counted with ballots and the rows are compacted from the same
// registers.
template <int RW, int CW>
__global__ __launch_bounds__(kGThreads) void select_global_rows_kernel(const float* __restrict__ S,
                                                                        int32_t* __restrict__ idx,
                                                                        int nb, int budget,
                                                                        int prior_diagonal) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem);          // [kGBins] histogram of the current digit
  int* ties = reinterpret_cast<int*>(hist + kGBins);           // [nb] keys == T per row, then exclusive scan
  int* shared_vals = ties + nb;                                // [4] broadcast slots
  int* wave_tot = shared_vals + 4;                             // [16] per-wave sums of the digit pick
  const long long head = blockIdx.x;
  const float* Sh = S + head * (long long)nb * nb;
  int32_t* out = idx + head * (long long)nb * nb;
  const int tid = threadIdx.x;
  const int w = wave_uniform(tid / kWave);
  const int lane = lane_id();
  const long long nfree = (long long)nb * nb - (prior_diagonal ? nb : 0);
  const bool none = budget == 0, all = (long long)budget >= nfree;

  // key 0: a block that does not take part (a prior, or outside the head);
  // every finite score's key is at least 0x00800000. The loads are
  // unconditional (outside the head: element 0) so that all of them are in
  // flight before the first is used.
  uint32_t key[RW][CW];
#pragma unroll
  for (int i = 0; i < RW; ++i) {
    const int x = w + kGWaves * i;
#pragma unroll
    for (int c = 0; c < CW; ++c) {
      const int y = lane + kWave * c;
      const bool inside = x < nb && y < nb;
      key[i][c] = __float_as_uint(Sh[inside ? (long long)x * nb + y : 0ll]);
    }
  }
#pragma unroll
  for (int i = 0; i < RW; ++i) {
    const int x = w + kGWaves * i;
#pragma unroll
    for (int c = 0; c < CW; ++c) {
      const int y = lane + kWave * c;
      const bool in = x < nb && y < nb && !(prior_diagonal && x == y);
      key[i][c] = in ? ordered_key(__uint_as_float(key[i][c])) : 0u;
    }
  }

  uint32_t T = 0;
  int need = 0;                        // keys equal to T to take (flat order)
  if (!none && !all) {
    uint32_t prefix = 0;
    int remaining = budget;
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      const int shift = p == 0 ? 20 : (p == 1 ? 10 : 0);
      const int bins = p == 0 ? kGBins : 1024;
      const uint32_t hi_mask = p == 0 ? 0u : ~((1u << (shift + (p == 0 ? 12 : 10))) - 1u);
      for (int i = tid; i < bins; i += kGThreads) hist[i] = 0u;
      __syncthreads();
#pragma unroll
      for (int i = 0; i < RW; ++i)
#pragma unroll
        for (int c = 0; c < CW; ++c)
          if (key[i][c] != 0u && (key[i][c] & hi_mask) == (prefix & hi_mask))
            atomicAdd(&hist[(key[i][c] >> shift) & (uint32_t)(bins - 1)], 1u);
      __syncthreads();
      pick_digit_block(hist, bins, remaining, tid, w, lane, wave_tot, shared_vals);
      prefix |= (uint32_t)shared_vals[0] << shift;
      remaining -= shared_vals[1];
      __syncthreads();                                       // slots reused by the next pass
    }
    T = prefix;
    need = remaining;                                        // >= 1
    // keys equal to T per row (ballots), then their exclusive scan over rows
#pragma unroll
    for (int i = 0; i < RW; ++i) {
      const int x = w + kGWaves * i;
      int t = 0;
#pragma unroll
      for (int c = 0; c < CW; ++c) t += __popcll(__ballot(key[i][c] == T));   // T > 0: never key 0
      if (x < nb && lane == 0) ties[x] = t;
    }
    __syncthreads();
    if (w == 0) scan_rows(ties, nb, lane);
    __syncthreads();
  }

  // ---- rows: compacted from the registers, blocks in ascending order. A
  // budget of zero takes the priors only, one of every free block takes the
  // whole head; otherwise T is a key of a finite score (at least 0x00800000),
  // so key 0 (a prior, or outside the head) is never above or equal to it and
  // a row takes its keys above T, those equal to T whose flat rank is below
  // `need`, and its prior (column px).
#pragma unroll
  for (int i = 0; i < RW; ++i) {
    const int x = w + kGWaves * i;
    if (x >= nb) break;
    int32_t* orow = out + (long long)x * nb;
    const int px = prior_diagonal ? x : -1;
    int written = 0;
    if (none || all) {
#pragma unroll
      for (int c = 0; c < CW; ++c) {
        const int y = lane + kWave * c;
        const bool take = all ? y < nb : y == px;
        const uint64_t tm = __ballot(take);
        if (take) orow[written + bits_below(tm)] = y;
        written += __popcll(tm);
      }
    } else {
      int tie_seen = ties[x];
#pragma unroll
      for (int c = 0; c < CW; ++c) {
        const int y = lane + kWave * c;
        const bool eq = key[i][c] == T;
        const uint64_t em = __ballot(eq);
        const int rank = tie_seen + bits_below(em);
        const bool take = (key[i][c] > T) | (y == px) | (eq & (rank < need));   // no short circuits
        tie_seen += __popcll(em);
        const uint64_t tm = __ballot(take);
        if (take) orow[written + bits_below(tm)] = y;
        written += __popcll(tm);
      }
    }
#pragma unroll
    for (int c = 0; c < CW; ++c) {
      const int k = lane + kWave * c;
      if (k >= written && k < nb) orow[k] = -1;
    }
  }
}

// Heads of more than 256 blocks per side: the four radix passes, the ties per
// row and the compaction run as separate launches over many workgroups per
// head (one workgroup per head would take milliseconds at 1024 x 1024
// blocks). Scratch per head in the first words of its own idx output
// (written last, by the compaction, after everything was read): the four
// 256-bin histograms, then the ties per row. Every launch recomputes the
// digits chosen so far from the histograms of the earlier passes, so no
// other state is kept.
constexpr int kSgThreads = 256;
constexpr int kSgKeysPerThread = 16;
constexpr int kSgTies = 4 * 256;                              // word offset of the ties per row
constexpr int kSgBatch = 4;                                    // row loads in flight per wave

// prefix and remaining count after `passes` digits (wave 0 of the workgroup;
// the result broadcast through shared_vals[2..3]).
__device__ __forceinline__ void digits_so_far(const uint32_t* hists, int passes, int budget, int w, int lane,
                                              int* shared_vals) {
  if (w == 0) {
    uint32_t prefix = 0;
    int remaining = budget;
    for (int p = 0; p < passes; ++p) {
      pick_digit(hists + 256 * p, remaining, lane, shared_vals);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      prefix |= (uint32_t)shared_vals[0] << (24 - 8 * p);
      remaining -= shared_vals[1];
      __builtin_amdgcn_wave_barrier();
    }
    if (lane == 0) {
      shared_vals[2] = (int)prefix;
      shared_vals[3] = remaining;
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(kSgThreads) void sg_zero_kernel(int32_t* __restrict__ idx, long long N) {
  uint32_t* h = reinterpret_cast<uint32_t*>(idx + blockIdx.x * N);
  for (int i = threadIdx.x; i < 4 * 256; i += kSgThreads) h[i] = 0u;
}

// Pass `pass` (digit bits 24 - 8 pass ..): every workgroup counts the keys of
// its slice that carry the digits chosen so far into histogram `pass`.
__global__ __launch_bounds__(kSgThreads) void sg_pass_kernel(const float* __restrict__ S, int32_t* __restrict__ idx,
                                                             int nb, int budget, int prior_diagonal, int pass) {
  __shared__ uint32_t hist[256];
  __shared__ int shared_vals[4];
  const long long N = (long long)nb * nb;
  const long long head = blockIdx.y;
  const float* Sh = S + head * N;
  uint32_t* hists = reinterpret_cast<uint32_t*>(idx + head * N);
  const int tid = threadIdx.x, w = tid / kWave, lane = lane_id();
  for (int i = tid; i < 256; i += kSgThreads) hist[i] = 0u;
  digits_so_far(hists, pass, budget, w, lane, shared_vals);
  const uint32_t prefix = (uint32_t)shared_vals[2];
  const int shift = 24 - 8 * pass;
  const uint32_t hi_mask = pass == 0 ? 0u : ~((1u << (shift + 8)) - 1u);
  const long long f0 = (long long)blockIdx.x * kSgThreads * kSgKeysPerThread;
  float v[kSgKeysPerThread];                                   // all loads in flight first
#pragma unroll
  for (int r = 0; r < kSgKeysPerThread; ++r) {
    const long long f = f0 + tid + (long long)kSgThreads * r;
    v[r] = Sh[f < N ? f : 0ll];
  }
  // block (x, y) of flat index f, stepped along with f (nb > kSgThreads here,
  // so a step wraps at most once)
  const long long fs = f0 + tid;
  int x = (int)(fs / nb), y = (int)(fs - (long long)x * nb);
#pragma unroll
  for (int r = 0; r < kSgKeysPerThread; ++r) {
    const long long f = fs + (long long)kSgThreads * r;
    if (f < N && !(prior_diagonal && x == y)) {
      const uint32_t k = ordered_key(v[r]);
      if ((k & hi_mask) == (prefix & hi_mask)) atomicAdd(&hist[(k >> shift) & 255u], 1u);
    }
    y += kSgThreads;
    if (y >= nb) {
      y -= nb;
      ++x;
    }
  }
  __syncthreads();
  for (int i = tid; i < 256; i += kSgThreads)
    if (hist[i] != 0u) atomicAdd(&hists[256 * pass + i], hist[i]);
}

// The keys equal to the threshold per row (one wave per row).
__global__ __launch_bounds__(kSgThreads) void sg_ties_kernel(const float* __restrict__ S, int32_t* __restrict__ idx,
                                                             int nb, int budget, int prior_diagonal) {
  __shared__ int shared_vals[4];
  const long long N = (long long)nb * nb;
  const long long head = blockIdx.y;
  const float* Sh = S + head * N;
  uint32_t* hists = reinterpret_cast<uint32_t*>(idx + head * N);
  const int tid = threadIdx.x, w = tid / kWave, lane = lane_id();
  digits_so_far(hists, 4, budget, w, lane, shared_vals);
  const uint32_t T = (uint32_t)shared_vals[2];
  const int x = blockIdx.x * (kSgThreads / kWave) + w;
  if (x >= nb) return;
  const float* row = Sh + (long long)x * nb;
  int t = 0;
  for (int y0 = 0; y0 < nb; y0 += kSgBatch * kWave) {
    float v[kSgBatch];                                         // a batch of loads in flight
#pragma unroll
    for (int j = 0; j < kSgBatch; ++j) {
      const int y = y0 + kWave * j + lane;
      v[j] = row[y < nb ? y : 0];
    }
#pragma unroll
    for (int j = 0; j < kSgBatch; ++j) {
      const int y = y0 + kWave * j + lane;
      const bool cand = y < nb && !(prior_diagonal && y == x);
      t += __popcll(__ballot(cand && ordered_key(v[j]) == T));
    }
  }
  if (lane == 0) reinterpret_cast<int*>(hists)[kSgTies + x] = t;
}

// Compaction of row x (one wave): priors, every key above the threshold T,
// and the keys equal to T whose flat rank (tie_before: such keys in earlier
// rows) is below `need`; then -1 up to nb entries.
__device__ __forceinline__ void compact_row(const float* __restrict__ row, int32_t* __restrict__ orow, int x, int nb,
                                            bool prior_diagonal, bool none, bool all, uint32_t T, int need,
                                            int tie_before, int lane) {
  int written = 0, tie_seen = tie_before;
  for (int y0 = 0; y0 < nb; y0 += kSgBatch * kWave) {
    float v[kSgBatch];                                         // a batch of loads in flight
#pragma unroll
    for (int j = 0; j < kSgBatch; ++j) {
      const int y = y0 + kWave * j + lane;
      v[j] = row[y < nb ? y : 0];
    }
#pragma unroll
    for (int j = 0; j < kSgBatch; ++j) {
      const int y = y0 + kWave * j + lane;
      const bool valid = y < nb;
      const bool prior = valid && prior_diagonal && y == x;
      const bool cand = valid && !prior && !none && !all;
      const uint32_t key = cand ? ordered_key(v[j]) : 0u;
      const bool eq = cand && key == T;
      const uint64_t em = __ballot(eq);
      const int rank = tie_seen + bits_below(em);
      tie_seen += __popcll(em);
      const bool take = prior | (valid & all) | (cand & ((key > T) | (eq & (rank < need))));
      const uint64_t tm = __ballot(take);
      if (take) orow[written + bits_below(tm)] = y;
      written += __popcll(tm);
    }
  }
  for (int i = written + lane; i < nb; i += kWave) orow[i] = -1;
}

// Rows that hold no scratch (x >= first): one wave per row; the row's tie
// offset is the sum of the ties of the rows before it.
__global__ __launch_bounds__(kSgThreads) void sg_rows_kernel(const float* __restrict__ S, int32_t* __restrict__ idx,
                                                             int nb, int budget, int prior_diagonal, int first) {
  __shared__ int shared_vals[4];
  const long long N = (long long)nb * nb;
  const long long head = blockIdx.y;
  int32_t* out = idx + head * N;
  const uint32_t* hists = reinterpret_cast<const uint32_t*>(out);
  const int tid = threadIdx.x, w = tid / kWave, lane = lane_id();
  const long long nfree = N - (prior_diagonal ? nb : 0);
  const bool none = budget == 0, all = (long long)budget >= nfree;
  uint32_t T = 0;
  int need = 0;
  if (!none && !all) {
    digits_so_far(hists, 4, budget, w, lane, shared_vals);
    T = (uint32_t)shared_vals[2];
    need = shared_vals[3];
  }
  const int x = first + blockIdx.x * (kSgThreads / kWave) + w;
  if (x >= nb) return;
  int before = 0;
  if (!none && !all) {
    const int* ties = reinterpret_cast<const int*>(hists) + kSgTies;
    for (int r = lane; r < x; r += kWave) before += ties[r];
    before = (int)wave_sum((float)before);                   // exact: counts below 2^24
  }
  compact_row(S + head * N + (long long)x * nb, out + (long long)x * nb, x, nb, prior_diagonal, none, all, T, need,
              before, lane);
}

// The rows that hold the scratch (x < first), one workgroup per head, which
// reads all the scratch it needs before writing a row.
__global__ __launch_bounds__(kSgThreads) void sg_first_rows_kernel(const float* __restrict__ S,
                                                                   int32_t* __restrict__ idx, int nb, int budget,
                                                                   int prior_diagonal, int first) {
  __shared__ int shared_vals[4];
  __shared__ int before_all[kSgThreads / kWave * 8];
  const long long N = (long long)nb * nb;
  const long long head = blockIdx.x;
  int32_t* out = idx + head * N;
  const uint32_t* hists = reinterpret_cast<const uint32_t*>(out);
  const int tid = threadIdx.x, w = tid / kWave, lane = lane_id();
  const long long nfree = N - (prior_diagonal ? nb : 0);
  const bool none = budget == 0, all = (long long)budget >= nfree;
  uint32_t T = 0;
  int need = 0;
  if (!none && !all) {
    digits_so_far(hists, 4, budget, w, lane, shared_vals);
    T = (uint32_t)shared_vals[2];
    need = shared_vals[3];
    const int* ties = reinterpret_cast<const int*>(hists) + kSgTies;
    for (int x = w; x < first; x += kSgThreads / kWave) {
      int before = 0;
      for (int r = lane; r < x; r += kWave) before += ties[r];
      before = (int)wave_sum((float)before);
      if (lane == 0) before_all[x] = before;
    }
  }
  __syncthreads();                                             // all scratch read: its rows may be written
  for (int x = w; x < first; x += kSgThreads / kWave)
    compact_row(S + head * N + (long long)x * nb, out + (long long)x * nb, x, nb, prior_diagonal, none, all, T, need,
                (!none && !all) ? before_all[x] : 0, lane);
}

hipError_t launch_select_global(const float* S, int32_t* idx, long long bh, int nb, int budget,
                                int prior_diagonal, hipStream_t stream) {
  const size_t tail = ((size_t)nb + 4 + kGWaves) * sizeof(int);
  const size_t hist16 = (size_t)kGBins * sizeof(int);
#define MRA_SG_ROWS(RW, CW) \
  select_global_rows_kernel<RW, CW><<<(unsigned)bh, kGThreads, hist16 + tail, stream>>>(S, idx, nb, budget, prior_diagonal)
  if (nb <= 16) MRA_SG_ROWS(1, 1);
  else if (nb <= 32) MRA_SG_ROWS(2, 1);
  else if (nb <= 64) MRA_SG_ROWS(4, 1);
  else if (nb <= 128) MRA_SG_ROWS(8, 2);
  else if (nb <= 256) MRA_SG_ROWS(16, 4);
  else {
    // heads of more than 256 blocks per side: passes spread over workgroups
    const long long N = (long long)nb * nb;
    const long long nfree = N - (prior_diagonal ? nb : 0);
    if (budget > 0 && (long long)budget < nfree) {
      const unsigned slices = (unsigned)((N + (long long)kSgThreads * kSgKeysPerThread - 1) /
                                         ((long long)kSgThreads * kSgKeysPerThread));
      sg_zero_kernel<<<(unsigned)bh, kSgThreads, 0, stream>>>(idx, N);
      for (int pass = 0; pass < 4; ++pass)
        sg_pass_kernel<<<dim3(slices, (unsigned)bh), kSgThreads, 0, stream>>>(S, idx, nb, budget, prior_diagonal,
                                                                            pass);
      const unsigned tiegroups = (unsigned)((nb + kSgThreads / kWave - 1) / (kSgThreads / kWave));
      sg_ties_kernel<<<dim3(tiegroups, (unsigned)bh), kSgThreads, 0, stream>>>(S, idx, nb, budget, prior_diagonal);
    }
    // rows holding the scratch (its first kSgTies + nb words) are written last
    const int first = (kSgTies + nb + nb - 1) / nb;
    const unsigned rowgroups = (unsigned)((nb - first + kSgThreads / kWave - 1) / (kSgThreads / kWave));
    sg_rows_kernel<<<dim3(rowgroups, (unsigned)bh), kSgThreads, 0, stream>>>(S, idx, nb, budget, prior_diagonal,
                                                                            first);
    sg_first_rows_kernel<<<(unsigned)bh, kSgThreads, 0, stream>>>(S, idx, nb, budget, prior_diagonal, first);
  }
#undef MRA_SG_ROWS
  return hipGetLastError();
}

}  // namespace mra
