// Matrix-core operands and products of one 32x32 tile (v_mfma_f32_32x32x16_bf16;
// 32x32x2_f32 for float32), shared by the forward tile pass and the two
// gradient passes.
//
// Operand layouts (bf16: 8 elements per 16-byte chunk, f32: 4):
//  * Row layout, 32 rows x d: lane (h, j) = (l/32, l%32) holds row j,
//    columns (d/2)h + e*s .. +e-1 in chunk s (KC chunks). Read straight from
//    row-major memory, or from the packed "K layout" (chunk s*64 + lane, 1 KB
//    per chunk and wave).
//  * Transposed layout, d rows x 32 (the A operand of C^T += X^T P^T): the
//    packed "V layout" (kernels.h), VC chunks per lane, which orders the 32
//    contraction indices exactly as the B-operand registers of a tile product
//    hold them.
//  * A product C = A B^T of two row-layout operands leaves, in lane l,
//    column l%32 of C (B's row) and its rows 8(r/4) + 4(l/32) + r%4 in
//    register r. Those 16 values are directly the B operand of the next
//    product over the same index (mfma_acc_*), so weights never move between
//    lanes.
#pragma once

#include "common.h"

namespace mra {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <int DT, int D>
struct TileCfg {
  static constexpr int kWaves = (DT == F32 && D == 128) ? 2 : 4;
  static constexpr int kPitch = DT == BF16 ? 40 : 36;           // LDS row pitch, elements
  static constexpr int kNT = D / 32;                            // output tiles over d
  // 16-byte transposed-layout chunks per lane per tile
  static constexpr int kVChunks = DT == BF16 ? 2 * kNT : 4 * kNT;
  static constexpr int kKChunks = DT == BF16 ? D / 16 : D / 8;  // 16-byte row-layout chunks per lane
  static constexpr int kChunks = kKChunks + kVChunks;           // 1 KB chunks per K/V tile
  using elem = typename std::conditional<DT == BF16, uint16_t, float>::type;
};

// Row j = l%32 of a 32-row block at `rows` (row-major, D columns) in the row
// layout: lane half h reads columns [h*D/2, (h+1)*D/2).
template <int DT, int D>
__device__ __forceinline__ void load_rows(const typename TileCfg<DT, D>::elem* rows,
                                          u32x4 (&f)[TileCfg<DT, D>::kKChunks]) {
  const int lane = lane_id(), j = lane & 31, h = lane >> 5;
  const u32x4* p = reinterpret_cast<const u32x4*>(rows + (long long)j * D + (D / 2) * h);
#pragma unroll
  for (int s = 0; s < TileCfg<DT, D>::kKChunks; ++s) f[s] = p[s];
}

// C = A B^T over the d columns, both in the row layout.
template <int DT, int KC>
__device__ __forceinline__ f32x16 mfma_abt(const u32x4 (&a)[KC], const u32x4 (&b)[KC]) {
  f32x16 s;
#pragma unroll
  for (int r = 0; r < 16; ++r) s[r] = 0.0f;
  if constexpr (DT == BF16) {
#pragma unroll
    for (int k = 0; k < KC; ++k)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[k]),
                                                  __builtin_bit_cast(bf16x8, b[k]), s, 0, 0, 0);
  } else {
#pragma unroll
    for (int k = 0; k < KC; ++k)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        s = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[k][e]), __uint_as_float(b[k][e]), s, 0, 0, 0);
  }
  return s;
}

// o[t] (d rows 32t.., 32 columns) += X^T W for bfloat16 weights pk (two per
// register, in the order of a product's result registers); `xa(c)` yields
// the 16-byte transposed-layout chunk c of X.
template <int NT, class XA>
__device__ __forceinline__ void mfma_acc_bf16(f32x16 (&o)[NT], const uint32_t (&pk)[8], XA xa) {
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const u32x4 pw = {pk[4 * u], pk[4 * u + 1], pk[4 * u + 2], pk[4 * u + 3]};
    const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
      o[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, xa(u * NT + tt)), pb, o[tt], 0, 0, 0);
  }
}

// The same for float32 weights p (one per register).
template <int NT, class XA>
__device__ __forceinline__ void mfma_acc_f32(f32x16 (&o)[NT], const float (&p)[16], XA xa) {
#pragma unroll
  for (int tt = 0; tt < NT; ++tt)
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const u32x4 v4 = xa(tt * 4 + a);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[tt] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(v4[e]), p[4 * a + e], o[tt], 0, 0, 0);
    }
}

// C consecutive 1 KB chunks HBM/L2 -> LDS, 16 bytes per lane each; chunk c is
// addressed through the load's immediate offset, which moves the global and
// the LDS address alike.
template <int C>
__device__ __forceinline__ void load_chunks_lds(const __attribute__((address_space(1))) char* src,
                                                __attribute__((address_space(3))) char* dst) {
  if constexpr (C > 0) {
    load_chunks_lds<C - 1>(src, dst);
    __builtin_amdgcn_global_load_lds(src, dst, 16, (C - 1) * 1024, 0);
  }
}

__device__ __forceinline__ void wait_lds_reads() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// Slot reads are issued as inline assembly: the compiler cannot tell the
// slot's parts apart and, seeing loads in flight into LDS, would wait for all
// of them before any slot read. Here the caller's wait_loads<> covers the part
// being read; lds_done() waits for the reads and ties each value to that wait
// so that no use is scheduled before it.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

template <int OFF>
__device__ __forceinline__ u32x4 lds_read16(uint32_t addr) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF) : "memory");
  return v;
}

// v[i] = chunk C0 + i of a part (chunks 1 KB apart) for this lane, i < C
template <int I, int C, int C0>
struct LdsChunks {
  static __device__ __forceinline__ void run(uint32_t addr, u32x4* v) {
    v[I] = lds_read16<(C0 + I) * 1024>(addr);
    LdsChunks<I + 1, C, C0>::run(addr, v);
  }
};
template <int C, int C0>
struct LdsChunks<C, C, C0> {
  static __device__ __forceinline__ void run(uint32_t, u32x4*) {}
};

template <int C, int C0 = 0>
__device__ __forceinline__ void lds_read_chunks(uint32_t addr, u32x4 (&v)[C]) {
  LdsChunks<0, C, C0>::run(addr, v);
}

template <int C>
__device__ __forceinline__ void lds_done(u32x4 (&v)[C]) {
  wait_lds_reads();
#pragma unroll
  for (int c = 0; c < C; ++c) asm volatile("" : "+v"(v[c]));
}

// gfx950's transposing read (ds_read_b64_tr_b16): within each group of 16
// lanes, lane i receives as value k (k = 0..3) the 16-bit element i%4 of the
// 8 bytes at the address that lane 4k + i/4 of the group supplies.
template <int OFF>
__device__ __forceinline__ u32x2 lds_read_tr16(uint32_t addr) {
  u32x2 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF) : "memory");
  return v;
}

// Two dwords per lane from addr + 256 OFF0 and addr + 256 OFF1 bytes
// (ds_read2st64_b32: offsets in units of 64 dwords).
template <int OFF0, int OFF1>
__device__ __forceinline__ u32x2 lds_read2st64(uint32_t addr) {
  u32x2 v;
  asm volatile("ds_read2st64_b32 %0, %1 offset0:%2 offset1:%3" : "=v"(v) : "v"(addr), "i"(OFF0), "i"(OFF1) : "memory");
  return v;
}

typedef const __attribute__((address_space(1))) char* gptr_t;
typedef __attribute__((address_space(3))) char* lptr_t;

// Raw bfloat16 tiles in LDS (d <= 64): a 32-row tile of consecutive rows
// (2d bytes each) copied with direct-to-LDS loads whose lanes each fetch the
// 16-byte block that belongs at their LDS position under an XOR swizzle F of
// the blocks within a row: block b of row r sits at block b ^ F(r).
// Byte offset of element (r, c) of such a tile in LDS:
template <int D, int (*F)(int)>
__host__ __device__ constexpr int raw_offset(int r, int c) {
  return r * (2 * D) + ((((2 * c) >> 4) ^ F(r)) << 4) + ((2 * c) & 15);
}

// Source byte offset (within the tile) of the 16 bytes lane `lane` copies to
// LDS byte i * 1024 + 16 lane under swizzle F.
template <int D, int (*F)(int)>
__device__ __forceinline__ int raw_copy_offset(int i, int lane) {
  const int q = i * 1024 + 16 * lane, r = q / (2 * D), blk = (q % (2 * D)) / 16;
  return r * (2 * D) + ((blk ^ F(r)) << 4);
}

// Buffer loads straight to LDS (16 bytes per lane): a raw buffer resource for
// `bytes` bytes from `base`, and one load of the 16 bytes at base + soff +
// voff into LDS byte dst + 16 lane. The hardware range check covers the
// vector and immediate offsets only, not the scalar offset, so a load is in
// bounds only because every caller validates the block it copies first (the
// tile passes take only block ids in [0, nb), filtered when the selection is
// staged); the resource's size is not a safety net for the scalar offset.
__device__ void mra_raw_buffer_load_lds(i32x4 rsrc, __attribute__((address_space(3))) void* lds, int size,
                                        int voffset, int soffset, int offset,
                                        int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

__device__ __forceinline__ void buffer_load_lds16(i32x4 rsrc, __attribute__((address_space(3))) char* dst,
                                                  unsigned voff, unsigned soff) {
  mra_raw_buffer_load_lds(rsrc, dst, 16, (int)voff, (int)soff, 0, 0);
}

// The D floats at src (a block's coarse-term vector, used by an epilogue)
// into LDS at dst with direct-to-LDS dword loads, 256 bytes per load (lanes
// past D read zero), so their latency passes during the tiles; a wait for the
// load counter (the tile copies' or one before the epilogue) completes them.
template <int D>
__device__ __forceinline__ void prefetch_vec_lds(const float* src, __attribute__((address_space(3))) char* dst) {
  const i32x4 rs = buffer_rsrc(src, (unsigned)D * (unsigned)sizeof(float));
  const int lane = lane_id();
#pragma unroll
  for (int p = 0; p < (D + 63) / 64; ++p) mra_raw_buffer_load_lds(rs, dst + 256 * p, 4, (lane + 64 * p) * 4, 0, 0, 0);
}
constexpr int add_lds_floats(int d) { return d < 64 ? 64 : d; }

// Copies a list of m block ids into LDS keeping only the entries in [0, nb),
// in their order, and returns how many there are (wave-uniform). Reading the
// ids from LDS keeps them off the vector-memory counter, so prefetched loads
// stay in flight; dropping entries outside [0, nb) here (the padding of a
// head-wide selection, for instance) keeps them out of the loop.
__device__ __forceinline__ int stage_selection(const int32_t* __restrict__ row, int m, int nb,
                                               int32_t* dst) {
  const int lane = lane_id();
  int cnt = 0;
  for (int i0 = 0; i0 < m; i0 += kWave) {
    const int y = i0 + lane < m ? row[i0 + lane] : -1;
    const bool ok = y >= 0 && y < nb;
    const uint64_t mk = __ballot(ok);
    if (ok) dst[cnt + __popcll(mk & lanemask_lt())] = y;
    cnt += __popcll(mk);
  }
  wave_lds_sync();
  return wave_uniform(cnt);
}

}  // namespace mra
