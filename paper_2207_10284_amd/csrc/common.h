// Device helpers shared by the MRA-2 kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace mra {

constexpr int kBlock = 32;          // MRA-2 coarse block size b (R = {32, 1})
constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

enum DType { F32 = 0, BF16 = 1 };

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// float32 -> bfloat16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ int wave_uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Two floats -> packed bf16 pair (lo in bits 0..15).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
}

// op(v, v of lane ^ 32) via the gfx950 half-wave swap (VALU only, no LDS
// round trip). The swap returns this lane's value and its partner's; only a
// symmetric combination of the two is used.
__device__ __forceinline__ float halves_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float halves_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Butterfly all-reduce over the wave without LDS: quad and row permutes (DPP),
// then the 16- and 32-lane swaps of gfx950. Every lane ends with the same value.
template <typename Op>
__device__ __forceinline__ float wave_allreduce(float v, Op op) {
  v = op(v, __uint_as_float(__builtin_amdgcn_mov_dpp(__float_as_uint(v), 0xB1, 0xF, 0xF, true)));   // lane ^ 1
  v = op(v, __uint_as_float(__builtin_amdgcn_mov_dpp(__float_as_uint(v), 0x4E, 0xF, 0xF, true)));   // lane ^ 2
  v = op(v, __uint_as_float(__builtin_amdgcn_mov_dpp(__float_as_uint(v), 0x141, 0xF, 0xF, true)));  // mirror in 8
  v = op(v, __uint_as_float(__builtin_amdgcn_mov_dpp(__float_as_uint(v), 0x140, 0xF, 0xF, true)));  // mirror in 16
  {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = op(__uint_as_float(r[0]), __uint_as_float(r[1]));                                          // rows 0<->1, 2<->3
  }
  {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = op(__uint_as_float(r[0]), __uint_as_float(r[1]));                                          // halves
  }
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
  return wave_allreduce(v, [](float a, float b) { return fmaxf(a, b); });
}

__device__ __forceinline__ float wave_sum(float v) {
  return wave_allreduce(v, [](float a, float b) { return a + b; });
}

// Lanes below this one, as a 64-bit mask.
__device__ __forceinline__ uint64_t lanemask_lt() {
  return (uint64_t(1) << lane_id()) - 1;
}

// A raw buffer resource for `bytes` bytes from `base` (stride 0, 32-bit
// data format). A buffer load returns zero where its vector plus immediate
// offset is at or past `bytes`; the scalar offset is not range-checked.
__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, unsigned bytes) {
  const unsigned long long a = (unsigned long long)base;
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(unsigned)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((a >> 32) & 0xffffu));   // stride 0
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);                    // byte range
  r[3] = 0x00020000;                                                    // 32-bit data format (gfx9)
  return r;
}

// One float (four floats) at byte voffset + soffset of the buffer (zero past
// its range).
__device__ float mra_raw_buffer_load_f32(i32x4 rsrc, int voffset, int soffset,
                                         int aux) __asm("llvm.amdgcn.raw.buffer.load.f32");
__device__ f32x4 mra_raw_buffer_load_f32x4(i32x4 rsrc, int voffset, int soffset,
                                           int aux) __asm("llvm.amdgcn.raw.buffer.load.v4f32");
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ f32x2 mra_raw_buffer_load_f32x2(i32x4 rsrc, int voffset, int soffset,
                                           int aux) __asm("llvm.amdgcn.raw.buffer.load.v2f32");

// Number of set bits of m below this lane (two mbcnt instructions).
__device__ __forceinline__ int bits_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Order-preserving map of a float's bits to uint32 (larger float -> larger
// key). -0.0 is mapped like +0.0 so the two rank equal.
__device__ __forceinline__ uint32_t ordered_key(float s) {
  if (s == 0.0f) s = 0.0f;
  uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup p runs on
// XCD p % 8). Remap so that each XCD receives one contiguous range of logical
// workgroup ids: neighbouring logical workgroups (same head) then share that
// XCD's L2.
__device__ __forceinline__ int xcd_remap(int p, int total) {
  constexpr int kXcd = 8;
  const int xcd = p % kXcd, slot = p / kXcd;
  const int q = total / kXcd, r = total % kXcd;
  return (xcd < r) ? xcd * (q + 1) + slot : r * (q + 1) + (xcd - r) * q + slot;
}

// One XCD's L2. Passes whose per-head working set exceeds it are launched one
// occupancy round at a time (see resident_items).
constexpr size_t kL2PerXcd = (size_t)4 << 20;

// Work items (waves) a launch of `kernel` keeps resident on the current
// device: CUs x workgroups per CU x items per workgroup; 0 if unknown. A
// pass launched this many items at a time starts all of them together, so
// rows that walk their ascending block lists stay in loose step and share the
// XCD's L2; launched whole, later items start as earlier ones finish and
// drift apart.
template <class Kernel>
inline long long resident_items(Kernel kernel, int threads, size_t smem, int items_per_wg) {
  int dev = 0, cus = 0, wgs = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&wgs, kernel, threads, smem) != hipSuccess)
    return 0;
  return (long long)cus * wgs * items_per_wg;
}

// Make LDS writes of this wave visible to the wave's other lanes.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace mra
