// mra_attention_forward_noalloc: the MRA-2 forward of mra_attention_forward
// with its workspace in a file-scope device array instead of a caller's
// buffer, for callers that cannot allocate device memory.
//
// `scratch` is one array per GPU, created when the code object is loaded on
// that GPU and held until the process ends. In host code its name is a
// host-side stand-in, not a device address, so the kernels are never given
// the name itself: on the first call on each device (with that device
// current) hipGetSymbolAddress looks up the array's device address, which is
// kept per device and passed to the kernels like any workspace. The forward
// writes every part of its workspace before reading it, so nothing needs to
// be cleared between calls. Calls that overlap on one GPU share the array and
// race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"
#include "mra.h"

namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;   // MRA_NOALLOC_SCRATCH_BYTES in mra.h
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch_dev[kMaxDevices] = {};                // device address of `scratch` per device

// Device address of this device's copy of `scratch` (looked up once per
// device, with that device current).
mra_status_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return mra::hip_error_status(e);
  if (dev < 0 || dev >= kMaxDevices) return MRA_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return mra::hip_error_status(e);
    if (p == nullptr) return MRA_ERR_UNSUPPORTED;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return MRA_OK;
}

}  // namespace

static_assert(kScratchBytes == MRA_NOALLOC_SCRATCH_BYTES, "mra.h states the scratch size");

extern "C" mra_status_t mra_attention_forward_noalloc(const void* q, const void* k, const void* v,
                                                      void* out, int32_t* idx_out, float* lse_out,
                                                      int B, int H, int n, int d, int block,
                                                      int budget, mra_dtype_t dtype, void* stream) {
  size_t need = 0;
  bool empty = true;
  const mra_status_t st = mra::forward_check(q, k, v, out, idx_out, lse_out, B, H, n, d, block, budget,
                                             dtype, &need, &empty);
  if (st != MRA_OK) return st;
  if (empty) return MRA_OK;
  if (need > kScratchBytes) return MRA_ERR_SCRATCH;
  void* ws = nullptr;
  const mra_status_t sa = scratch_address(&ws);
  if (sa != MRA_OK) return sa;
  return mra::forward_enqueue(q, k, v, out, idx_out, lse_out, ws, B, H, n, d, budget, dtype, stream);
}
