// wbmm_backward_noalloc: the fused backward with the table-gradient scratch
// (the per-slab partial sums) in a static device buffer of this library, for
// callers that cannot allocate device memory.
//
// The buffer `scratch` is a device-side array: in host code its name is only
// a host-side stand-in.  Its device address is looked up once per device
// (hipGetSymbolAddress with that device current) and only that address is
// ever handed to kernels.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "wbmm.h"
#include "wbmm_internal.h"

namespace {

constexpr size_t kScratchBytes = WBMM_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void *g_scratch[kMaxDevices];  // device address of `scratch` per device; null until looked up

// Device address of this device's scratch (looked up on first use).
hipError_t scratch_address(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[dev] == nullptr) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

extern "C" wbmm_status wbmm_backward_noalloc(const void *x, const void *dy, const void *table, void *dx,
                                             float *dtable, int64_t B, int64_t C, int64_t H, int64_t W, int w,
                                             wbmm_dtype dtype, void *stream) {
  wbmm::Geom g;
  int64_t bytes = 0;
  wbmm_status s = wbmm::check_backward_args(x, dy, table, dx, dtable, B, C, H, W, w, dtype, &g, &bytes);
  if (s != WBMM_OK) return s;
  const size_t need = wbmm::dtable_workspace_bytes((wbmm::Dt)dtype, g);
  if (need > kScratchBytes) return WBMM_ERR_SCRATCH;
  hipStream_t st = (hipStream_t)stream;
  void *ws = nullptr;
  // the partial sums are written before they are read within the call, so
  // the buffer needs no clearing
  if (need > 0 && scratch_address(&ws) != hipSuccess) return WBMM_ERR_HIP;
  return wbmm::launch_backward((wbmm::Dt)dtype, x, dy, table, dx, dtable, ws, g, st) == hipSuccess ? WBMM_OK
                                                                                                  : WBMM_ERR_HIP;
}
