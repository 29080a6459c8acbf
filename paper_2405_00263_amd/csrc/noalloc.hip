// Allocation-free entry point: clover_op_linear with its split-K partials in a device array
// the library owns, for callers that cannot allocate device memory (code under HIP graph
// capture, serving loops that forbid allocation).
//
// The array `scratch` below lives in the code object: every GPU the library runs on holds
// its own copy from the first launch until the process ends.  Host code cannot use the
// array's name as a device address (in host code it names a host-side stand-in), so the
// first call on each device looks its device address up with hipGetSymbolAddress, with that
// device current, and keeps it per device; every launch then takes that pointer.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/clover.h"
#include "kernels.h"

static constexpr size_t kScratchBytes = size_t(16) << 20;  // 16 MiB per device

static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// The device address of this device's copy of `scratch`, looked up once per device.
hipError_t scratch_ptr(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

size_t clover_op_linear_noalloc_max_bytes(void) { return kScratchBytes; }

clover_status clover_op_linear_noalloc(int32_t dtype, const void* X, int32_t M, int32_t K, const void* Wp,
                                       int32_t N, float* Y, void* hip_stream) {
  const size_t need = clover_op_scratch_bytes(dtype, M, N, K);
  if (!need || !X || !Wp || !Y) {
    clover::set_last_error("op_linear_noalloc: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  if (need > kScratchBytes) {
    clover::set_last_error("op_linear_noalloc: the split-K partials of this shape need more than the "
                           "16 MiB device scratch array");
    return CLOVER_ERR_CAPACITY;
  }
  void* p = nullptr;
  const hipError_t e = scratch_ptr(&p);
  if (e != hipSuccess) {
    clover::set_last_error("op_linear_noalloc: hipGetSymbolAddress failed");
    return CLOVER_ERR_DEVICE;
  }
  return clover_op_linear(dtype, X, M, K, Wp, N, Y, p, kScratchBytes, hip_stream);
}

}  // extern "C"
