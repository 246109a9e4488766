// Device scratch of the entry point that allocates nothing (lora_apply_noalloc):
// one fixed array per GPU, in the code object.  Its address on a device comes
// from hipGetSymbolAddress, taken once per device with that device current;
// host code uses only that address (the array's name in host code is a
// host-side stand-in, not device memory).
#include <hip/hip_runtime.h>

#include <mutex>

#include "lora_internal.h"

static __device__ __align__(256) unsigned char scratch[LORA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int SCRATCH_DEVICES = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[SCRATCH_DEVICES] = {};

}  // namespace

namespace lora {

hipError_t noalloc_scratch(hipStream_t stream, void** out) {
  *out = nullptr;
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  int dev = cur;
  if (stream != nullptr && (e = hipStreamGetDevice(stream, &dev)) != hipSuccess) return e;
  if (dev < 0 || dev >= SCRATCH_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) {
      const hipError_t r = hipSetDevice(cur);
      if (e == hipSuccess) e = r;
    }
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace lora
