// Scratch memory of the entry point that allocates nothing (kv_window_mu_sigma_noalloc): one
// file-scope device array of kNoAllocScratchBytes, which every GPU the library runs on holds until
// the process ends.  In host code `scratch` names a host-side stand-in, not device memory: its
// device address is looked up once per device (with that device current) and only that address is
// handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

namespace kv {
namespace {

constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

void* g_scratch_dev[kMaxDevices];  // device address of `scratch` on each device, once looked up
std::mutex g_scratch_mutex;

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_dev[dev] = p;
  }
  *ptr = g_scratch_dev[dev];
  return hipSuccess;
}

}  // namespace kv
