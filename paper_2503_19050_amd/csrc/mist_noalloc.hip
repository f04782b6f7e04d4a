// Device scratch of the allocation-free entry point (mist_eval_ids_noalloc): a fixed,
// file-scope device array, so that the entry point needs no device allocation at all.  Every
// GPU the library runs on holds its own copy of the array until the process ends.

#include <hip/hip_runtime.h>

#include <mutex>

#include "mist_internal.h"

namespace mist {
namespace {

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_ptr[kMaxDevices] = {};  // device address of scratch, per device (nullptr: not looked up yet)

}  // namespace

// The current device's address of the scratch array.  The array's name is a host-side stand-in
// in host code, not a device address: the address is looked up once per device (with that
// device current) and kept; callers use only the returned pointer.
__attribute__((visibility("hidden"))) int noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return 0;
}

}  // namespace mist
