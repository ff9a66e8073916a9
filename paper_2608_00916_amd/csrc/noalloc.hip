// Static scratch of the allocation-free forward (moe_fwd_noalloc): a
// file-scope device array that each GPU the library runs on holds until the
// process ends.  Host code never uses the array's name as an address (on the
// host it is only a stand-in for the symbol): the device address is looked up
// once per device, with that device current, and cached.
#include <hip/hip_runtime.h>

#include <mutex>

#include "launch.hpp"

static __device__ __align__(256) unsigned char scratch[MOE_NOALLOC_SCRATCH_BYTES];

namespace moe {

namespace {
constexpr int kMaxDevices = 64;
}

hipError_t static_scratch(void** ptr, size_t* bytes) {
  static std::mutex lock;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> guard(lock);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  *bytes = MOE_NOALLOC_SCRATCH_BYTES;
  return hipSuccess;
}

}  // namespace moe
