// Library-held scratch for rrs_linear_noalloc: the one entry point that
// allocates nothing, for callers that cannot call hipMalloc (code under HIP
// graph capture, tight serving loops, harnesses that forbid allocation).
//
// The scratch is a file-scope device array. Host code never uses the
// array's name as an address (on the host it is only a stand-in for the
// symbol): the first call on each device, with that device current, asks
// the runtime for the array's device address (hipGetSymbolAddress) and keeps
// it per device; every later use takes that pointer. Each device holds its
// own copy of the array until the process ends.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "rrs_internal.h"

namespace rrs {
namespace {

static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  *ptr = nullptr;
  int dev = 0;
  if (hipError_t e = hipGetDevice(&dev)) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      // `dev` is current: this is its copy of the array.
      if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) return e;
      if (!p) return hipErrorInvalidSymbol;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return hipSuccess;
}

}  // namespace rrs
