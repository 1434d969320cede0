// The library's one fixed device array: scratch memory for the decode entry
// point that allocates nothing (hswa_decode_noalloc). Its FULL split-KV
// partials live here instead of in a caller workspace.
//
// The array sits in a translation unit of its own, so a device only holds it
// once this entry point has been used there (the code object that defines it
// is loaded on first use); it then stays until the process ends. Host code
// never passes the array's name to a kernel (on the host it is only a stand-in
// for the symbol): the device address comes from hipGetSymbolAddress, looked
// up once per device with that device current, and kernels receive it as an
// ordinary pointer argument.
#include <atomic>

#include "../../include/hswa.h"
#include "hswa_launch.h"

static __device__ __align__(256) unsigned char scratch[HSWA_NOALLOC_SCRATCH_BYTES];

namespace hswa {
namespace {
constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch_ptr[kMaxDevices];
}  // namespace

hipError_t noalloc_scratch(void **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    // two threads may both look it up the first time: same address either way
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return hipSuccess;
}

}  // namespace hswa
