// Library-owned scratch memory for s2moe_verify_moe_noalloc: the SwiGLU
// activations (and, for int4 weights, the fp16 copy of x) live in one
// file-scope device array instead of a caller workspace, so that callers
// that cannot allocate (graph capture, tight serving loops) still get the
// verify pass.  Every GPU the library runs on holds its own copy of the
// array until the process ends.
#include <atomic>

#include "kernels.h"
#include "s2moe.h"

namespace s2moe {

static __device__ __align__(256) unsigned char scratch[S2MOE_NOALLOC_SCRATCH_BYTES];

namespace {

// Device address of `scratch` on each device, looked up once per device
// (hipGetSymbolAddress with that device current).  Host code must use these
// addresses: the array's name on the host is a stand-in, not a device
// pointer.
std::atomic<void*> g_scratch_ptr[64];

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    if (p == nullptr) return hipErrorInvalidSymbol;
    // Concurrent first calls on one device store the same address.
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return hipSuccess;
}

}  // namespace s2moe
