// noalloc.hip -- the library-owned scratch region of the allocation-free
// entry point (cf_conv3d_bwd_weight_noalloc).
//
// The region is a file-scope device array: each GPU the library runs on gets
// its own copy, at its own address, when the code object is loaded there, and
// keeps it until the process ends.  Host code never uses the array's name as
// an address (on the host it is only a stand-in symbol): the device address is
// resolved once per device with hipGetSymbolAddress, with that device
// current, and that pointer is what the kernels receive.

#include "cf_kernels.h"

#include <mutex>

namespace cf {
namespace {

__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
void *g_ptr[kMaxDevices];
hipError_t g_err[kMaxDevices];

}  // namespace

hipError_t noalloc_scratch(void **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::call_once(g_once[dev], [dev] {
    void *p = nullptr;
    g_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_ptr[dev] = g_err[dev] == hipSuccess ? p : nullptr;
  });
  if (g_err[dev] != hipSuccess) return g_err[dev];
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace cf
