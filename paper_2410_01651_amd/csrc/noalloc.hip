// Device scratch memory of the allocation-free forward (gca_forward_noalloc).
//
// The array lives in the library's code object: every device that runs the
// library holds its own copy, at its own address, until the process ends.  Host
// code never passes the array's name to a kernel (on the host that name is a
// stand-in, not a device address); it looks the device address up once per
// device and passes that.
#include <hip/hip_runtime.h>

#include <mutex>

#include "gca_plan.hpp"

namespace gca {

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

void* scratch_ptr(hipError_t* err) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess && (dev < 0 || dev >= kMaxDevices)) e = hipErrorInvalidDevice;
  if (e != hipSuccess) {
    *err = e;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      *err = e != hipSuccess ? e : hipErrorInvalidSymbol;
      return nullptr;
    }
    addr[dev] = p;
  }
  *err = hipSuccess;
  return addr[dev];
}

}  // namespace gca
