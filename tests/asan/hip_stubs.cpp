// Host-only stand-ins for what the C ABI layer (api.cpp, plan.cpp) calls outside
// itself: the few HIP runtime functions it uses and the kernel launchers.  With
// these the validation layer builds and runs under AddressSanitizer and
// UndefinedBehaviorSanitizer on a machine without a GPU.  A launcher is reached
// only by a call that passed validation; it reports a launch failure.
#include <hip/hip_runtime_api.h>

#include "gca_plan.hpp"

extern "C" {
const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "stubbed HIP error"; }
hipError_t hipGetLastError(void) { return hipSuccess; }
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t, int) {
  *v = 256;
  return hipSuccess;
}
hipError_t hipPointerGetAttributes(hipPointerAttribute_t* a, const void*) {
  a->type = hipMemoryTypeDevice;
  return hipSuccess;
}
hipError_t hipHostGetDevicePointer(void** d, void*, unsigned int) {
  *d = nullptr;
  return hipErrorInvalidValue;
}
}

namespace gca {
static int g_launches = 0;
int stub_launches() { return g_launches; }
static hipError_t launched() {
  ++g_launches;
  return hipErrorLaunchFailure;
}
hipError_t launch_chunk_scores(const Shape&, const void*, const void*, float*, hipStream_t) { return launched(); }
hipError_t launch_topk(const Shape&, const float*, int32_t*, float*, hipStream_t) { return launched(); }
hipError_t launch_decode_scan(const Shape&, const void*, const void*, void*, hipStream_t) { return launched(); }
hipError_t launch_xattn_decode(const Shape&, const float*, const int*, const void*, const void*, const void*,
                               int32_t*, float*, void*, float*, float*, const void*, const void*, hipStream_t) {
  return launched();
}
hipError_t launch_fused_select(const Shape&, const void*, const void*, int32_t*, float*, void*, hipStream_t) {
  return launched();
}
hipError_t launch_xattn_fwd(const Shape&, const void*, const void*, const void*, const int32_t*, const float*,
                            void*, float*, float*, hipStream_t) {
  return launched();
}
hipError_t launch_xattn_bwd(const Shape&, const void*, const void*, const void*, const int32_t*, const float*,
                            const float*, const void*, void*, void*, void*, float*, const void*, const void*, float*,
                            float*, void*, hipStream_t) {
  return launched();
}
void* scratch_ptr(hipError_t* err) {
  static unsigned char fake[256] __attribute__((aligned(256)));
  *err = hipSuccess;
  return fake;
}
}  // namespace gca
