// Kernel launches for the kernel files: every kernel is launched through
// launch_kernel, which converts the arguments to the kernel's parameter types,
// feeds the per-kernel timing hook and, with GCA_DEBUG_SYNC, checks each launch.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <tuple>
#include <utility>

#include "gca_plan.hpp"

namespace gca {

template <typename Tup, size_t... I>
inline void kernel_arg_ptrs(Tup& t, void** p, std::index_sequence<I...>) {
  ((p[I] = static_cast<void*>(&std::get<I>(t))), ...);
}

// While the timing hook is armed the dispatch itself carries a start and a stop
// event (hipExtLaunchKernel), so timing a kernel adds no packets to the stream
// and measures the kernel alone.  With GCA_DEBUG_SYNC every launch is followed
// by a synchronisation of its stream, so that a fault is reported with the name
// of the kernel that caused it.
template <typename... KArgs, typename... Args>
inline void launch_kernel(const char* name, void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t smem,
                          hipStream_t stream, Args... args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel argument count");
  std::tuple<KArgs...> a{static_cast<KArgs>(args)...};
  void* ptrs[sizeof...(KArgs)];
  kernel_arg_ptrs(a, ptrs, std::index_sequence_for<KArgs...>{});
  hipEvent_t start = nullptr, stop = nullptr;
  const void* f = reinterpret_cast<const void*>(kernel);
  hipError_t e;
  if (profile_slot(name, &start, &stop))
    e = hipExtLaunchKernel(f, grid, block, ptrs, smem, stream, start, stop, 0);
  else
    e = hipLaunchKernel(f, grid, block, ptrs, smem, stream);
  if (e == hipSuccess && debug_sync()) {
    e = hipStreamSynchronize(stream);
    if (e == hipSuccess) e = hipGetLastError();
  }
  note_launch_error(e, name);
}

}  // namespace gca
