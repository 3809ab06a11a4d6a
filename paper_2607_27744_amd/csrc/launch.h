// hipLaunchKernel wrapper: returns the launch status directly instead of
// going through the thread's sticky last-error state.
#pragma once

#include <hip/hip_runtime.h>

#include <tuple>

namespace rocs {

template <typename... KArgs, typename... Args>
hipError_t launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t stream,
                         Args... args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel argument count mismatch");
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return hipSuccess;
  std::tuple<KArgs...> packed(static_cast<KArgs>(args)...);
  void* ptrs[sizeof...(KArgs)];
  std::apply([&](auto&... e) {
    int i = 0;
    ((ptrs[i++] = static_cast<void*>(&e)), ...);
  }, packed);
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, 0, stream);
}

}  // namespace rocs
