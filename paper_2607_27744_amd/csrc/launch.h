// hipLaunchKernel wrapper: returns the launch status directly instead of
// going through the thread's sticky last-error state.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <tuple>

namespace rocs {

// A launch may hold fewer than 2^32 work items per grid dimension. Launchers
// test their computed 1-D grids with this before narrowing them to 32 bits.
inline bool grid_fits(int64_t blocks, int64_t threads) {
  return blocks >= 0 && blocks * threads < (int64_t(1) << 32);
}

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

// Compute units of the current device, queried once per device and cached:
// persistent kernels size their grids by it on every launch.
inline hipError_t current_cu_count(int* cus) {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cache[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const bool slot = dev >= 0 && dev < kMaxDevices;
  if (slot) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) {
      *cus = c;
      return hipSuccess;
    }
  }
  int c = 0;
  e = hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (slot) cache[dev].store(c, std::memory_order_relaxed);
  *cus = c;
  return hipSuccess;
}

}  // namespace rocs
