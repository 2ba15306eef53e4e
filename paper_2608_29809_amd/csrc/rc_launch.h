// Kernel launch helper shared by every launch site of the library.
//
// Launches go through hipExtLaunchKernel so that, while a timing span is
// open on the calling thread, the dispatch itself stamps the span's events
// with the kernel's own start and end times (no marker packets between the
// kernels of a step).  Arguments are converted to the kernel's parameter
// types before their addresses are handed over.
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <tuple>
#include <utility>

namespace rc {

// Open span: the first launch stamps `start` with its start time, every
// launch stamps `stop` with its end time; `launches` counts them.
struct LaunchTiming {
  hipEvent_t start = nullptr, stop = nullptr;
  int launches = 0;
};
LaunchTiming &launch_timing();

template <typename... KArgs, typename... Args>
inline hipError_t rc_launch(void (*kernel)(KArgs...), dim3 grid, dim3 block, uint32_t shmem, hipStream_t s,
                            Args &&...args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "argument count must match the kernel");
  std::tuple<KArgs...> held(std::forward<Args>(args)...);
  LaunchTiming &t = launch_timing();
  hipEvent_t start = nullptr, stop = nullptr;
  if (t.stop) {
    start = t.start;
    stop = t.stop;
    t.start = nullptr;
    ++t.launches;
  }
  return std::apply(
      [&](auto &...e) {
        void *ptrs[sizeof...(KArgs) + 1] = {(void *)&e...};
        return hipExtLaunchKernel((const void *)kernel, grid, block, ptrs, shmem, s, start, stop, 0);
      },
      held);
}

}  // namespace rc
