// launch.h -- the one kernel-launch path of the library.
//
// Kernel timing: a caller that wants the GPU time of a launcher's kernels
// sets launch_timing (this thread's start / stop events) before calling the
// launcher.  The first kernel then records `start` and every kernel records
// `stop` in its own dispatch packet (hipExtLaunchKernelGGL), so the interval
// covers exactly the kernels' execution, with no extra packets on the
// stream.  Without timing events kernels launch normally.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

namespace lpp {

struct LaunchTiming {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};
LaunchTiming& launch_timing();   // this thread's events (runtime.cpp)

template <typename... Args, typename F>
inline void launch(F kernel, const dim3& grid, const dim3& block, uint32_t shmem, hipStream_t st, Args... args) {
    LaunchTiming& t = launch_timing();
    if (t.stop) {
        hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, t.start, t.stop, 0u, args...);
        t.start = nullptr;
    } else {
        hipLaunchKernelGGL(kernel, grid, block, shmem, st, args...);
    }
}

}  // namespace lpp
