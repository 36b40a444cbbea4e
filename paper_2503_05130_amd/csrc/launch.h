// Kernel launch helper and storage types shared by every kernel file (gfx950).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace iefwd {

// Kernel-only timing: when a pair of events is armed on this host thread, the
// next kernel launch records its own dispatch start and end into them (the
// timestamps of the kernel itself, not of markers around it) and disarms.
struct LaunchEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};
// Events armed by the caller for the next launches on this thread: the first
// kernel records `start` as it begins, and every kernel records `stop` as it
// ends, so for an operation of several kernels the pair spans all of them.
LaunchEvents &armed_launch_events();
// Kernels launched by this thread so far.
uint64_t &launch_count();

template <typename F, typename... Args>
hipError_t launch_kernel(F kernel, dim3 grid, dim3 block, hipStream_t stream, Args... args) {
    LaunchEvents &ev = armed_launch_events();
    if (ev.stop) {
        hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, ev.start, ev.stop, 0, args...);
        ev.start = nullptr;
    } else {
        hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
    }
    ++launch_count();
    return hipGetLastError();
}

using bf16_t = uint16_t;   // bf16 storage: the upper half of an fp32 bit pattern

}  // namespace iefwd
