// profile.h -- optional per-kernel timing of the library's own launches.
//
// While a thread has profiling enabled (sbp_profile_begin), every kernel the
// library launches from that thread goes through hipExtLaunchKernelGGL with a
// start/stop event pair recorded together with the dispatch, and its name is
// kept; sbp_profile_end waits for the events and returns the durations.
// Otherwise kernels are launched with hipLaunchKernelGGL as usual.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdio.h>

namespace sbpi {

struct ProfileSlot {
    hipEvent_t start, stop;
    char name[160];
};

// Next free slot of this thread's profile, or nullptr when not profiling
// (or when the profile is full).
ProfileSlot *profile_next();

template <typename F, typename... Args>
hipError_t launch_kernel(F kernel, const char *name, dim3 grid, dim3 block, hipStream_t s,
                         Args... args) {
    ProfileSlot *p = profile_next();
    if (p) {
        snprintf(p->name, sizeof(p->name), "%s", name);
        hipExtLaunchKernelGGL(kernel, grid, block, 0, s, p->start, p->stop, 0, args...);
    } else {
        hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
    }
    return hipGetLastError();
}

}  // namespace sbpi
