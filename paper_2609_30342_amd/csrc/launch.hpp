// launch.hpp -- kernel launch with optional timing events attached to the
// dispatch itself.
//
// hipExtLaunchKernelGGL records `start` when the kernel begins and `stop`
// when it ends, from the dispatch's own timestamps: no marker packets go
// into the stream, so a timed step runs exactly like an untimed one.  A
// phase of several launches puts `start` on its first dispatch and `stop`
// on its last.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

namespace rk {

template <typename K, typename... Args>
inline hipError_t launch(K kernel, dim3 grid, dim3 block, hipStream_t stream, hipEvent_t start,
                         hipEvent_t stop, Args... args)
{
    if (start || stop)
        hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, start, stop, 0u, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
    return hipGetLastError();
}

// Index of the last group with tiles (the dispatch that carries `stop`).
template <typename G>
inline int last_group(const G *groups, int ngroups)
{
    int last = -1;
    for (int q = 0; q < ngroups; ++q)
        if (groups[q].count > 0) last = q;
    return last;
}

}  // namespace rk
