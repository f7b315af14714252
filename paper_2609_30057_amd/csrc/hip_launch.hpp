// hip_launch.hpp -- host-side launch helpers shared by the kernel sources.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include <tuple>
#include <utility>

namespace krex {

// hipLaunchKernel with the kernel's own parameter types, returning the
// launch status directly instead of through the sticky last-error state.
template <typename... KArgs, typename... Actual>
static hipError_t launch(void (*kern)(KArgs...), dim3 grid, dim3 block, hipStream_t s, Actual &&...a)
{
    std::tuple<KArgs...> args(std::forward<Actual>(a)...);
    void *argv[sizeof...(KArgs)];
    std::apply([&](auto &...x) {
        int i = 0;
        ((argv[i++] = (void *)&x), ...);
    }, args);
    return hipLaunchKernel((const void *)kern, grid, block, argv, 0, s);
}

// A launch-shape setting from the environment (positive integer), else dflt.
inline uint32_t tune_env(const char *name, uint32_t dflt)
{
    const char *e = getenv(name);
    if (!e) return dflt;
    const unsigned long v = strtoul(e, nullptr, 10);
    return v ? (uint32_t)v : dflt;
}

}  // namespace krex
