// Score of a prompt group (Appendix B: the full method aggregates scores by
// the mean within prompt groups). Consecutive trajectories form the groups:
// group g holds trajectories [go[g], go[g+1]), offsets clamped to [0, n].
#pragma once

#include "device_util.hpp"

#pragma clang fp contract(off)

namespace pace {

// The members' scores added in member order starting from 0, then one
// division by the member count; an empty group scores 0. Members are loaded
// eight at a time (one round trip per eight); the additions keep member order.
__device__ __forceinline__ double group_mean(const double *__restrict__ score, int64_t n,
                                             const int64_t *__restrict__ go, int64_t g) {
    const int64_t lo = clamp64(go[g], 0, n), hi = clamp64(go[g + 1], 0, n);
    double sum = 0.0;
    for (int64_t b = lo; b < hi; b += 8) {
        double x[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] = b + k < hi ? score[b + k] : 0.0;
#pragma unroll
        for (int k = 0; k < 8; ++k)
            if (b + k < hi) sum = sum + x[k];
    }
    return (hi > lo) ? sum / (double)(hi - lo) : 0.0;
}

}  // namespace pace
