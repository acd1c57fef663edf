// Wave64 helpers for the gfx950 kernels of the PACE filter step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pace {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

__device__ __forceinline__ uint64_t ballot(bool p) { return (uint64_t)__ballot(p); }

// Lanes below the caller's lane.
__device__ __forceinline__ uint64_t lanes_below() {
    return (lane_id() == 0) ? 0ull : (~0ull >> (kWave - lane_id()));
}

__device__ __forceinline__ int32_t readlane_i32(int32_t v, int lane) {
    return __builtin_amdgcn_readlane(v, lane);
}

__device__ __forceinline__ int64_t readlane_i64(int64_t v, int lane) {
    uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), lane);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m, kWave);
        uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m, kWave);
        v += ((uint64_t)hi << 32) | lo;
    }
    return v;
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
    return (int64_t)wave_sum_u64((uint64_t)v);
}

// Inclusive prefix sum across the wave (lane order).
__device__ __forceinline__ int64_t wave_incl_scan_i64(int64_t v) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        uint32_t lo = (uint32_t)__shfl_up((int)(uint32_t)(uint64_t)v, d, kWave);
        uint32_t hi = (uint32_t)__shfl_up((int)(uint32_t)((uint64_t)v >> 32), d, kWave);
        int64_t o = (int64_t)(((uint64_t)hi << 32) | lo);
        if (lane_id() >= d) v += o;
    }
    return v;
}

__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        uint32_t o = (uint32_t)__shfl_up((int)v, d, kWave);
        if (lane_id() >= d) v += o;
    }
    return v;
}

// Last index i in [0, n] with a[i] <= p (a non-decreasing), or -1. Every lane
// of the wave must call it with the same (a, n, p); the result is uniform.
// For an array that is not monotone the result is still an index in [-1, n]
// and every load stays inside a[0..n].
__device__ __forceinline__ int64_t wave_last_le(const int64_t *__restrict__ a, int64_t n, int64_t p) {
    const int lane = lane_id();
    int64_t base = 0, len = n + 1;
    while (len > kWave) {
        int64_t step = (len + kWave - 1) / kWave;
        int64_t idx = base + (int64_t)lane * step;
        bool le = (idx < base + len) && (a[idx] <= p);
        int cnt = __popcll(ballot(le));
        if (cnt == 0) return base - 1;
        int64_t nb = base + (int64_t)(cnt - 1) * step;
        int64_t rem = base + len - nb;
        len = rem < step ? rem : step;
        base = nb;
    }
    bool le = (lane < len) && (a[base + lane] <= p);
    return base + (int64_t)__popcll(ballot(le)) - 1;
}

__device__ __forceinline__ int64_t clamp64(int64_t v, int64_t lo, int64_t hi) {
    return v < lo ? lo : (v > hi ? hi : v);
}

}  // namespace pace
