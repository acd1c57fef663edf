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

// DPP moves within a wave64: row_shr:k shifts inside each 16-lane row,
// row_bcast:15 / row_bcast:31 carry a row's last lane into the following
// row(s). Lanes without a source (or outside row_mask) receive `old`.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, kCtrl, kRowMask, 0xf, false);
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t old, uint64_t v) {
    const uint32_t lo = dpp_u32<kCtrl, kRowMask>((uint32_t)old, (uint32_t)v);
    const uint32_t hi = dpp_u32<kCtrl, kRowMask>((uint32_t)(old >> 32), (uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// Inclusive scan in lane order for an associative op with identity `id`
// (row shifts 1,2,4,8, then the two row broadcasts). Lane 63 ends with the
// reduction of the whole wave. All 64 lanes must be active.
template <typename Op>
__device__ __forceinline__ uint32_t wave_scan_u32(uint32_t v, uint32_t id, Op op) {
    v = op(v, dpp_u32<0x111, 0xf>(id, v));
    v = op(v, dpp_u32<0x112, 0xf>(id, v));
    v = op(v, dpp_u32<0x114, 0xf>(id, v));
    v = op(v, dpp_u32<0x118, 0xf>(id, v));
    v = op(v, dpp_u32<0x142, 0xa>(id, v));
    v = op(v, dpp_u32<0x143, 0xc>(id, v));
    return v;
}
template <typename Op>
__device__ __forceinline__ uint64_t wave_scan_u64(uint64_t v, uint64_t id, Op op) {
    v = op(v, dpp_u64<0x111, 0xf>(id, v));
    v = op(v, dpp_u64<0x112, 0xf>(id, v));
    v = op(v, dpp_u64<0x114, 0xf>(id, v));
    v = op(v, dpp_u64<0x118, 0xf>(id, v));
    v = op(v, dpp_u64<0x142, 0xa>(id, v));
    v = op(v, dpp_u64<0x143, 0xc>(id, v));
    return v;
}

__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) {
    return wave_scan_u32(v, 0u, [](uint32_t a, uint32_t b) { return a + b; });
}
__device__ __forceinline__ int64_t wave_incl_scan_i64(int64_t v) {
    return (int64_t)wave_scan_u64((uint64_t)v, 0ull, [](uint64_t a, uint64_t b) { return a + b; });
}
// Inclusive scans inside each row of 16 lanes (row_shr 1, 2, 4, 8): lane
// 16 r + 15 ends with the sum of its row.
__device__ __forceinline__ int64_t row_incl_scan_i64(int64_t v) {
    uint64_t x = (uint64_t)v;
    x += dpp_u64<0x111, 0xf>(0ull, x);
    x += dpp_u64<0x112, 0xf>(0ull, x);
    x += dpp_u64<0x114, 0xf>(0ull, x);
    x += dpp_u64<0x118, 0xf>(0ull, x);
    return (int64_t)x;
}
__device__ __forceinline__ uint32_t row_incl_scan_u32(uint32_t x) {
    x += dpp_u32<0x111, 0xf>(0u, x);
    x += dpp_u32<0x112, 0xf>(0u, x);
    x += dpp_u32<0x114, 0xf>(0u, x);
    x += dpp_u32<0x118, 0xf>(0u, x);
    return x;
}
// Wave-wide reductions, broadcast to every lane.
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
    return (uint64_t)readlane_i64((int64_t)wave_scan_u64(v, 0ull, [](uint64_t a, uint64_t b) { return a + b; }), kWave - 1);
}
__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) { return (int64_t)wave_sum_u64((uint64_t)v); }
__device__ __forceinline__ uint64_t wave_or_u64(uint64_t v) {
    return (uint64_t)readlane_i64((int64_t)wave_scan_u64(v, 0ull, [](uint64_t a, uint64_t b) { return a | b; }), kWave - 1);
}
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
    return (uint64_t)readlane_i64((int64_t)wave_scan_u64(v, ~0ull, [](uint64_t a, uint64_t b) { return a < b ? a : b; }), kWave - 1);
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
    return (uint64_t)readlane_i64((int64_t)wave_scan_u64(v, 0ull, [](uint64_t a, uint64_t b) { return a > b ? a : b; }), kWave - 1);
}
__device__ __forceinline__ uint64_t wave_and_u64(uint64_t v) {
    return (uint64_t)readlane_i64((int64_t)wave_scan_u64(v, ~0ull, [](uint64_t a, uint64_t b) { return a & b; }), kWave - 1);
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

// Exclusive prefix sums over a block of kWaves waves in thread order; the
// block total goes to *total. wsum: kWaves words of LDS. Two barriers.
template <int kWaves>
__device__ __forceinline__ uint32_t block_excl_sum_u32(uint32_t v, uint32_t &total, uint32_t *wsum) {
    const uint32_t incl = wave_incl_scan_u32(v);
    const int w = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) wsum[w] = incl;
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < kWaves; ++k) {
        const uint32_t x = wsum[k];
        tot += x;
        before += (k < w) ? x : 0u;
    }
    __syncthreads();
    total = tot;
    return before + incl - v;
}

template <int kWaves>
__device__ __forceinline__ int64_t block_excl_sum_i64(int64_t v, int64_t &total, int64_t *wsum) {
    const int64_t incl = wave_incl_scan_i64(v);
    const int w = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) wsum[w] = incl;
    __syncthreads();
    int64_t before = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < kWaves; ++k) {
        const int64_t x = wsum[k];
        tot += x;
        before += (k < w) ? x : 0;
    }
    __syncthreads();
    total = tot;
    return before + incl - v;
}

// Streaming (non-temporal) 16-byte accesses: data touched once per step
// should not displace reusable lines from L2 and MALL.
typedef int pace_v4i __attribute__((ext_vector_type(4)));
typedef unsigned pace_v4u __attribute__((ext_vector_type(4)));
__device__ __forceinline__ int4 load_nt(const int4 *p) {
    const pace_v4i x = __builtin_nontemporal_load(reinterpret_cast<const pace_v4i *>(p));
    return make_int4(x.x, x.y, x.z, x.w);
}
__device__ __forceinline__ uint4 load_nt(const uint4 *p) {
    const pace_v4u x = __builtin_nontemporal_load(reinterpret_cast<const pace_v4u *>(p));
    return make_uint4(x.x, x.y, x.z, x.w);
}
// 16 bytes from an address that is only 4-byte aligned (one dwordx4 load).
typedef unsigned pace_v4u_a4 __attribute__((ext_vector_type(4), aligned(4)));
__device__ __forceinline__ uint4 load_a4(const void *p) {
    const pace_v4u_a4 x = *reinterpret_cast<const pace_v4u_a4 *>(p);
    return make_uint4(x.x, x.y, x.z, x.w);
}
__device__ __forceinline__ void store_nt(uint4 *p, const uint4 &v) {
    const pace_v4u x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<pace_v4u *>(p));
}

// 64-bit key whose unsigned order is the order of binary64 scores: the
// sign-magnitude flip, with -0 mapped to +0 (equal scores) and NaN above +inf.
__device__ __forceinline__ uint64_t score_key(double d) {
    if (__builtin_isnan(d)) return ~0ull;    // precondition violation: above +inf
    if (d == 0.0) d = 0.0;                    // -0 and +0 are the same score
    const uint64_t b = (uint64_t)__double_as_longlong(d);
    return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ int64_t clamp64(int64_t v, int64_t lo, int64_t hi) {
    return v < lo ? lo : (v > hi ? hi : v);
}

}  // namespace pace
