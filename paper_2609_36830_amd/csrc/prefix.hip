// Prefix Forgetting Score for gfx950 (Eq. (5), Sec. 3.2; the scoring caps
// and the 32-token minimum of Appendix B): per rescored prefix, the mean of
// |lp_new - lp_behavior| over its first `cap` eligible (tag != -1) tokens, or
// NaN when fewer than `min_tokens` are eligible.
//
// One wave per prefix, four prefixes per 256-thread workgroup, so a pool's
// few thousand prefixes are all resident at once and each waits on one round
// trip. HBM-bound (8 bytes per token, 12 with tags). A round covers 1024
// tokens as four sub-rounds of 256, four consecutive tokens per lane in each,
// read as one 16-byte vector per array (dword-aligned loads); all twelve
// loads of a round are in flight together, and one round covers a whole
// capped prefix unless many tokens are masked. A lane wholly past the
// prefix's end re-reads the round's first vector (no extra traffic) and
// masks it, so no load sits behind a branch; only a round that reaches the
// last tokens of the whole array reads element by element. A token's position in the
// eligible order is the running count plus a wave exclusive scan of the
// lanes' eligible counts plus the eligible tokens before it in its lane;
// tokens at position >= cap are skipped and the walk stops once the cap is
// reached. Each lane adds its terms in binary64 and a butterfly of shuffles
// sums the wave (a fixed order, so results repeat bit for bit).
#include "device_util.hpp"
#include "kernels.hpp"

#pragma clang fp contract(off)

namespace pace {

namespace {

constexpr int kPT4 = 4;                        // tokens per lane per sub-round
constexpr int kPSub = 4;                       // sub-rounds per round
constexpr int kPWaves = 4;                     // prefixes per workgroup
constexpr int64_t kPSubSpan = (int64_t)kWave * kPT4;     // 256 tokens
constexpr int64_t kPRound = kPSubSpan * kPSub;            // 1024 tokens

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int off = kWave / 2; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Four consecutive 4-byte elements at a (dword-aligned), as one load.
template <typename T>
__device__ __forceinline__ void vec4(const T *a, T (&v)[kPT4]) {
    const uint4 x = load_a4(a);
    const uint32_t w[kPT4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < kPT4; ++e) v[e] = __builtin_bit_cast(T, w[e]);
}

// Elements [q, q + 4) of a 4-byte array of NT elements, those at or past NT
// as `fill`.
template <typename T>
__device__ __forceinline__ void load4(const T *__restrict__ a, int64_t q, int64_t NT, T fill, T (&v)[kPT4]) {
    if (q + kPT4 <= NT) {
        const uint4 x = load_a4(a + q);
        const uint32_t w[kPT4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int e = 0; e < kPT4; ++e) v[e] = __builtin_bit_cast(T, w[e]);
    } else {
#pragma unroll
        for (int e = 0; e < kPT4; ++e) v[e] = q + e < NT ? a[q + e] : fill;
    }
}

template <bool kTags>
__global__ __launch_bounds__(256) void prefix_score_kernel(const float *__restrict__ lp_new,
                                                          const float *__restrict__ lp_beh,
                                                          const int32_t *__restrict__ tags,
                                                          const int64_t *__restrict__ po, int64_t n,
                                                          int64_t NT, int64_t cap, int64_t min_tokens,
                                                          double *__restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * kPWaves + threadIdx.x / kWave;
    if (i >= n) return;                              // whole waves; no workgroup barrier below
    const int lane = lane_id();
    // The same for the whole wave: read through lane 0 so that the walk's
    // control flow is scalar.
    const int64_t lo = readlane_i64(clamp64(po[i], 0, NT), 0);
    const int64_t hi = readlane_i64(clamp64(po[i + 1], 0, NT), 0);
    double acc = 0.0;
    int64_t m = 0;                                   // eligible tokens before the current sub-round
    for (int64_t w = lo; w < hi && m < cap; w += kPRound) {
        float a[kPSub][kPT4], b[kPSub][kPT4];
        int32_t tg[kPSub][kPT4];
        // Every lane reads [q, q + 4) with q <= w + kPRound - 4. A round whose
        // vectors all lie inside the array (the same answer for the whole
        // wave) takes plain vector loads; only a round that reaches the
        // array's last tokens takes the element-by-element form.
        if (w + kPRound <= NT) {
#pragma unroll
            for (int u = 0; u < kPSub; ++u) {
                const int64_t p = w + u * kPSubSpan + (int64_t)lane * kPT4;
                const int64_t q = p < hi ? p : w;    // w < hi <= NT
                vec4<float>(lp_new + q, a[u]);
                vec4<float>(lp_beh + q, b[u]);
                if (kTags) vec4<int32_t>(tags + q, tg[u]);
            }
        } else {
#pragma unroll
            for (int u = 0; u < kPSub; ++u) {
                const int64_t p = w + u * kPSubSpan + (int64_t)lane * kPT4;
                const int64_t q = p < hi ? p : w;
                load4<float>(lp_new, q, NT, 0.0f, a[u]);
                load4<float>(lp_beh, q, NT, 0.0f, b[u]);
                if (kTags) load4<int32_t>(tags, q, NT, -1, tg[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < kPSub; ++u) {
            const int64_t p = w + u * kPSubSpan + (int64_t)lane * kPT4;
            bool e[kPT4];
            uint32_t cnt = 0;
#pragma unroll
            for (int k = 0; k < kPT4; ++k) {
                e[k] = p + k < hi && (!kTags || tg[u][k] != -1);
                cnt += e[k] ? 1u : 0u;
            }
            const uint32_t incl = wave_incl_scan_u32(cnt);
            const uint32_t total = (uint32_t)readlane_i32((int32_t)incl, kWave - 1);
            int64_t idx = m + (incl - cnt);
#pragma unroll
            for (int k = 0; k < kPT4; ++k) {
                if (e[k]) {
                    if (idx < cap) acc += __builtin_fabs((double)a[u][k] - (double)b[u][k]);
                    ++idx;
                }
            }
            m += total;
        }
    }
    const double sum = wave_sum_f64(acc);
    if (lane == 0) {
        const int64_t mm = m < cap ? m : cap;
        out[i] = (mm >= min_tokens && mm > 0) ? sum / (double)mm : __builtin_nan("");
    }
}

}  // namespace

hipError_t launch_prefix_score(const float *lp_new, const float *lp_beh, const int32_t *tags,
                               const int64_t *prefix_offsets, int64_t n, int64_t n_tokens, int64_t cap,
                               int64_t min_tokens, double *s_pre, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const dim3 grid((unsigned)((n + kPWaves - 1) / kPWaves));
    if (tags)
        return launch(kPhasePrefix, prefix_score_kernel<true>, grid, dim3(256), stream, lp_new, lp_beh, tags,
                      prefix_offsets, n, n_tokens, cap, min_tokens, s_pre);
    return launch(kPhasePrefix, prefix_score_kernel<false>, grid, dim3(256), stream, lp_new, lp_beh, tags, prefix_offsets,
                  n, n_tokens, cap, min_tokens, s_pre);
}

}  // namespace pace
