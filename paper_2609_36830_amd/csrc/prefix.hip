// Prefix Forgetting Score for gfx950 (Eq. (5), Sec. 3.2; the scoring caps
// and the 32-token minimum of Appendix B): per rescored prefix, the mean of
// |lp_new - lp_behavior| over its first `cap` eligible (tag != -1) tokens, or
// NaN when fewer than `min_tokens` are eligible.
//
// One wave per prefix, HBM-bound (8 bytes per token, 12 with tags). The wave
// reads the prefix in windows of 256 tokens, as four rows of 64 consecutive
// tokens, so every load instruction reads 256 contiguous bytes. A token's
// position in the eligible order is the running count plus the eligible
// tokens of earlier rows (ballot) and of lower lanes in its row; tokens at
// position >= cap are skipped and the walk stops once the cap is reached.
// Each lane adds its terms in binary64; a butterfly of shuffles sums the
// lanes (a fixed order, so results repeat bit for bit).
#include "device_util.hpp"
#include "kernels.hpp"

#pragma clang fp contract(off)

namespace pace {

namespace {

constexpr int kPRows = 4;

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int off = kWave / 2; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

template <bool kTags>
__global__ __launch_bounds__(256) void prefix_score_kernel(const float *__restrict__ lp_new,
                                                          const float *__restrict__ lp_beh,
                                                          const int32_t *__restrict__ tags,
                                                          const int64_t *__restrict__ po, int64_t n,
                                                          int64_t NT, int64_t cap, int64_t min_tokens,
                                                          double *__restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (i >= n) return;
    const int lane = lane_id();
    const int64_t lo = clamp64(po[i], 0, NT), hi = clamp64(po[i + 1], 0, NT);
    const uint64_t below = lanes_below();
    double acc = 0.0;
    int64_t m = 0;                                   // eligible tokens before the current window
    for (int64_t w = lo; w < hi && m < cap; w += (int64_t)kWave * kPRows) {
        float a[kPRows], b[kPRows];
        bool e[kPRows];
#pragma unroll
        for (int k = 0; k < kPRows; ++k) {
            const int64_t p = w + (int64_t)k * kWave + lane;
            const bool in = p < hi;
            e[k] = in && (!kTags || tags[p] != -1);
            a[k] = in ? lp_new[p] : 0.0f;
            b[k] = in ? lp_beh[p] : 0.0f;
        }
        int64_t row_base = m;
#pragma unroll
        for (int k = 0; k < kPRows; ++k) {
            const uint64_t bal = ballot(e[k]);
            const int64_t idx = row_base + (int64_t)__popcll(bal & below);
            if (e[k] && idx < cap) {
                const double d = (double)a[k] - (double)b[k];
                acc += __builtin_fabs(d);
            }
            row_base += (int64_t)__popcll(bal);
        }
        m = row_base;
    }
    const double total = wave_sum_f64(acc);
    if (lane == 0) {
        const int64_t mm = m < cap ? m : cap;
        out[i] = (mm >= min_tokens && mm > 0) ? total / (double)mm : __builtin_nan("");
    }
}

}  // namespace

hipError_t launch_prefix_score(const float *lp_new, const float *lp_beh, const int32_t *tags,
                               const int64_t *prefix_offsets, int64_t n, int64_t n_tokens, int64_t cap,
                               int64_t min_tokens, double *s_pre, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const dim3 grid((unsigned)((n + 3) / 4));
    if (tags)
        return launch(-1, prefix_score_kernel<true>, grid, dim3(256), stream, lp_new, lp_beh, tags,
                      prefix_offsets, n, n_tokens, cap, min_tokens, s_pre);
    return launch(-1, prefix_score_kernel<false>, grid, dim3(256), stream, lp_new, lp_beh, tags, prefix_offsets,
                  n, n_tokens, cap, min_tokens, s_pre);
}

}  // namespace pace
