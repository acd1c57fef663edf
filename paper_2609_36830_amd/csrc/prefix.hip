// Prefix Forgetting Score for gfx950 (Eq. (5), Sec. 3.2; the scoring caps
// and the 32-token minimum of Appendix B): per rescored prefix, the mean of
// |lp_new - lp_behavior| over its first `cap` eligible (tag != -1) tokens, or
// NaN when fewer than `min_tokens` are eligible.
//
// One 256-thread workgroup per prefix, HBM-bound (8 bytes per token, 12 with
// tags). A round covers 1024 tokens: each wave takes 256 of them as four rows
// of 64 consecutive tokens, so every load instruction reads 256 contiguous
// bytes, and all of a round's loads are in flight together (one round covers
// a whole capped prefix unless many tokens are masked). A token's position in
// the eligible order is the running count plus the eligible tokens of earlier
// waves (LDS), earlier rows (ballot) and lower lanes in its row; tokens at
// position >= cap are skipped and the walk stops once the cap is reached.
// Each lane adds its terms in binary64; a butterfly of shuffles sums a wave,
// and thread 0 adds the four wave sums in order (a fixed order, so results
// repeat bit for bit).
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
    constexpr int kW = 256 / kWave;                   // waves per prefix
    constexpr int64_t kSpan = (int64_t)256 * kPRows;  // tokens per round (1024)
    __shared__ int64_t wcnt[kW];
    __shared__ double wacc[kW];
    const int64_t i = blockIdx.x;
    if (i >= n) return;
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    const int64_t lo = clamp64(po[i], 0, NT), hi = clamp64(po[i + 1], 0, NT);
    const uint64_t below = lanes_below();
    double acc = 0.0;
    int64_t m = 0;                                   // eligible tokens before the current round
    for (int64_t w = lo; w < hi && m < cap; w += kSpan) {
        // this wave's 256 tokens, four rows of 64
        const int64_t wb = w + (int64_t)wave * kWave * kPRows;
        float a[kPRows], b[kPRows];
        bool e[kPRows];
        uint64_t bal[kPRows];
        int64_t mine = 0;
#pragma unroll
        for (int k = 0; k < kPRows; ++k) {
            const int64_t p = wb + (int64_t)k * kWave + lane;
            const bool in = p < hi;
            e[k] = in && (!kTags || tags[p] != -1);
            a[k] = in ? lp_new[p] : 0.0f;
            b[k] = in ? lp_beh[p] : 0.0f;
        }
#pragma unroll
        for (int k = 0; k < kPRows; ++k) {
            bal[k] = ballot(e[k]);
            mine += (int64_t)__popcll(bal[k]);
        }
        if (lane == 0) wcnt[wave] = mine;
        __syncthreads();
        int64_t row_base = m, total = m;
#pragma unroll
        for (int v = 0; v < kW; ++v) {
            row_base += (v < wave) ? wcnt[v] : 0;
            total += wcnt[v];
        }
#pragma unroll
        for (int k = 0; k < kPRows; ++k) {
            const int64_t idx = row_base + (int64_t)__popcll(bal[k] & below);
            if (e[k] && idx < cap) {
                const double d = (double)a[k] - (double)b[k];
                acc += __builtin_fabs(d);
            }
            row_base += (int64_t)__popcll(bal[k]);
        }
        m = total;
        __syncthreads();
    }
    const double ws = wave_sum_f64(acc);
    if (lane == 0) wacc[wave] = ws;
    __syncthreads();
    if (threadIdx.x == 0) {
        double sum = 0.0;
#pragma unroll
        for (int v = 0; v < kW; ++v) sum += wacc[v];
        const int64_t mm = m < cap ? m : cap;
        out[i] = (mm >= min_tokens && mm > 0) ? sum / (double)mm : __builtin_nan("");
    }
}

}  // namespace

hipError_t launch_prefix_score(const float *lp_new, const float *lp_beh, const int32_t *tags,
                               const int64_t *prefix_offsets, int64_t n, int64_t n_tokens, int64_t cap,
                               int64_t min_tokens, double *s_pre, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const dim3 grid((unsigned)n);
    if (tags)
        return launch(kPhasePrefix, prefix_score_kernel<true>, grid, dim3(256), stream, lp_new, lp_beh, tags,
                      prefix_offsets, n, n_tokens, cap, min_tokens, s_pre);
    return launch(kPhasePrefix, prefix_score_kernel<false>, grid, dim3(256), stream, lp_new, lp_beh, tags, prefix_offsets,
                  n, n_tokens, cap, min_tokens, s_pre);
}

}  // namespace pace
