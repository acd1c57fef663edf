// Prefix Forgetting Score for gfx950 (Eq. (5), Sec. 3.2; the scoring caps
// and the 32-token minimum of Appendix B): per rescored prefix, the mean of
// |lp_new - lp_behavior| over its first `cap` eligible (tag != -1) tokens, or
// NaN when fewer than `min_tokens` are eligible.
//
// One 256-thread workgroup per prefix, HBM-bound (8 bytes per token, 12 with
// tags). A round covers 1024 tokens, four consecutive ones per thread, read
// as one 16-byte vector per array (dword-aligned loads; the prefix's last
// partial vector element by element), all of a round's loads in flight
// together (one round covers a whole capped prefix unless many tokens are
// masked). A token's position in the eligible order is the running count plus
// a block exclusive scan of the threads' eligible counts plus the eligible
// tokens before it in its thread; tokens at position >= cap are skipped and
// the walk stops once the cap is reached. Each lane adds its terms in
// binary64; a butterfly of shuffles sums a wave, and thread 0 adds the four
// wave sums in order (a fixed order, so results repeat bit for bit).
#include "device_util.hpp"
#include "kernels.hpp"

#pragma clang fp contract(off)

namespace pace {

namespace {

constexpr int kPT4 = 4;   // tokens per thread per round

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int off = kWave / 2; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Elements [p, p + 4) of a 4-byte array, those at or past hi as `fill`.
template <typename T>
__device__ __forceinline__ void load4(const T *__restrict__ a, int64_t p, int64_t hi, T fill, T (&v)[kPT4]) {
    if (p + kPT4 <= hi) {
        const uint4 x = load_a4(a + p);
        const uint32_t w[kPT4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int e = 0; e < kPT4; ++e) v[e] = __builtin_bit_cast(T, w[e]);
    } else {
#pragma unroll
        for (int e = 0; e < kPT4; ++e) v[e] = p + e < hi ? a[p + e] : fill;
    }
}

template <bool kTags>
__global__ __launch_bounds__(256) void prefix_score_kernel(const float *__restrict__ lp_new,
                                                          const float *__restrict__ lp_beh,
                                                          const int32_t *__restrict__ tags,
                                                          const int64_t *__restrict__ po, int64_t n,
                                                          int64_t NT, int64_t cap, int64_t min_tokens,
                                                          double *__restrict__ out) {
    constexpr int kW = 256 / kWave;                   // waves per prefix
    constexpr int64_t kSpan = (int64_t)256 * kPT4;    // tokens per round (1024)
    __shared__ uint32_t wsum[kW];
    __shared__ double wacc[kW];
    const int64_t i = blockIdx.x;
    if (i >= n) return;
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    const int64_t lo = clamp64(po[i], 0, NT), hi = clamp64(po[i + 1], 0, NT);
    double acc = 0.0;
    int64_t m = 0;                                   // eligible tokens before the current round
    for (int64_t w = lo; w < hi && m < cap; w += kSpan) {
        const int64_t p = w + (int64_t)threadIdx.x * kPT4;
        float a[kPT4], b[kPT4];
        int32_t tg[kPT4];
        load4<float>(lp_new, p, hi, 0.0f, a);
        load4<float>(lp_beh, p, hi, 0.0f, b);
        if (kTags) load4<int32_t>(tags, p, hi, -1, tg);
        bool e[kPT4];
        uint32_t cnt = 0;
#pragma unroll
        for (int k = 0; k < kPT4; ++k) {
            e[k] = p + k < hi && (!kTags || tg[k] != -1);
            cnt += e[k] ? 1u : 0u;
        }
        uint32_t total;
        const uint32_t before = block_excl_sum_u32<kW>(cnt, total, wsum);
        int64_t idx = m + before;
#pragma unroll
        for (int k = 0; k < kPT4; ++k) {
            if (e[k]) {
                if (idx < cap) acc += __builtin_fabs((double)a[k] - (double)b[k]);
                ++idx;
            }
        }
        m += total;
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
