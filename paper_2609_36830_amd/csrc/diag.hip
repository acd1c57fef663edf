// Stale-k admission and admission diagnostics for gfx950.
//
// Stale-k (Sec. 2, the controlled Stale-k setting): admit a trajectory iff
// its policy lag of Eq. (1), the mean over response tokens of j - v_t, is at
// most k. By Lemma 1 the lag's numerator is S + (j - c) T, exact in int64
// from pace_score's S and T, so the test num <= k T is exact. A trajectory
// with T = 0 has lag j - c. One thread per trajectory.
//
// Diagnostics (Sec. 4, the staleness distribution diagnostics): histograms
// of K_wait, K_gen and K_eff over the candidates, retained versus rejected,
// and exact integer totals per class. One workgroup: LDS histograms with LDS
// atomics (integer, so the result does not depend on their order) and block
// sums, written once at the end; no zeroed global memory is needed.
#include "device_util.hpp"
#include "kernels.hpp"

#pragma clang fp contract(off)

namespace pace {

namespace {

__global__ __launch_bounds__(256) void stale_k_kernel(const int64_t *__restrict__ S, const int64_t *__restrict__ T,
                                                     const int32_t *__restrict__ completion, int32_t V, int64_t n,
                                                     int64_t k, uint8_t *__restrict__ keep,
                                                     double *__restrict__ lag) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int64_t t = T[i];
    const int64_t wait = (int64_t)V - (int64_t)completion[i];
    if (t > 0) {
        const int64_t num = S[i] + wait * t;
        keep[i] = (num <= k * t) ? 1 : 0;
        if (lag) lag[i] = (double)num / (double)t;
    } else {
        keep[i] = (wait <= k) ? 1 : 0;
        if (lag) lag[i] = (double)wait;
    }
}

constexpr int kDT = 1024;
constexpr int kDNW = kDT / kWave;

// Number of edges <= x (edges ascending): 0 below the first edge, nbins + 1
// at or above the last; NaN counts as below.
__device__ __forceinline__ int bin_of(const double *e, int nb1, double x) {
    int lo = 0, hi = nb1;                 // answer in [lo, hi]
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (e[mid] <= x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(kDT) void diagnostics_kernel(
    const double *__restrict__ score, const int64_t *__restrict__ S, const int64_t *__restrict__ T,
    const int32_t *__restrict__ completion, int32_t V, const uint8_t *__restrict__ keep, int64_t n,
    const double *__restrict__ edges, int nbins, int64_t *__restrict__ hist_out, int64_t *__restrict__ totals_out) {
    __shared__ double e_lds[3 * (kDiagBinsMax + 1)];
    __shared__ uint32_t h_lds[3 * 2 * (kDiagBinsMax + 2)];
    __shared__ int64_t wsum[kDNW];
    const int t = threadIdx.x;
    const int nb1 = nbins + 1, nb2 = nbins + 2;
    for (int x = t; x < 3 * nb1; x += kDT) e_lds[x] = edges[x];
    for (int x = t; x < 6 * nb2; x += kDT) h_lds[x] = 0;
    __syncthreads();
    int64_t tot[2][4] = {{0, 0, 0, 0}, {0, 0, 0, 0}};
    for (int64_t i = t; i < n; i += kDT) {
        const int64_t c = completion[i], s = S[i], tt = T[i];
        const int cls = keep[i] ? 1 : 0;
        const double m0 = (double)((int64_t)V - c);
        const double m1 = (tt > 0) ? (double)s / (double)tt : 0.0;
        const double m2 = score[i];
        atomicAdd(&h_lds[(0 * 2 + cls) * nb2 + bin_of(e_lds, nb1, m0)], 1u);
        atomicAdd(&h_lds[(1 * 2 + cls) * nb2 + bin_of(e_lds + nb1, nb1, m1)], 1u);
        atomicAdd(&h_lds[(2 * 2 + cls) * nb2 + bin_of(e_lds + 2 * nb1, nb1, m2)], 1u);
        tot[cls][0] += 1;
        tot[cls][1] += (int64_t)V - c;
        tot[cls][2] += s;
        tot[cls][3] += tt;
    }
    __syncthreads();
    for (int x = t; x < 6 * nb2; x += kDT) hist_out[x] = (int64_t)h_lds[x];
#pragma unroll
    for (int cls = 0; cls < 2; ++cls) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            int64_t total;
            (void)block_excl_sum_i64<kDNW>(tot[cls][q], total, wsum);
            if (t == 0) totals_out[cls * 4 + q] = total;
        }
    }
}

}  // namespace

hipError_t launch_stale_k(const int64_t *S, const int64_t *T, const int32_t *completion, int32_t V, int64_t n,
                          int64_t k, uint8_t *keep, double *lag, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    return launch(kPhaseAux, stale_k_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), stream, S, T, completion, V, n,
                  k, keep, lag);
}

hipError_t launch_diagnostics(const double *score, const int64_t *S, const int64_t *T, const int32_t *completion,
                              int32_t V, const uint8_t *keep, int64_t n, const double *edges, int nbins,
                              int64_t *hist, int64_t *totals, hipStream_t stream) {
    return launch(kPhaseAux, diagnostics_kernel, dim3(1), dim3(kDT), stream, score, S, T, completion, V, keep, n, edges,
                  nbins, hist, totals);
}

}  // namespace pace
