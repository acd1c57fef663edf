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
// and exact integer totals per class. One workgroup per metric and one for
// the totals, each over every trajectory: an LDS histogram with LDS atomics
// (integer, so the result does not depend on their order) written once at the
// end to its own rows. No zeroed global memory is needed.
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
constexpr int kDItems = 4;                // trajectories per thread per round
// LDS length of one metric's edges: a power of two >= 2 * largest power of
// two <= kDiagBinsMax + 1, so every probe of the search below is in range.
constexpr int kEdgeStride = 2048;
static_assert(kDiagBinsMax + 1 < kEdgeStride, "edge stride covers the search's probes");

// Histograms of one metric: M = 0 K_wait = V - c, 1 K_gen = S / T (0 when
// T = 0), 2 K_eff = the score; the workgroup writes rows hist_out[M][0..1][*].
template <int M>
__device__ __forceinline__ void diagnostics_metric(
    const double *__restrict__ score, const int64_t *__restrict__ S, const int64_t *__restrict__ T,
    const int32_t *__restrict__ completion, int32_t V, const uint8_t *__restrict__ keep, int64_t n,
    const double *__restrict__ edges, int nbins, int64_t *__restrict__ hist_out, double *e_lds, uint32_t *h_lds) {
    const int t = threadIdx.x;
    const int nb1 = nbins + 1, nb2 = nbins + 2;
    const int top = 1 << (31 - __builtin_clz((unsigned)nb1));   // largest power of two <= nb1
    // This metric's edges, NaN past the last.
    for (int x = t; x < nb1; x += kDT) e_lds[x] = edges[M * nb1 + x];
    for (int x = nb1 + t; x < kEdgeStride; x += kDT) e_lds[x] = __builtin_nan("");
    for (int x = t; x < 2 * nb2; x += kDT) h_lds[x] = 0;
    __syncthreads();
    // Rounds of kDItems trajectories per thread, every load of a round issued
    // before any is used: a lane past the end reads trajectory n - 1 (the loop
    // runs only when n >= 1) and drops it, so no load sits behind a branch.
    for (int64_t base = 0; base < n; base += (int64_t)kDT * kDItems) {
        int32_t c[kDItems];
        int64_t sv[kDItems], tv[kDItems];
        double m[kDItems];
        uint8_t kp[kDItems];
#pragma unroll
        for (int u = 0; u < kDItems; ++u) {
            const int64_t i = min(base + t + (int64_t)u * kDT, n - 1);
            kp[u] = keep[i];
            if constexpr (M == 0) c[u] = completion[i];
            if constexpr (M == 1) {
                sv[u] = S[i];
                tv[u] = T[i];
            }
            if constexpr (M == 2) m[u] = score[i];
        }
#pragma unroll
        for (int u = 0; u < kDItems; ++u) {
            // V and c are int32, so V - c is exact in binary64.
            if constexpr (M == 0) m[u] = (double)V - (double)c[u];
            if constexpr (M == 1) m[u] = (tv[u] > 0) ? (double)sv[u] / (double)tv[u] : 0.0;
        }
        // Bin = number of edges <= x (0 below the first edge, nbins + 1 at or
        // above the last; NaN counts as below): a branchless search by halving
        // power-of-two steps, the same number for every lane, with the
        // kDItems probes of a step issued together (a probe past the last edge
        // reads NaN and is not taken; the largest index is 2 * top - 2 <
        // kEdgeStride).
        int pos[kDItems];
#pragma unroll
        for (int u = 0; u < kDItems; ++u) pos[u] = 0;
        for (int step = top; step > 0; step >>= 1) {
#pragma unroll
            for (int u = 0; u < kDItems; ++u) {
                const int nxt = pos[u] + step;
                pos[u] = (e_lds[nxt - 1] <= m[u]) ? nxt : pos[u];
            }
        }
#pragma unroll
        for (int u = 0; u < kDItems; ++u)
            if (base + t + (int64_t)u * kDT < n) atomicAdd(&h_lds[(kp[u] ? nb2 : 0) + pos[u]], 1u);
    }
    __syncthreads();
    for (int x = t; x < 2 * nb2; x += kDT) hist_out[M * 2 * nb2 + x] = (int64_t)h_lds[x];
}

// The eight totals, by the first kTotW waves of the workgroup (kTotItems
// trajectories per thread per round); the other waves only meet the barrier.
// Counts come from ballots; the sums are kept over all candidates and over
// the retained ones, the rejected class is their difference, and
// sum (V - c) = V * count - sum c: exact integers throughout.
constexpr int kTotW = 8;
constexpr int kTotT = kTotW * kWave;
constexpr int kTotItems = 8;
__device__ __forceinline__ void diagnostics_totals(const int64_t *__restrict__ S, const int64_t *__restrict__ T,
                                                   const int32_t *__restrict__ completion, int32_t V,
                                                   const uint8_t *__restrict__ keep, int64_t n,
                                                   int64_t *__restrict__ totals_out, int64_t (*wtot)[8]) {
    const int t = threadIdx.x;
    if (t < kTotT) {
        int64_t a_c = 0, a_s = 0, a_t = 0, r_c = 0, r_s = 0, r_t = 0;
        int64_t n_a = 0, n_r = 0;   // wave-uniform
        for (int64_t base = 0; base < n; base += (int64_t)kTotT * kTotItems) {
            int32_t c[kTotItems];
            int64_t sv[kTotItems], tv[kTotItems];
            uint8_t kp[kTotItems];
#pragma unroll
            for (int u = 0; u < kTotItems; ++u) {
                const int64_t i = min(base + t + (int64_t)u * kTotT, n - 1);
                c[u] = completion[i];
                sv[u] = S[i];
                tv[u] = T[i];
                kp[u] = keep[i];
            }
#pragma unroll
            for (int u = 0; u < kTotItems; ++u) {
                const bool in = base + t + (int64_t)u * kTotT < n;
                const bool ret = in && kp[u] != 0;
                n_a += __popcll(ballot(in));
                n_r += __popcll(ballot(ret));
                a_c += in ? (int64_t)c[u] : 0;
                a_s += in ? sv[u] : 0;
                a_t += in ? tv[u] : 0;
                r_c += ret ? (int64_t)c[u] : 0;
                r_s += ret ? sv[u] : 0;
                r_t += ret ? tv[u] : 0;
            }
        }
        const int w = t / kWave;
        const int64_t sums[6] = {wave_sum_i64(a_c), wave_sum_i64(a_s), wave_sum_i64(a_t),
                                 wave_sum_i64(r_c), wave_sum_i64(r_s), wave_sum_i64(r_t)};
        if (lane_id() == 0) {
#pragma unroll
            for (int q = 0; q < 6; ++q) wtot[w][q] = sums[q];
            wtot[w][6] = n_a;
            wtot[w][7] = n_r;
        }
    }
    __syncthreads();
    if (t == 0) {
        int64_t A[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int w = 0; w < kTotW; ++w)
#pragma unroll
            for (int q = 0; q < 8; ++q) A[q] += wtot[w][q];
        const int64_t cnt_r = A[7], cnt_j = A[6] - A[7];
        totals_out[0] = cnt_j;                                 // rejected
        totals_out[1] = (int64_t)V * cnt_j - (A[0] - A[3]);
        totals_out[2] = A[1] - A[4];
        totals_out[3] = A[2] - A[5];
        totals_out[4] = cnt_r;                                 // retained
        totals_out[5] = (int64_t)V * cnt_r - A[3];
        totals_out[6] = A[4];
        totals_out[7] = A[5];
    }
}

// Four workgroups, each over every trajectory: blockIdx.x 0..2 the histograms
// of K_wait, K_gen, K_eff, 3 the totals.
__global__ __launch_bounds__(kDT) void diagnostics_kernel(
    const double *__restrict__ score, const int64_t *__restrict__ S, const int64_t *__restrict__ T,
    const int32_t *__restrict__ completion, int32_t V, const uint8_t *__restrict__ keep, int64_t n,
    const double *__restrict__ edges, int nbins, int64_t *__restrict__ hist_out, int64_t *__restrict__ totals_out) {
    __shared__ double e_lds[kEdgeStride];
    __shared__ uint32_t h_lds[2 * (kDiagBinsMax + 2)];
    __shared__ int64_t wtot[kTotW][8];
    switch (blockIdx.x) {
        case 0:
            diagnostics_metric<0>(score, S, T, completion, V, keep, n, edges, nbins, hist_out, e_lds, h_lds);
            break;
        case 1:
            diagnostics_metric<1>(score, S, T, completion, V, keep, n, edges, nbins, hist_out, e_lds, h_lds);
            break;
        case 2:
            diagnostics_metric<2>(score, S, T, completion, V, keep, n, edges, nbins, hist_out, e_lds, h_lds);
            break;
        default:
            diagnostics_totals(S, T, completion, V, keep, n, totals_out, wtot);
            break;
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
    return launch(kPhaseAux, diagnostics_kernel, dim3(4), dim3(kDT), stream, score, S, T, completion, V, keep, n, edges,
                  nbins, hist, totals);
}

}  // namespace pace
