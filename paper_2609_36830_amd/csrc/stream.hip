// The streaming admission rule for gfx950 (Sec. 3.1, Algorithm 1): the
// cutoff kappa is the (1 - r_hat)-quantile of a sliding window of recently
// observed scores; the trainer draws candidates in pool order, rejects those
// scoring above kappa and retains the rest until the batch is full.
//
// One workgroup of 1024 threads:
//   1. the window (at most kStreamWindowMax entries) goes to LDS; kappa is
//      its ceil(p * cnt)-th smallest entry, p = 1 - rate (the lower empirical
//      quantile), found by ranking every entry against all others (ties by
//      position); with fewer than window_min entries or a rate of 0 it is
//      +inf;
//   2. the draw needs no sequential walk: candidate i is drawn iff fewer
//      than batch_size candidates before it are retained, so one ordered
//      count of the retained flags (block scans over tiles of the pool)
//      gives every candidate's status, the rejected ids in order
//      (i minus the retained before i) and the draw length;
//   3. the drawn scores enter the ring in draw order (only the last `cap`
//      of them can survive), and the ring state is advanced.
#include "device_util.hpp"
#include "kernels.hpp"

#pragma clang fp contract(off)

namespace pace {

namespace {

constexpr int kST = 1024;
constexpr int kSNW = kST / kWave;
constexpr int kSItems = 8;
constexpr int64_t kSTile = (int64_t)kST * kSItems;

__global__ __launch_bounds__(kST) void stream_admit_kernel(
    const double *__restrict__ score, int64_t n, double rate, int64_t window_min, int64_t B,
    double *__restrict__ ring, int64_t cap, int64_t *__restrict__ state, uint8_t *__restrict__ status,
    uint8_t *__restrict__ keep, int32_t *__restrict__ reject_ids, double *__restrict__ kappa_out,
    int64_t *__restrict__ counts) {
    __shared__ double win[kStreamWindowMax];
    __shared__ uint32_t wsum[kSNW];
    __shared__ double s_kappa;
    __shared__ int64_t s_state[2];
    const int t = threadIdx.x;
    // The first tile's scores do not depend on the cutoff: their loads go
    // out first (a slot past the end reads the last score and is dropped).
    double sc[kSItems];
    if (n > 0) {
#pragma unroll
        for (int q = 0; q < kSItems; ++q) sc[q] = score[min((int64_t)t * kSItems + q, n - 1)];
    }
    if (t == 0) {
        s_state[0] = state[0];
        s_state[1] = state[1];
        s_kappa = __builtin_inf();
    }
    __syncthreads();
    const int64_t head = clamp64(s_state[0], 0, cap - 1);
    const int64_t cnt = clamp64(s_state[1], 0, cap);

    // 1. The cutoff, from the window as it stands before this draw (the cnt
    //    most recent entries end just before head).
    for (int64_t u = t; u < cnt; u += kST) {
        const int64_t at = head - cnt + u;        // in [-cap, cap): head < cap, u < cnt <= cap
        win[u] = ring[at < 0 ? at + cap : at];
    }
    __syncthreads();
    if (cnt >= window_min && cnt > 0 && rate > 0.0) {
        const double p = 1.0 - rate;
        int64_t k = (int64_t)ceil(p * (double)cnt);
        if (k < 1) k = 1;
        // P adjacent lanes share an entry, each counting over a 1/P slice of
        // the window (P = 8, 4, 2 or 1, as many as the threads allow); the
        // lanes' counts are added by shuffles.
        const int P = (8 * cnt <= kST) ? 8 : (4 * cnt <= kST) ? 4 : (2 * cnt <= kST) ? 2 : 1;
        const int sub = t & (P - 1);
        const int64_t slice = (cnt + P - 1) / P;
        const int64_t v0 = sub * slice, v1 = (v0 + slice < cnt) ? v0 + slice : cnt;
        for (int64_t u0 = 0; u0 < cnt; u0 += kST / P) {
            const int64_t u = u0 + t / P;
            const bool has = u < cnt;
            const double x = has ? win[u] : 0.0;
            uint32_t r = 0;
            if (has)
                for (int64_t v = v0; v < v1; ++v) {
                    const double y = win[v];
                    r += (y < x || (y == x && v < u)) ? 1u : 0u;
                }
            for (int o = 1; o < P; o <<= 1) r += (uint32_t)__shfl_xor((int)r, o, kWave);
            if (has && sub == 0 && (int64_t)r == k - 1) s_kappa = x;
        }
        __syncthreads();
    }
    const double kappa = s_kappa;

    // 2. The draw.
    int64_t run_ret = 0, drawn = 0;
    for (int64_t base = 0; base < n; base += kSTile) {
        const int64_t i0 = base + (int64_t)t * kSItems;
        bool in[kSItems], ret[kSItems];
        uint32_t c = 0;
        if (base > 0) {
#pragma unroll
            for (int q = 0; q < kSItems; ++q) sc[q] = score[min(i0 + q, n - 1)];
        }
#pragma unroll
        for (int q = 0; q < kSItems; ++q) {
            in[q] = i0 + q < n;
            ret[q] = in[q] && !(sc[q] > kappa);
            c += ret[q] ? 1u : 0u;
        }
        uint32_t tot;
        const uint32_t before = block_excl_sum_u32<kSNW>(c, tot, wsum);
        int64_t rb = run_ret + before;          // retained before item i0 + q
        uint32_t d = 0;
#pragma unroll
        for (int q = 0; q < kSItems; ++q) {
            if (!in[q]) continue;
            const int64_t i = i0 + q;
            const bool is_drawn = rb < B;
            uint8_t st = 2;
            if (is_drawn) {
                st = ret[q] ? 1 : 0;
                if (!ret[q]) reject_ids[i - rb] = (int32_t)i;
                d += 1;
            }
            status[i] = st;
            keep[i] = st == 1 ? 1 : 0;
            rb += ret[q] ? 1 : 0;
        }
        uint32_t dtot;
        (void)block_excl_sum_u32<kSNW>(d, dtot, wsum);
        drawn += dtot;
        run_ret += tot;
    }
    const int64_t retained = run_ret < B ? run_ret : B;

    // 3. The window takes the drawn scores, oldest first.
    const int64_t first = drawn > cap ? drawn - cap : 0;
    for (int64_t u = first + t; u < drawn; u += kST) ring[(head + u) % cap] = score[u];
    if (t == 0) {
        state[0] = (head + drawn) % cap;
        state[1] = (cnt + drawn < cap) ? cnt + drawn : cap;
        *kappa_out = kappa;
        counts[0] = drawn;
        counts[1] = retained;
        counts[2] = drawn - retained;
    }
}

}  // namespace

hipError_t launch_stream_admit(const double *score, int64_t n, double rate, int64_t window_min, int64_t B,
                               double *ring, int64_t cap, int64_t *state, uint8_t *status, uint8_t *keep,
                               int32_t *reject_ids, double *kappa, int64_t *counts, hipStream_t stream) {
    return launch(kPhaseSelect, stream_admit_kernel, dim3(1), dim3(kST), stream, score, n, rate, window_min, B,
                  ring, cap, state, status, keep, reject_ids, kappa, counts);
}

}  // namespace pace
