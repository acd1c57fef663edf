// pace_validate kernels for gfx950: device check of the preconditions of
// Lemma 1 (every generated token has v_t <= c(tau) <= j; versions are
// non-negative) and of the CSR layout and prefix window. Not on the hot path.
#include "../../include/pace.h"
#include "device_util.hpp"
#include "kernels.hpp"

namespace pace {

namespace {

constexpr int64_t kValChunk = 8192;   // tokens per wave

__global__ void validate_init_kernel(int32_t *err) { *err = 0; }

// One thread per trajectory (plus the window): offsets and completion versions.
__global__ __launch_bounds__(256) void validate_meta_kernel(
    const int64_t *__restrict__ off, int64_t n, int64_t NT, const int32_t *__restrict__ completion,
    int32_t V, const double *__restrict__ window, int64_t W, int32_t *err) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int32_t bad = 0;
    if (i == 0 && (off[0] != 0 || off[n] != NT)) bad |= PACE_BAD_OFFSETS;
    if (i < n) {
        if (off[i + 1] < off[i]) bad |= PACE_BAD_OFFSETS;
        const int32_t c = completion[i];
        if (c < 0 || c > V) bad |= PACE_BAD_COMPLETION;
    }
    if (i < W) {
        const double a = window[i];
        if (__builtin_isnan(a) || (i + 1 < W && !(a <= window[i + 1]))) bad |= PACE_BAD_WINDOW;
    }
    if (bad) atomicOr(err, bad);
}

// One wave per token chunk: every tag is -1 or within [0, c] of its trajectory.
__global__ __launch_bounds__(256) void validate_tags_kernel(
    const int32_t *__restrict__ tags, const int64_t *__restrict__ off, int64_t n, int64_t NT,
    const int32_t *__restrict__ completion, int64_t n_chunks, int32_t *err) {
    const int lane = lane_id();
    const int64_t chunk = (int64_t)blockIdx.x * 4 + threadIdx.x / kWave;
    if (chunk >= n_chunks) return;
    const int64_t cs = chunk * kValChunk;
    const int64_t ce = (cs + kValChunk < NT) ? cs + kValChunk : NT;
    int64_t cur = wave_last_le(off, n, cs);
    if (cur < 0) cur = 0;             // malformed offsets are reported by the meta kernel
    bool bad = false;
    while (cur < n && clamp64(off[cur + 1], 0, NT) <= cs) ++cur;
    for (int64_t w = cs; w < ce; w += kWave) {
        const int64_t p = w + lane;
        const bool in = p < ce;
        const int32_t x = in ? tags[p] : -1;
        // trajectories that meet this window of 64 tokens
        int64_t lo = w;
        const int64_t we = (w + kWave < ce) ? w + kWave : ce;
        while (cur < n) {
            const int64_t hi = clamp64(off[cur + 1], 0, NT);
            const int32_t c = completion[cur];
            if (in && p >= lo && p < hi && x != -1 && (x < 0 || x > c)) bad = true;
            if (hi >= we) break;
            lo = hi;
            ++cur;
        }
    }
    if (__popcll(ballot(bad)) && lane == 0) atomicOr(err, PACE_BAD_TAG);
}

}  // namespace

hipError_t launch_validate(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                           const int32_t *completion, int32_t V, const double *window, int64_t W,
                           int32_t *err_word, hipStream_t stream) {
    validate_init_kernel<<<1, 1, 0, stream>>>(err_word);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t m = (n + 1 > W) ? n + 1 : W;
    validate_meta_kernel<<<(unsigned)((m + 255) / 256), 256, 0, stream>>>(offsets, n, n_tokens, completion, V, window, W, err_word);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (n > 0 && n_tokens > 0) {
        const int64_t ch = (n_tokens + kValChunk - 1) / kValChunk;
        validate_tags_kernel<<<(unsigned)((ch + 3) / 4), 256, 0, stream>>>(tags, offsets, n, n_tokens, completion, ch, err_word);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace pace
