// Group-level admission for gfx950 (Appendix B: the full method aggregates
// scores by the mean within prompt groups, and its score window and
// diagnostics count groups). Consecutive trajectories form prompt groups:
// group g holds trajectories [group_offsets[g], group_offsets[g+1]). A group
// is scored by the mean of its members' scores, budgeted, selected and
// compacted as one unit. Group offsets are clamped to [0, n] on the device,
// so malformed ones give unspecified results but no out-of-bounds access.
#include "../../include/pace.h"
#include "device_util.hpp"
#include "kernels.hpp"

#pragma clang fp contract(off)

namespace pace {

namespace {

// One thread per group: the members' scores added in member order, then one
// division by the member count (the oracle's order, so the result is
// bit-identical). An empty group scores 0.
__global__ __launch_bounds__(256) void group_score_kernel(const double *__restrict__ score, int64_t n,
                                                         const int64_t *__restrict__ go, int64_t ng,
                                                         double *__restrict__ out) {
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= ng) return;
    const int64_t lo = clamp64(go[g], 0, n), hi = clamp64(go[g + 1], 0, n);
    double sum = 0.0;
    for (int64_t i = lo; i < hi; ++i) sum = sum + score[i];
    out[g] = (hi > lo) ? sum / (double)(hi - lo) : 0.0;
}

// One wave per group: every member takes its group's keep flag.
__global__ __launch_bounds__(256) void group_expand_kernel(const int64_t *__restrict__ go, int64_t ng,
                                                          int64_t n, const uint8_t *__restrict__ gkeep,
                                                          uint8_t *__restrict__ keep) {
    const int64_t g = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (g >= ng) return;
    const int64_t lo = clamp64(go[g], 0, n), hi = clamp64(go[g + 1], 0, n);
    const uint8_t k = gkeep[g] ? 1 : 0;
    for (int64_t i = lo + lane_id(); i < hi; i += kWave) keep[i] = k;
}

__global__ void group_validate_init_kernel(int32_t *err) { *err = 0; }

// group_offsets[0] = 0, non-decreasing, group_offsets[ng] = n.
__global__ __launch_bounds__(256) void group_validate_kernel(const int64_t *__restrict__ go, int64_t ng,
                                                            int64_t n, int32_t *err) {
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    bool bad = false;
    if (g == 0 && (go[0] != 0 || go[ng] != n)) bad = true;
    if (g < ng && go[g + 1] < go[g]) bad = true;
    if (bad) atomicOr(err, PACE_BAD_GROUPS);
}

}  // namespace

hipError_t launch_group_score(const double *score, int64_t n, const int64_t *group_offsets, int64_t ng,
                              double *group_score, hipStream_t stream) {
    if (ng == 0) return hipSuccess;
    return launch(kPhaseAux, group_score_kernel, dim3((unsigned)((ng + 255) / 256)), dim3(256), stream, score, n,
                  group_offsets, ng, group_score);
}

hipError_t launch_group_expand(const int64_t *group_offsets, int64_t ng, int64_t n, const uint8_t *group_keep,
                               uint8_t *keep, hipStream_t stream) {
    if (ng == 0 || n == 0) return hipSuccess;
    return launch(kPhaseAux, group_expand_kernel, dim3((unsigned)((ng + 3) / 4)), dim3(256), stream, group_offsets,
                  ng, n, group_keep, keep);
}

hipError_t launch_group_validate(const int64_t *group_offsets, int64_t ng, int64_t n, int32_t *err,
                                 hipStream_t stream) {
    group_validate_init_kernel<<<1, 1, 0, stream>>>(err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch(-1, group_validate_kernel, dim3((unsigned)(ng / 256 + 1)), dim3(256), stream, group_offsets,
                  ng, n, err);
}

hipError_t launch_group_filter_step(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                                    const int32_t *completion, int32_t V, const double *prefix,
                                    const double *window, int64_t W, bool use_prefix, double w_wait,
                                    int gamma, const int64_t *group_offsets, int64_t ng, int64_t budget,
                                    double *score, int64_t *gen_sum, int64_t *gen_count,
                                    double *group_score, uint8_t *group_keep, int32_t *reject_group_ids,
                                    uint8_t *keep, const CompactCols &cols, int n_cols,
                                    int64_t *offsets_out, int32_t *kept_ids, int64_t *n_kept_tokens,
                                    void *ws, bool vec_ok, hipStream_t stream) {
    // The workspace is a filter-step workspace sized for max(n, ng) entries.
    const int64_t N = n > ng ? n : ng;
    char *p = (char *)ws;
    const ScoreWorkspace sws = score_ws_carve(p, N, n_tokens);
    p += align256(score_ws_bytes(N, n_tokens));
    void *cws = p;
    p += align256(compact_ws_bytes(N, n_tokens));
    void *sel_ws = p;
    hipError_t e = launch_score(tags, offsets, n, n_tokens, completion, V, prefix, window, W, use_prefix,
                                w_wait, gamma, score, gen_sum, gen_count, sws, vec_ok, stream);
    if (e != hipSuccess) return e;
    e = launch_group_score(score, n, group_offsets, ng, group_score, stream);
    if (e != hipSuccess) return e;
    e = launch_select(group_score, ng, budget, group_keep, reject_group_ids, sel_ws, stream);
    if (e != hipSuccess) return e;
    e = launch_group_expand(group_offsets, ng, n, group_keep, keep, stream);
    if (e != hipSuccess) return e;
    return launch_compact(offsets, n, n_tokens, keep, cols, n_cols, offsets_out, kept_ids, n_kept_tokens, cws,
                          stream);
}

}  // namespace pace
