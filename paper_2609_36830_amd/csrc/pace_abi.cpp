// C ABI of the PACE filter step (declared in include/pace.h): host-side
// argument checks, workspace carving and kernel launches. All device work is
// enqueued on the caller's stream; nothing here allocates or synchronises.
#include <math.h>
#include <atomic>
#include <stdint.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "../../include/pace.h"
#include "kernels.hpp"

#pragma clang fp contract(off)

using namespace pace;

namespace {

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

pace_params params_or_default(const pace_params *p) {
    pace_params d;
    pace_default_params(&d);
    return p ? *p : d;
}

int64_t ipow_checked(int64_t x, int g, bool *overflow) {
    // x^g for the 2^53 check of the prefix window; saturates on overflow
    int64_t r = 1;
    for (int k = 0; k < g; ++k) {
        if (x != 0 && r > INT64_MAX / x) {
            *overflow = true;
            return INT64_MAX;
        }
        r *= x;
    }
    return r;
}

int hip_status(hipError_t e) { return e == hipSuccess ? PACE_OK : PACE_ERR_HIP; }

}  // namespace

namespace pace {

int64_t resident_waves() {
    // CU count per device, queried once per device (the attribute is constant).
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256 * 16;
    int cu = cache[dev].load(std::memory_order_relaxed);
    if (cu <= 0) {
        if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cu <= 0)
            cu = 256;
        cache[dev].store(cu, std::memory_order_relaxed);
    }
    return (int64_t)cu * 16;
}

namespace {
// Armed timers, per host thread: [phase][start, stop].
thread_local hipEvent_t g_phase_timer[kPhaseCount][2];
}  // namespace

bool take_phase_timer(int phase, hipEvent_t *start, hipEvent_t *stop) {
    if (phase < 0 || phase >= kPhaseCount || g_phase_timer[phase][0] == nullptr) return false;
    *start = g_phase_timer[phase][0];
    *stop = g_phase_timer[phase][1];
    g_phase_timer[phase][0] = g_phase_timer[phase][1] = nullptr;
    return true;
}

namespace {
// Every entry point that enqueues device work holds one of these: when the
// call returns, the thread's armed timers are dropped, used or not, so a
// timer never reaches a later call.
struct TimerScope {
    TimerScope() = default;
    TimerScope(const TimerScope &) = delete;
    TimerScope &operator=(const TimerScope &) = delete;
    ~TimerScope() {
        for (int k = 0; k < kPhaseCount; ++k) g_phase_timer[k][0] = g_phase_timer[k][1] = nullptr;
    }
};
}  // namespace

}  // namespace pace

extern "C" {

void pace_default_params(pace_params *p) {
    if (!p) return;
    p->w_wait = 1.0;
    p->gamma = 4;
    p->window_min = 32;
    p->beta = 0.0;
    p->r_max = 0.9;
}

const char *pace_strerror(int code) {
    switch (code) {
        case PACE_OK: return "ok";
        case PACE_ERR_INVALID_ARG: return "invalid argument";
        case PACE_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
        case PACE_ERR_PRECONDITION: return "data precondition violated";
        case PACE_ERR_HIP: return "HIP launch failure";
        case PACE_ERR_SCRATCH_LIMIT: return "pool too large for the fixed device scratch";
        default: return "unknown error code";
    }
}

int pace_workspace_bytes(int which, int64_t n_traj, int64_t n_tokens, size_t *bytes_out) {
    if (!bytes_out || n_traj < 0 || n_tokens < 0) return PACE_ERR_INVALID_ARG;
    switch (which) {
        case PACE_WS_SCORE: *bytes_out = score_ws_bytes(n_traj, n_tokens); return PACE_OK;
        case PACE_WS_SELECT: *bytes_out = select_ws_bytes(n_traj); return PACE_OK;
        case PACE_WS_COMPACT: *bytes_out = compact_ws_bytes(n_traj, n_tokens); return PACE_OK;
        case PACE_WS_FILTER_STEP: *bytes_out = filter_step_ws_bytes(n_traj, n_tokens); return PACE_OK;
        default: return PACE_ERR_INVALID_ARG;
    }
}

static int check_score_args(const int32_t *tags, const int64_t *offsets, int64_t n_traj,
                            int64_t n_tokens, const int32_t *completion, int32_t current_version,
                            const double *prefix_score, const double *window_sorted,
                            int64_t window_n, const pace_params &p, const double *score_out,
                            const int64_t *gen_sum_out, const int64_t *gen_count_out) {
    if (n_traj < 0 || n_traj >= INT32_MAX || n_tokens < 0 || window_n < 0) return PACE_ERR_INVALID_ARG;
    if (!offsets || (n_traj > 0 && (!completion || !score_out)) || (n_tokens > 0 && !tags))
        return PACE_ERR_INVALID_ARG;
    if (!aligned(tags, 4) || !aligned(offsets, 8) || !aligned(completion, 4) ||
        !aligned(score_out, 8) || !aligned(gen_sum_out, 8) || !aligned(gen_count_out, 8) ||
        !aligned(prefix_score, 8) || !aligned(window_sorted, 8))
        return PACE_ERR_INVALID_ARG;
    if (current_version < 0 || current_version == INT32_MAX) return PACE_ERR_INVALID_ARG;
    if (!(p.w_wait >= 0.0) || isinf(p.w_wait) || p.gamma < 1 || p.gamma > 4 || p.window_min < 0)
        return PACE_ERR_INVALID_ARG;
    if (window_n > 0 && !window_sorted) return PACE_ERR_INVALID_ARG;
    bool of = false;
    if (window_n > 0 && (ipow_checked(window_n, p.gamma, &of) >= ((int64_t)1 << 53) || of))
        return PACE_ERR_INVALID_ARG;
    return PACE_OK;
}

static int check_compact_args(const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                              const uint8_t *keep, int n_cols, const void *const *cols_in,
                              const int32_t *elem_bytes, void *const *cols_out,
                              const int64_t *offsets_out, const int32_t *kept_ids_out,
                              const int64_t *n_kept_tokens_out, CompactCols *cols) {
    if (n_traj < 0 || n_traj >= INT32_MAX || n_tokens < 0 || n_cols < 0 || n_cols > kMaxCols)
        return PACE_ERR_INVALID_ARG;
    if (!offsets || !offsets_out || !n_kept_tokens_out || (n_traj > 0 && (!keep || !kept_ids_out)))
        return PACE_ERR_INVALID_ARG;
    if (!aligned(offsets, 8) || !aligned(offsets_out, 8) || !aligned(n_kept_tokens_out, 8) ||
        !aligned(kept_ids_out, 4))
        return PACE_ERR_INVALID_ARG;
    if (n_cols > 0 && (!cols_in || !cols_out || !elem_bytes)) return PACE_ERR_INVALID_ARG;
    memset(cols, 0, sizeof(*cols));
    for (int c = 0; c < n_cols; ++c) {
        const int32_t e = elem_bytes[c];
        if (!(e == 1 || e == 2 || e == 4 || e == 8)) return PACE_ERR_INVALID_ARG;
        if (n_tokens > 0 && (!cols_in[c] || !cols_out[c])) return PACE_ERR_INVALID_ARG;
        if (!aligned(cols_in[c], (uintptr_t)e) || !aligned(cols_out[c], (uintptr_t)e))
            return PACE_ERR_INVALID_ARG;
        if (n_tokens > INT64_MAX / 8) return PACE_ERR_INVALID_ARG;
        cols->in[c] = cols_in[c];
        cols->out[c] = cols_out[c];
        cols->elem[c] = e;
        cols->vec[c] = (aligned(cols_in[c], 16) && aligned(cols_out[c], 16)) ? 1 : 0;
    }
    return PACE_OK;
}

int pace_score(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
               const int32_t *completion, int32_t current_version, const double *prefix_score,
               const double *window_sorted, int64_t window_n, const pace_params *params,
               double *score_out, int64_t *gen_sum_out, int64_t *gen_count_out, void *workspace,
               size_t workspace_bytes, void *stream) {
    const TimerScope timers;
    const pace_params p = params_or_default(params);
    int rc = check_score_args(tags, offsets, n_traj, n_tokens, completion, current_version,
                              prefix_score, window_sorted, window_n, p, score_out, gen_sum_out,
                              gen_count_out);
    if (rc != PACE_OK) return rc;
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < score_ws_bytes(n_traj, n_tokens))
        return PACE_ERR_WORKSPACE;
    const int64_t wmin = p.window_min > 1 ? p.window_min : 1;
    const bool use_prefix = prefix_score != nullptr && window_n >= wmin;
    const ScoreWorkspace ws = score_ws_carve(workspace, n_traj, n_tokens);
    return hip_status(launch_score(tags, offsets, n_traj, n_tokens, completion, current_version,
                                   prefix_score, window_sorted, window_n, use_prefix, p.w_wait,
                                   p.gamma, score_out, gen_sum_out, gen_count_out, ws,
                                   aligned(tags, 16), (hipStream_t)stream));
}

static int budget_impl(int64_t occupancy, int64_t capacity, const pace_params *params,
                       double *r_hat_inout, int64_t *budget_out) {
    const pace_params p = params_or_default(params);
    if (!r_hat_inout || !budget_out || occupancy < 0 || capacity < 0) return PACE_ERR_INVALID_ARG;
    if (!(p.beta >= 0.0 && p.beta < 1.0) || !(p.r_max >= 0.0 && p.r_max <= 1.0))
        return PACE_ERR_INVALID_ARG;
    const double prev = *r_hat_inout;
    if (!(prev >= 0.0) || isinf(prev)) return PACE_ERR_INVALID_ARG;
    // Eq. (3): fraction of the pool above the target occupancy, clipped.
    const double surplus_frac = (double)(occupancy - capacity) / (double)(occupancy > 1 ? occupancy : 1);
    const double r = surplus_frac < 0.0 ? 0.0 : (surplus_frac > 1.0 ? 1.0 : surplus_frac);
    // Eq. (4): exponential smoothing (two products then one sum, never fused).
    const double kept_part = p.beta * prev;
    const double new_part = (1.0 - p.beta) * r;
    const double r_hat = kept_part + new_part;
    int64_t b = 0;
    if (occupancy > capacity) {
        const double capped = r_hat < p.r_max ? r_hat : p.r_max;
        b = (int64_t)nearbyint(capped * (double)occupancy);   // ties to even
        const int64_t surplus = occupancy - capacity;
        if (b > surplus) b = surplus;
        if (b < 0) b = 0;
    }
    *r_hat_inout = r_hat;
    *budget_out = b;
    return PACE_OK;
}

int pace_budget(int64_t occupancy, int64_t capacity, const pace_params *params,
                double *r_hat_inout, int64_t *budget_out) {
    return budget_impl(occupancy, capacity, params, r_hat_inout, budget_out);
}

int pace_select(const double *score, int64_t n_traj, int64_t budget, uint8_t *keep_out,
                int32_t *reject_ids_out, void *workspace, size_t workspace_bytes, void *stream) {
    const TimerScope timers;
    if (n_traj < 0 || n_traj >= INT32_MAX || budget < 0 || budget > n_traj) return PACE_ERR_INVALID_ARG;
    if (n_traj > 0 && (!score || !keep_out)) return PACE_ERR_INVALID_ARG;
    if (budget > 0 && !reject_ids_out) return PACE_ERR_INVALID_ARG;
    if (!aligned(score, 8) || !aligned(reject_ids_out, 4)) return PACE_ERR_INVALID_ARG;
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < select_ws_bytes(n_traj))
        return PACE_ERR_WORKSPACE;
    return hip_status(launch_select(score, n_traj, budget, keep_out, reject_ids_out, workspace,
                                    (hipStream_t)stream));
}

int pace_compact(const int64_t *offsets, int64_t n_traj, int64_t n_tokens, const uint8_t *keep,
                 int n_cols, const void *const *cols_in, const int32_t *elem_bytes,
                 void *const *cols_out, int64_t *offsets_out, int32_t *kept_ids_out,
                 int64_t *n_kept_tokens_out, void *workspace, size_t workspace_bytes,
                 void *stream) {
    const TimerScope timers;
    CompactCols cols;
    int rc = check_compact_args(offsets, n_traj, n_tokens, keep, n_cols, cols_in, elem_bytes, cols_out,
                                offsets_out, kept_ids_out, n_kept_tokens_out, &cols);
    if (rc != PACE_OK) return rc;
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < compact_ws_bytes(n_traj, n_tokens))
        return PACE_ERR_WORKSPACE;
    return hip_status(launch_compact(offsets, n_traj, n_tokens, keep, cols, n_cols, offsets_out,
                                     kept_ids_out, n_kept_tokens_out, workspace, (hipStream_t)stream));
}

// pace_filter_step's checks and launches. With scratch_limit set, the
// workspace is the fixed device scratch: a pool whose workspace exceeds it is
// refused with PACE_ERR_SCRATCH_LIMIT after the argument checks, and
// `workspace` is looked up only then.
static int filter_step_impl(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                            const int32_t *completion, int32_t current_version,
                            const double *prefix_score, const double *window_sorted, int64_t window_n,
                            int64_t occupancy, int64_t capacity, const pace_params *params,
                            double *r_hat_inout, int64_t *budget_out, double *score_out,
                            int64_t *gen_sum_out, int64_t *gen_count_out, uint8_t *keep_out,
                            int32_t *reject_ids_out, int n_cols, const void *const *cols_in,
                            const int32_t *elem_bytes, void *const *cols_out, int64_t *offsets_out,
                            int32_t *kept_ids_out, int64_t *n_kept_tokens_out, void *workspace,
                            size_t workspace_bytes, bool scratch_limit, void *stream) {
    const pace_params p = params_or_default(params);
    int rc = check_score_args(tags, offsets, n_traj, n_tokens, completion, current_version,
                              prefix_score, window_sorted, window_n, p, score_out, gen_sum_out,
                              gen_count_out);
    if (rc != PACE_OK) return rc;
    CompactCols cols;
    rc = check_compact_args(offsets, n_traj, n_tokens, keep_out, n_cols, cols_in, elem_bytes,
                            cols_out, offsets_out, kept_ids_out, n_kept_tokens_out, &cols);
    if (rc != PACE_OK) return rc;
    if (n_traj > 0 && !keep_out) return PACE_ERR_INVALID_ARG;
    if (!r_hat_inout || !budget_out || !aligned(reject_ids_out, 4)) return PACE_ERR_INVALID_ARG;
    if (scratch_limit) {
        if (filter_step_ws_bytes(n_traj, n_tokens) > (size_t)PACE_NOALLOC_SCRATCH_BYTES)
            return PACE_ERR_SCRATCH_LIMIT;
        if (noalloc_scratch(&workspace) != hipSuccess) return PACE_ERR_HIP;
        workspace_bytes = PACE_NOALLOC_SCRATCH_BYTES;
    }
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < filter_step_ws_bytes(n_traj, n_tokens))
        return PACE_ERR_WORKSPACE;
    double r_hat = *r_hat_inout;
    int64_t budget = 0;
    rc = budget_impl(occupancy, capacity, &p, &r_hat, &budget);
    if (rc != PACE_OK) return rc;
    if (budget > n_traj || (budget > 0 && !reject_ids_out)) return PACE_ERR_INVALID_ARG;
    const int64_t wmin = p.window_min > 1 ? p.window_min : 1;
    const bool use_prefix = prefix_score != nullptr && window_n >= wmin;
    rc = hip_status(launch_filter_step(tags, offsets, n_traj, n_tokens, completion, current_version,
                                       prefix_score, window_sorted, window_n, use_prefix, p.w_wait,
                                       p.gamma, budget, score_out, gen_sum_out, gen_count_out,
                                       keep_out, reject_ids_out, cols, n_cols, offsets_out,
                                       kept_ids_out, n_kept_tokens_out, workspace, aligned(tags, 16),
                                       (hipStream_t)stream));
    if (rc != PACE_OK) return rc;
    *r_hat_inout = r_hat;
    *budget_out = budget;
    return PACE_OK;
}

int pace_filter_step(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                     const int32_t *completion, int32_t current_version,
                     const double *prefix_score, const double *window_sorted, int64_t window_n,
                     int64_t occupancy, int64_t capacity, const pace_params *params,
                     double *r_hat_inout, int64_t *budget_out, double *score_out,
                     int64_t *gen_sum_out, int64_t *gen_count_out, uint8_t *keep_out,
                     int32_t *reject_ids_out, int n_cols, const void *const *cols_in,
                     const int32_t *elem_bytes, void *const *cols_out, int64_t *offsets_out,
                     int32_t *kept_ids_out, int64_t *n_kept_tokens_out, void *workspace,
                     size_t workspace_bytes, void *stream) {
    const TimerScope timers;
    return filter_step_impl(tags, offsets, n_traj, n_tokens, completion, current_version, prefix_score,
                            window_sorted, window_n, occupancy, capacity, params, r_hat_inout, budget_out,
                            score_out, gen_sum_out, gen_count_out, keep_out, reject_ids_out, n_cols, cols_in,
                            elem_bytes, cols_out, offsets_out, kept_ids_out, n_kept_tokens_out, workspace,
                            workspace_bytes, false, stream);
}

int pace_filter_step_noalloc(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                             const int32_t *completion, int32_t current_version,
                             const double *prefix_score, const double *window_sorted, int64_t window_n,
                             int64_t occupancy, int64_t capacity, const pace_params *params,
                             double *r_hat_inout, int64_t *budget_out, double *score_out,
                             int64_t *gen_sum_out, int64_t *gen_count_out, uint8_t *keep_out,
                             int32_t *reject_ids_out, int n_cols, const void *const *cols_in,
                             const int32_t *elem_bytes, void *const *cols_out, int64_t *offsets_out,
                             int32_t *kept_ids_out, int64_t *n_kept_tokens_out, void *stream) {
    const TimerScope timers;
    return filter_step_impl(tags, offsets, n_traj, n_tokens, completion, current_version, prefix_score,
                            window_sorted, window_n, occupancy, capacity, params, r_hat_inout, budget_out,
                            score_out, gen_sum_out, gen_count_out, keep_out, reject_ids_out, n_cols, cols_in,
                            elem_bytes, cols_out, offsets_out, kept_ids_out, n_kept_tokens_out, nullptr, 0,
                            true, stream);
}

static int check_groups_arg(const int64_t *group_offsets, int64_t n_groups) {
    if (n_groups < 0 || n_groups >= INT32_MAX || !group_offsets || !aligned(group_offsets, 8))
        return PACE_ERR_INVALID_ARG;
    return PACE_OK;
}

int pace_group_score(const double *score, int64_t n_traj, const int64_t *group_offsets, int64_t n_groups,
                     double *group_score_out, void *stream) {
    const TimerScope timers;
    if (n_traj < 0 || n_traj >= INT32_MAX || check_groups_arg(group_offsets, n_groups) != PACE_OK)
        return PACE_ERR_INVALID_ARG;
    if ((n_traj > 0 && !score) || (n_groups > 0 && !group_score_out) || !aligned(score, 8) ||
        !aligned(group_score_out, 8))
        return PACE_ERR_INVALID_ARG;
    return hip_status(launch_group_score(score, n_traj, group_offsets, n_groups, group_score_out,
                                         (hipStream_t)stream));
}

int pace_group_expand(const int64_t *group_offsets, int64_t n_groups, int64_t n_traj,
                      const uint8_t *group_keep, uint8_t *keep_out, void *stream) {
    const TimerScope timers;
    if (n_traj < 0 || n_traj >= INT32_MAX || check_groups_arg(group_offsets, n_groups) != PACE_OK)
        return PACE_ERR_INVALID_ARG;
    if ((n_groups > 0 && !group_keep) || (n_traj > 0 && !keep_out)) return PACE_ERR_INVALID_ARG;
    return hip_status(launch_group_expand(group_offsets, n_groups, n_traj, group_keep, keep_out,
                                          (hipStream_t)stream));
}

int pace_validate_groups(const int64_t *group_offsets, int64_t n_groups, int64_t n_traj,
                         int32_t *err_word_out, void *stream) {
    const TimerScope timers;
    if (n_traj < 0 || n_traj >= INT32_MAX || check_groups_arg(group_offsets, n_groups) != PACE_OK)
        return PACE_ERR_INVALID_ARG;
    if (!err_word_out || !aligned(err_word_out, 4)) return PACE_ERR_INVALID_ARG;
    return hip_status(launch_group_validate(group_offsets, n_groups, n_traj, err_word_out,
                                            (hipStream_t)stream));
}

int pace_group_filter_step(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                           const int32_t *completion, int32_t current_version,
                           const double *prefix_score, const double *window_sorted, int64_t window_n,
                           const int64_t *group_offsets, int64_t n_groups, int64_t occupancy,
                           int64_t capacity, const pace_params *params, double *r_hat_inout,
                           int64_t *budget_out, double *score_out, int64_t *gen_sum_out,
                           int64_t *gen_count_out, double *group_score_out, uint8_t *group_keep_out,
                           int32_t *reject_group_ids_out, uint8_t *keep_out, int n_cols,
                           const void *const *cols_in, const int32_t *elem_bytes, void *const *cols_out,
                           int64_t *offsets_out, int32_t *kept_ids_out, int64_t *n_kept_tokens_out,
                           void *workspace, size_t workspace_bytes, void *stream) {
    const TimerScope timers;
    const pace_params p = params_or_default(params);
    int rc = check_score_args(tags, offsets, n_traj, n_tokens, completion, current_version,
                              prefix_score, window_sorted, window_n, p, score_out, gen_sum_out,
                              gen_count_out);
    if (rc != PACE_OK) return rc;
    if (check_groups_arg(group_offsets, n_groups) != PACE_OK) return PACE_ERR_INVALID_ARG;
    if (n_groups > 0 && (!group_score_out || !group_keep_out)) return PACE_ERR_INVALID_ARG;
    if (!aligned(group_score_out, 8) || !aligned(reject_group_ids_out, 4)) return PACE_ERR_INVALID_ARG;
    CompactCols cols;
    rc = check_compact_args(offsets, n_traj, n_tokens, keep_out, n_cols, cols_in, elem_bytes,
                            cols_out, offsets_out, kept_ids_out, n_kept_tokens_out, &cols);
    if (rc != PACE_OK) return rc;
    if (!r_hat_inout || !budget_out) return PACE_ERR_INVALID_ARG;
    const int64_t N = n_traj > n_groups ? n_traj : n_groups;
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < filter_step_ws_bytes(N, n_tokens))
        return PACE_ERR_WORKSPACE;
    double r_hat = *r_hat_inout;
    int64_t budget = 0;
    rc = budget_impl(occupancy, capacity, &p, &r_hat, &budget);
    if (rc != PACE_OK) return rc;
    if (budget > n_groups || (budget > 0 && !reject_group_ids_out)) return PACE_ERR_INVALID_ARG;
    const int64_t wmin = p.window_min > 1 ? p.window_min : 1;
    const bool use_prefix = prefix_score != nullptr && window_n >= wmin;
    rc = hip_status(launch_group_filter_step(
        tags, offsets, n_traj, n_tokens, completion, current_version, prefix_score, window_sorted, window_n,
        use_prefix, p.w_wait, p.gamma, group_offsets, n_groups, budget, score_out, gen_sum_out, gen_count_out,
        group_score_out, group_keep_out, reject_group_ids_out, keep_out, cols, n_cols, offsets_out, kept_ids_out,
        n_kept_tokens_out, workspace, aligned(tags, 16), (hipStream_t)stream));
    if (rc != PACE_OK) return rc;
    *r_hat_inout = r_hat;
    *budget_out = budget;
    return PACE_OK;
}

int pace_stream_admit(const double *score, int64_t n_traj, double r_hat, const pace_params *params,
                      int64_t batch_size, double *window_ring, int64_t window_cap, int64_t *window_state,
                      uint8_t *status_out, uint8_t *keep_out, int32_t *reject_ids_out, double *kappa_out,
                      int64_t *counts_out, void *stream) {
    const TimerScope timers;
    const pace_params p = params_or_default(params);
    if (n_traj < 0 || n_traj >= INT32_MAX || batch_size < 0) return PACE_ERR_INVALID_ARG;
    if (!(r_hat >= 0.0) || isinf(r_hat) || !(p.r_max >= 0.0 && p.r_max <= 1.0) || p.window_min < 0)
        return PACE_ERR_INVALID_ARG;
    if (window_cap < 1 || window_cap > kStreamWindowMax || !window_ring || !window_state || !kappa_out ||
        !counts_out)
        return PACE_ERR_INVALID_ARG;
    if (n_traj > 0 && (!score || !status_out || !keep_out || !reject_ids_out)) return PACE_ERR_INVALID_ARG;
    if (!aligned(score, 8) || !aligned(window_ring, 8) || !aligned(window_state, 8) || !aligned(kappa_out, 8) ||
        !aligned(counts_out, 8) || !aligned(reject_ids_out, 4))
        return PACE_ERR_INVALID_ARG;
    const double rate = r_hat < p.r_max ? r_hat : p.r_max;
    return hip_status(launch_stream_admit(score, n_traj, rate, p.window_min, batch_size, window_ring,
                                          window_cap, window_state, status_out, keep_out, reject_ids_out,
                                          kappa_out, counts_out, nullptr, 0, PieceParts{}, (hipStream_t)stream));
}

int pace_stream_step(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                     const int32_t *completion, int32_t current_version, const double *prefix_score,
                     const double *window_sorted, int64_t window_n, int64_t occupancy, int64_t capacity,
                     const pace_params *params, double *r_hat_inout, int64_t batch_size,
                     double *window_ring, int64_t window_cap, int64_t *window_state, double *score_out,
                     int64_t *gen_sum_out, int64_t *gen_count_out, uint8_t *status_out, uint8_t *keep_out,
                     int32_t *reject_ids_out, double *kappa_out, int64_t *counts_out, int n_cols,
                     const void *const *cols_in, const int32_t *elem_bytes, void *const *cols_out,
                     int64_t *offsets_out, int32_t *kept_ids_out, int64_t *n_kept_tokens_out,
                     void *workspace, size_t workspace_bytes, void *stream) {
    const TimerScope timers;
    const pace_params p = params_or_default(params);
    int rc = check_score_args(tags, offsets, n_traj, n_tokens, completion, current_version,
                              prefix_score, window_sorted, window_n, p, score_out, gen_sum_out,
                              gen_count_out);
    if (rc != PACE_OK) return rc;
    CompactCols cols;
    rc = check_compact_args(offsets, n_traj, n_tokens, keep_out, n_cols, cols_in, elem_bytes,
                            cols_out, offsets_out, kept_ids_out, n_kept_tokens_out, &cols);
    if (rc != PACE_OK) return rc;
    if (!r_hat_inout || batch_size < 0 || window_cap < 1 || window_cap > kStreamWindowMax || !window_ring ||
        !window_state || !kappa_out || !counts_out)
        return PACE_ERR_INVALID_ARG;
    if (n_traj > 0 && (!status_out || !keep_out || !reject_ids_out)) return PACE_ERR_INVALID_ARG;
    if (!aligned(window_ring, 8) || !aligned(window_state, 8) || !aligned(kappa_out, 8) ||
        !aligned(counts_out, 8) || !aligned(reject_ids_out, 4))
        return PACE_ERR_INVALID_ARG;
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < filter_step_ws_bytes(n_traj, n_tokens))
        return PACE_ERR_WORKSPACE;
    double r_hat = *r_hat_inout;
    int64_t budget = 0;
    rc = budget_impl(occupancy, capacity, &p, &r_hat, &budget);
    if (rc != PACE_OK) return rc;
    const int64_t wmin = p.window_min > 1 ? p.window_min : 1;
    const bool use_prefix = prefix_score != nullptr && window_n >= wmin;
    char *w = (char *)workspace;
    const ScoreWorkspace sws = score_ws_carve(w, n_traj, n_tokens);
    void *cws = w + align256(score_ws_bytes(n_traj, n_tokens));
    hipStream_t st = (hipStream_t)stream;
    hipError_t e = launch_score(tags, offsets, n_traj, n_tokens, completion, current_version, prefix_score,
                                window_sorted, window_n, use_prefix, p.w_wait, p.gamma, score_out, gen_sum_out,
                                gen_count_out, sws, aligned(tags, 16), st);
    // Pools the piece compaction takes get their block partials from the
    // draw itself; the kept trajectories are at most min(batch_size, n).
    const bool pieces = compact_piece_ok(n_traj, n_tokens);
    const CompactWs cw = compact_ws_carve(cws, n_traj, n_tokens);
    if (e == hipSuccess) {
        const double rate = r_hat < p.r_max ? r_hat : p.r_max;
        e = launch_stream_admit(score_out, n_traj, rate, p.window_min, batch_size, window_ring, window_cap,
                                window_state, status_out, keep_out, reject_ids_out, kappa_out, counts_out,
                                pieces ? offsets : nullptr, n_tokens, pieces ? cw.parts : PieceParts{}, st);
    }
    if (e == hipSuccess) {
        if (pieces)
            e = launch_compact_pieces(offsets, n_traj, n_tokens, keep_out, cw.parts, cols, n_cols, offsets_out,
                                      kept_ids_out, n_kept_tokens_out, nullptr, 0,
                                      batch_size < n_traj ? batch_size : n_traj, st);
        else
            e = launch_compact(offsets, n_traj, n_tokens, keep_out, cols, n_cols, offsets_out, kept_ids_out,
                               n_kept_tokens_out, cws, st);
    }
    rc = hip_status(e);
    if (rc != PACE_OK) return rc;
    *r_hat_inout = r_hat;
    return PACE_OK;
}

int pace_prefix_score(const float *lp_new, const float *lp_behavior, const int32_t *tags,
                      const int64_t *prefix_offsets, int64_t n, int64_t n_tokens, int64_t cap,
                      int64_t min_tokens, double *s_pre_out, void *stream) {
    const TimerScope timers;
    if (n < 0 || n >= INT32_MAX || n_tokens < 0 || cap < 0 || min_tokens < 0 || !prefix_offsets)
        return PACE_ERR_INVALID_ARG;
    if ((n > 0 && !s_pre_out) || (n_tokens > 0 && (!lp_new || !lp_behavior))) return PACE_ERR_INVALID_ARG;
    if (!aligned(lp_new, 4) || !aligned(lp_behavior, 4) || !aligned(tags, 4) || !aligned(prefix_offsets, 8) ||
        !aligned(s_pre_out, 8))
        return PACE_ERR_INVALID_ARG;
    return hip_status(launch_prefix_score(lp_new, lp_behavior, tags, prefix_offsets, n, n_tokens, cap, min_tokens,
                                          s_pre_out, (hipStream_t)stream));
}

int pace_stale_k(const int64_t *gen_sum, const int64_t *gen_count, const int32_t *completion,
                 int32_t current_version, int64_t n_traj, int64_t k, uint8_t *keep_out, double *lag_out,
                 void *stream) {
    const TimerScope timers;
    if (n_traj < 0 || n_traj >= INT32_MAX || k < 0 || k >= INT32_MAX || current_version < 0)
        return PACE_ERR_INVALID_ARG;
    if (n_traj > 0 && (!gen_sum || !gen_count || !completion || !keep_out)) return PACE_ERR_INVALID_ARG;
    if (!aligned(gen_sum, 8) || !aligned(gen_count, 8) || !aligned(completion, 4) || !aligned(lag_out, 8))
        return PACE_ERR_INVALID_ARG;
    return hip_status(launch_stale_k(gen_sum, gen_count, completion, current_version, n_traj, k, keep_out, lag_out,
                                     (hipStream_t)stream));
}

int pace_diagnostics(const double *score, const int64_t *gen_sum, const int64_t *gen_count,
                     const int32_t *completion, int32_t current_version, const uint8_t *keep, int64_t n_traj,
                     const double *edges, int nbins, int64_t *hist_out, int64_t *totals_out, void *stream) {
    const TimerScope timers;
    if (n_traj < 0 || n_traj >= INT32_MAX || nbins < 1 || nbins > kDiagBinsMax || current_version < 0)
        return PACE_ERR_INVALID_ARG;
    if (!edges || !hist_out || !totals_out) return PACE_ERR_INVALID_ARG;
    if (n_traj > 0 && (!score || !gen_sum || !gen_count || !completion || !keep)) return PACE_ERR_INVALID_ARG;
    if (!aligned(score, 8) || !aligned(gen_sum, 8) || !aligned(gen_count, 8) || !aligned(completion, 4) ||
        !aligned(edges, 8) || !aligned(hist_out, 8) || !aligned(totals_out, 8))
        return PACE_ERR_INVALID_ARG;
    return hip_status(launch_diagnostics(score, gen_sum, gen_count, completion, current_version, keep, n_traj,
                                         edges, nbins, hist_out, totals_out, (hipStream_t)stream));
}

static_assert(PACE_PHASE_COUNT == kPhaseCount, "phase count");

int pace_time_next_kernel(int phase, void *start_event, void *stop_event) {
    if (phase < 0 || phase >= PACE_PHASE_COUNT) return PACE_ERR_INVALID_ARG;
    if ((start_event == nullptr) != (stop_event == nullptr)) return PACE_ERR_INVALID_ARG;
    g_phase_timer[phase][0] = (hipEvent_t)start_event;
    g_phase_timer[phase][1] = (hipEvent_t)stop_event;
    return PACE_OK;
}

int pace_validate(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                  const int32_t *completion, int32_t current_version, const double *window_sorted,
                  int64_t window_n, int32_t *err_word_out, void *stream) {
    const TimerScope timers;
    if (n_traj < 0 || n_traj >= INT32_MAX || n_tokens < 0 || window_n < 0) return PACE_ERR_INVALID_ARG;
    if (!offsets || !err_word_out || (n_traj > 0 && !completion) || (n_tokens > 0 && !tags) ||
        (window_n > 0 && !window_sorted))
        return PACE_ERR_INVALID_ARG;
    if (!aligned(tags, 4) || !aligned(offsets, 8) || !aligned(completion, 4) ||
        !aligned(err_word_out, 4) || !aligned(window_sorted, 8))
        return PACE_ERR_INVALID_ARG;
    return hip_status(launch_validate(tags, offsets, n_traj, n_tokens, completion, current_version,
                                      window_sorted, window_n, err_word_out, (hipStream_t)stream));
}

}  // extern "C"
