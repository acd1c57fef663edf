/*
 * PACE filter step -- CPU ORACLE (test infrastructure only).
 *
 * A plain, slow, single-threaded reference of what the filter step computes,
 * written from the paper's definitions. Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg load it. It shares no source, header,
 * table or helper with the GPU library, and the GPU library never calls it.
 *
 * Every floating-point expression is evaluated in IEEE binary64 with
 * round-to-nearest, one operation at a time (built with -ffp-contract=off and
 * without fast-math), in the order written here.
 *
 * Readings of the paper that this file adopts (where it is silent):
 *   - a token tagged -1 is non-generated (tool output): it is not one of the
 *     T response tokens of Eq. (1), so it is excluded from T and from the
 *     staleness sums, but it stays in the trajectory's span when compacted;
 *   - T = 0 gives Generation Staleness 0;
 *   - the empirical CDF of Eq. (8) counts window entries <= s;
 *   - gamma is an integer in [1,4], so phi_gamma(a/W) is evaluated exactly
 *     as a^g / (a^g + (W-a)^g) and rounded once;
 *   - a missing prefix score (NaN), no window, or fewer than window_min
 *     observations gives F = 1 (the full Generation Staleness penalty);
 *   - the rejection budget is an integer count: rint(min(r_hat, r_max) * N),
 *     forced to 0 when N <= N^tar and capped at the surplus N - N^tar;
 *   - the quantile rule "reject M > kappa" is taken over the current pool
 *     with exactly `budget` rejections; equal scores reject the lower
 *     trajectory id first.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_ERR_ARG (-1)
#define ORC_ERR_PRECONDITION (-3)

/* ------------------------------------------------------------------------
 * Preconditions of Lemma 1: every generated token's version v_t satisfies
 * v_t <= c(tau) <= j (Sec. 2, Lemma 1 and its proof in App. A), versions are
 * non-negative indices, and the CSR offsets describe the token array.
 * ---------------------------------------------------------------------- */
int oracle_validate(const int32_t *tags, const int64_t *offsets, int64_t n,
                    int64_t n_tokens, const int32_t *completion, int32_t V)
{
    if (n < 0 || n_tokens < 0 || !offsets || (n > 0 && !completion) ||
        (n_tokens > 0 && !tags))
        return ORC_ERR_ARG;
    if (offsets[0] != 0 || offsets[n] != n_tokens)
        return ORC_ERR_PRECONDITION;
    for (int64_t i = 0; i < n; i++) {
        if (offsets[i + 1] < offsets[i])
            return ORC_ERR_PRECONDITION;
        int32_t c = completion[i];
        if (c < 0 || c > V)
            return ORC_ERR_PRECONDITION;
        for (int64_t t = offsets[i]; t < offsets[i + 1]; t++) {
            int32_t v = tags[t];
            if (v == -1)
                continue;
            if (v < 0 || v > c)
                return ORC_ERR_PRECONDITION;
        }
    }
    return ORC_OK;
}

/* Integer power for the exact form of phi_gamma (callers keep x^g < 2^53). */
static int64_t ipow(int64_t x, int g)
{
    int64_t r = 1;
    for (int k = 0; k < g; k++)
        r *= x;
    return r;
}

/* 1 when W^g < 2^53, so that every a^g and (W-a)^g with 0 <= a <= W, and
 * their sum W^g at most, is an exact integer in a double; 0 otherwise. Each
 * factor is tested against the bound before it is multiplied in, so no
 * intermediate product can overflow. */
static int window_power_fits(int64_t W, int g)
{
    const int64_t limit = ((int64_t)1 << 53) - 1;
    int64_t r = 1;
    for (int k = 0; k < g; k++) {
        if (W != 0 && r > limit / W)
            return 0;
        r *= W;
    }
    return 1;
}

/* ------------------------------------------------------------------------
 * Scores, Sec. 2 and Sec. 3.2.
 *
 * For trajectory i with completion version c_i, consumed at version j = V:
 *   T_i       = number of generated (tag != -1) tokens          (Eq. (1))
 *   S_i       = sum over those tokens of (c_i - v_t)            (Eq. (2))
 *   K_gen     = S_i / T_i   (0 when T_i = 0)                     (Eq. (2))
 *   K_wait    = V - c_i                                          (Eq. (2))
 *   q         = #{w in window : w <= s_pre} / W                  (Eq. (8))
 *   F         = phi_gamma(q) = q^g / (q^g + (1-q)^g)             (Eq. (9))
 *   M         = w_wait * K_wait + F * K_gen                     (Eq. (6),(7))
 * With prefix == NULL the weight is F = 1: PACE (Raw Staleness), whose score
 * equals the trajectory lag of Eq. (1). With w_wait = 0 it is the
 * generation-only variant (Sec. 3.2, "Other Variants").
 * ---------------------------------------------------------------------- */
int oracle_score(const int32_t *tags, const int64_t *offsets, int64_t n,
                 int64_t n_tokens, const int32_t *completion, int32_t V,
                 const double *prefix, const double *window, int64_t W,
                 double w_wait, int32_t gamma, int64_t window_min,
                 double *score_out, int64_t *S_out, int64_t *T_out)
{
    if (!score_out || gamma < 1 || gamma > 4 || window_min < 0 || W < 0 ||
        !(w_wait >= 0.0) || isinf(w_wait) || (W > 0 && !window))
        return ORC_ERR_ARG;
    /* the exact form needs W^gamma representable in a double */
    if (W > 0 && !window_power_fits(W, gamma))
        return ORC_ERR_ARG;
    int rc = oracle_validate(tags, offsets, n, n_tokens, completion, V);
    if (rc != ORC_OK)
        return rc;
    for (int64_t k = 1; k < W; k++)
        if (!(window[k - 1] <= window[k]))
            return ORC_ERR_PRECONDITION;   /* window must be sorted, no NaN */
    if (W > 0 && isnan(window[0]))
        return ORC_ERR_PRECONDITION;

    for (int64_t i = 0; i < n; i++) {
        int64_t c = completion[i];
        int64_t T = 0, S = 0;
        for (int64_t t = offsets[i]; t < offsets[i + 1]; t++) {
            int32_t v = tags[t];
            if (v == -1)
                continue;            /* non-generated token */
            T += 1;
            S += c - (int64_t)v;
        }
        double K_wait = (double)((int64_t)V - c);
        double K_gen = (T > 0) ? (double)S / (double)T : 0.0;

        double F = 1.0;
        if (prefix && W > 0 && W >= window_min && !isnan(prefix[i])) {
            int64_t a = 0;
            for (int64_t k = 0; k < W; k++)
                if (window[k] <= prefix[i])
                    a += 1;
            int64_t A = ipow(a, gamma);
            int64_t B = ipow(W - a, gamma);
            F = (double)A / (double)(A + B);
        }
        double wait_term = w_wait * K_wait;
        double gen_term = F * K_gen;
        score_out[i] = wait_term + gen_term;
        if (S_out)
            S_out[i] = S;
        if (T_out)
            T_out[i] = T;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Rejection budget, Sec. 3.1.
 *   r_j    = clip((N - N^tar) / max(N, 1), 0, 1)                 (Eq. (3))
 *   r_hat  = beta * r_hat_prev + (1 - beta) * r_j                (Eq. (4))
 *   budget = 0 if N <= N^tar, else
 *            min(rint(min(r_hat, r_max) * N), N - N^tar)
 * r_max is the maximum rejection budget of App. B (0.9 there).
 * ---------------------------------------------------------------------- */
int oracle_budget(int64_t N, int64_t N_tar, double beta, double r_max,
                  double *r_hat_inout, int64_t *budget_out)
{
    if (!r_hat_inout || !budget_out || N < 0 || N_tar < 0 ||
        !(beta >= 0.0 && beta < 1.0) || !(r_max >= 0.0 && r_max <= 1.0) ||
        !(*r_hat_inout >= 0.0) || isinf(*r_hat_inout))
        return ORC_ERR_ARG;
    double denom = (double)(N > 1 ? N : 1);
    double x = (double)(N - N_tar) / denom;
    double r = x < 0.0 ? 0.0 : (x > 1.0 ? 1.0 : x);
    double r_hat = beta * (*r_hat_inout) + (1.0 - beta) * r;
    int64_t b = 0;
    if (N > N_tar) {
        double rc = r_hat < r_max ? r_hat : r_max;
        b = (int64_t)nearbyint(rc * (double)N);   /* default mode: ties to even */
        if (b > N - N_tar)
            b = N - N_tar;
        if (b < 0)
            b = 0;
    }
    *r_hat_inout = r_hat;
    *budget_out = b;
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Selection, Sec. 3.1 and Algorithm 1 (trainer side): the trajectories with
 * the highest scores are rejected. Here exactly `budget` of them: sort all
 * ids by (score descending, id ascending) and reject the first `budget`.
 * ---------------------------------------------------------------------- */
static const double *g_sort_scores;   /* comparator context (single thread) */

static int by_score_desc_id_asc(const void *pa, const void *pb)
{
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    double sa = g_sort_scores[a], sb = g_sort_scores[b];
    if (sa > sb)
        return -1;
    if (sa < sb)
        return 1;
    return (a < b) ? -1 : (a > b);
}

int oracle_select(const double *score, int64_t n, int64_t budget,
                  uint8_t *keep_out, int32_t *reject_ids_out)
{
    if (n < 0 || n > INT32_MAX || budget < 0 || budget > n ||
        (n > 0 && (!score || !keep_out)) || (budget > 0 && !reject_ids_out))
        return ORC_ERR_ARG;
    for (int64_t i = 0; i < n; i++)
        if (isnan(score[i]))
            return ORC_ERR_PRECONDITION;
    int32_t *order = (int32_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    if (!order)
        return ORC_ERR_ARG;
    for (int64_t i = 0; i < n; i++)
        order[i] = (int32_t)i;
    g_sort_scores = score;
    qsort(order, (size_t)n, sizeof(int32_t), by_score_desc_id_asc);
    for (int64_t i = 0; i < n; i++)
        keep_out[i] = 1;
    for (int64_t r = 0; r < budget; r++)
        keep_out[order[r]] = 0;
    int64_t k = 0;
    for (int64_t i = 0; i < n; i++)
        if (!keep_out[i])
            reject_ids_out[k++] = (int32_t)i;
    free(order);
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Compaction: the survivors form the training batch (Sec. 3.1, Algorithm 1).
 * Kept trajectories stay in pool order; each payload column's kept spans are
 * concatenated (non-generated tokens included, they stay in context).
 * ---------------------------------------------------------------------- */
int oracle_compact(const int64_t *offsets, int64_t n, int64_t n_tokens,
                   const uint8_t *keep, int n_cols,
                   const void *const *cols_in, const int32_t *elem_bytes,
                   void *const *cols_out, int64_t *offsets_out,
                   int32_t *kept_ids_out, int64_t *n_kept_tokens_out)
{
    if (n < 0 || n > INT32_MAX || !offsets || !offsets_out || !n_kept_tokens_out ||
        n_cols < 0 || (n > 0 && (!keep || !kept_ids_out)) ||
        (n_cols > 0 && (!cols_in || !cols_out || !elem_bytes)))
        return ORC_ERR_ARG;
    for (int c = 0; c < n_cols; c++) {
        int32_t e = elem_bytes[c];
        if (!(e == 1 || e == 2 || e == 4 || e == 8) || (n_tokens > 0 && (!cols_in[c] || !cols_out[c])))
            return ORC_ERR_ARG;
    }
    if (offsets[0] != 0 || offsets[n] != n_tokens)
        return ORC_ERR_PRECONDITION;
    for (int64_t i = 0; i < n; i++)
        if (offsets[i + 1] < offsets[i])
            return ORC_ERR_PRECONDITION;

    int64_t pos = 0, k = 0;
    for (int64_t i = 0; i < n; i++) {
        if (!keep[i])
            continue;
        int64_t len = offsets[i + 1] - offsets[i];
        offsets_out[k] = pos;
        kept_ids_out[k] = (int32_t)i;
        for (int c = 0; c < n_cols; c++) {
            size_t e = (size_t)elem_bytes[c];
            memcpy((char *)cols_out[c] + (size_t)pos * e,
                   (const char *)cols_in[c] + (size_t)offsets[i] * e, (size_t)len * e);
        }
        pos += len;
        k += 1;
    }
    offsets_out[k] = pos;
    *n_kept_tokens_out = pos;
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Group-level admission (Appendix B: the full method aggregates by the mean
 * within prompt groups; the score window and the diagnostics count groups).
 * Consecutive trajectories form prompt groups: group g holds trajectories
 * [group_offsets[g], group_offsets[g+1]). A group's score is the mean of its
 * members' scores -- summed in member order, then divided by the member
 * count -- and an empty group scores 0. Groups are then budgeted, selected
 * and compacted as whole units: the budget counts groups, and a rejected
 * group drops all of its members.
 * ---------------------------------------------------------------------- */
static int check_groups(const int64_t *group_offsets, int64_t n_groups, int64_t n)
{
    if (group_offsets[0] != 0 || group_offsets[n_groups] != n)
        return ORC_ERR_PRECONDITION;
    for (int64_t g = 0; g < n_groups; g++)
        if (group_offsets[g + 1] < group_offsets[g])
            return ORC_ERR_PRECONDITION;
    return ORC_OK;
}

int oracle_group_score(const double *score, int64_t n, const int64_t *group_offsets,
                       int64_t n_groups, double *group_score_out)
{
    if (n < 0 || n_groups < 0 || !group_offsets || (n > 0 && !score) ||
        (n_groups > 0 && !group_score_out))
        return ORC_ERR_ARG;
    int rc = check_groups(group_offsets, n_groups, n);
    if (rc != ORC_OK)
        return rc;
    for (int64_t g = 0; g < n_groups; g++) {
        int64_t lo = group_offsets[g], hi = group_offsets[g + 1];
        double sum = 0.0;
        for (int64_t i = lo; i < hi; i++)
            sum = sum + score[i];
        group_score_out[g] = (hi > lo) ? sum / (double)(hi - lo) : 0.0;
    }
    return ORC_OK;
}

/* Trajectory keep flags from group keep flags: every member shares its
 * group's fate. */
int oracle_group_expand(const int64_t *group_offsets, int64_t n_groups, int64_t n,
                        const uint8_t *group_keep, uint8_t *keep_out)
{
    if (n < 0 || n_groups < 0 || !group_offsets || (n_groups > 0 && !group_keep) ||
        (n > 0 && !keep_out))
        return ORC_ERR_ARG;
    int rc = check_groups(group_offsets, n_groups, n);
    if (rc != ORC_OK)
        return rc;
    for (int64_t g = 0; g < n_groups; g++)
        for (int64_t i = group_offsets[g]; i < group_offsets[g + 1]; i++)
            keep_out[i] = group_keep[g] ? 1 : 0;
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * The streaming admission rule (Sec. 3.1, Algorithm 1), literally: at step j
 * the cutoff kappa is the (1 - r_hat)-quantile of a sliding window of
 * recently observed scores; the trainer then draws candidates from the pool
 * in pool order, observes each one's score, rejects it when its score exceeds
 * kappa and retains it otherwise, until batch_size candidates are retained
 * or the pool is exhausted.
 *
 * Readings (the paper leaves these open):
 *   - kappa is fixed for the whole step, from the window as it stood before
 *     the draw; every drawn candidate's score then enters the window, in draw
 *     order, after the draw;
 *   - the quantile is the lower empirical one: the ceil(p * cnt)-th smallest
 *     of the cnt window entries, p = 1 - min(r_hat, r_max);
 *   - with fewer than window_min entries, or a rate of 0, nothing is
 *     rejected (kappa = +inf);
 *   - the window is a ring of window_cap entries: once full, each new score
 *     replaces the oldest.
 * status_out[i]: 0 drawn and rejected, 1 drawn and retained, 2 not drawn.
 * ---------------------------------------------------------------------- */
static int cmp_double_asc(const void *pa, const void *pb)
{
    double x = *(const double *)pa, y = *(const double *)pb;
    if (x < y)
        return -1;
    return x > y ? 1 : 0;
}

int oracle_stream_admit(const double *score, int64_t n, double r_hat, double r_max,
                        int64_t window_min, int64_t batch_size, double *ring, int64_t cap,
                        int64_t *head_inout, int64_t *count_inout, uint8_t *status_out,
                        double *kappa_out, int64_t *n_drawn_out, int64_t *n_retained_out)
{
    if (n < 0 || cap < 1 || batch_size < 0 || window_min < 0 || !ring || !head_inout ||
        !count_inout || !kappa_out || !n_drawn_out || !n_retained_out ||
        (n > 0 && (!score || !status_out)))
        return ORC_ERR_ARG;
    int64_t head = *head_inout, cnt = *count_inout;
    if (head < 0 || head >= cap || cnt < 0 || cnt > cap || !(r_hat >= 0.0) || !(r_max >= 0.0))
        return ORC_ERR_ARG;

    /* the cutoff, from the window before this step's draw */
    double rate = r_hat < r_max ? r_hat : r_max;
    double kappa = INFINITY;
    if (cnt >= window_min && cnt > 0 && rate > 0.0) {
        double *sorted = (double *)malloc((size_t)cnt * sizeof(double));
        if (!sorted)
            return ORC_ERR_ARG;
        /* the cnt most recent entries end just before head */
        for (int64_t t = 0; t < cnt; t++)
            sorted[t] = ring[(head - cnt + t + cap) % cap];
        qsort(sorted, (size_t)cnt, sizeof(double), cmp_double_asc);
        double p = 1.0 - rate;
        int64_t k = (int64_t)ceil(p * (double)cnt);   /* 1-based rank */
        if (k < 1)
            k = 1;
        kappa = sorted[k - 1];
        free(sorted);
    }

    /* the draw */
    int64_t drawn = 0, retained = 0;
    for (int64_t i = 0; i < n; i++)
        status_out[i] = 2;
    for (int64_t i = 0; i < n && retained < batch_size; i++) {
        drawn += 1;
        if (score[i] > kappa) {
            status_out[i] = 0;
        } else {
            status_out[i] = 1;
            retained += 1;
        }
    }

    /* the window takes every drawn score, oldest first */
    for (int64_t i = 0; i < drawn; i++) {
        ring[head] = score[i];
        head = (head + 1) % cap;
        if (cnt < cap)
            cnt += 1;
    }
    *head_inout = head;
    *count_inout = cnt;
    *kappa_out = kappa;
    *n_drawn_out = drawn;
    *n_retained_out = retained;
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Prefix Forgetting Score (Eq. (5), Sec. 3.2; collection rules in
 * Appendix B): the mean absolute difference between the rescoring policy's
 * log-probabilities and the behaviour log-probabilities recorded during
 * generation, over the rescored prefix's response tokens.
 * Prefix i holds tokens [prefix_offsets[i], prefix_offsets[i+1]) of the
 * packed arrays. Readings: a token tagged -1 (non-generated, tool output) is
 * not eligible; only the first `cap` eligible tokens count (the scoring cap);
 * a prefix with fewer than `min_tokens` eligible tokens gets no score (NaN);
 * each term is |(double)lp_new - (double)lp_behavior| and the terms are
 * added in token order in binary64, then divided once by their count.
 * tags may be NULL (every token eligible).
 * ---------------------------------------------------------------------- */
int oracle_prefix_score(const float *lp_new, const float *lp_behavior, const int32_t *tags,
                        const int64_t *prefix_offsets, int64_t n, int64_t n_tokens, int64_t cap,
                        int64_t min_tokens, double *s_pre_out)
{
    if (n < 0 || n_tokens < 0 || cap < 0 || min_tokens < 0 || !prefix_offsets ||
        (n > 0 && !s_pre_out) || (n_tokens > 0 && (!lp_new || !lp_behavior)))
        return ORC_ERR_ARG;
    if (prefix_offsets[0] != 0 || prefix_offsets[n] != n_tokens)
        return ORC_ERR_PRECONDITION;
    for (int64_t i = 0; i < n; i++)
        if (prefix_offsets[i + 1] < prefix_offsets[i])
            return ORC_ERR_PRECONDITION;
    for (int64_t i = 0; i < n; i++) {
        double sum = 0.0;
        int64_t m = 0;
        for (int64_t t = prefix_offsets[i]; t < prefix_offsets[i + 1]; t++) {
            if (tags && tags[t] == -1)
                continue;                /* non-generated token */
            if (m == cap)
                break;
            double d = (double)lp_new[t] - (double)lp_behavior[t];
            sum = sum + fabs(d);
            m += 1;
        }
        s_pre_out[i] = (m >= min_tokens && m > 0) ? sum / (double)m : NAN;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Stale-k admission (Sec. 2, the controlled Stale-k setting): only
 * trajectories whose policy lag, Eq. (1) -- the mean over response tokens of
 * j - v_t -- is at most k are admitted. Computed from the tags as written:
 * the integer sum of (j - v_t) over the response tokens against k T, so the
 * comparison is exact. Reading: a trajectory without response tokens
 * (T = 0) has no Generation Staleness and its lag is taken as j - c.
 * lag_out (may be NULL) receives the lag as a double (sum / T, or j - c).
 * ---------------------------------------------------------------------- */
int oracle_stale_k(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                   const int32_t *completion, int32_t V, int64_t k, uint8_t *keep_out, double *lag_out)
{
    if (n < 0 || n_tokens < 0 || !offsets || (n > 0 && (!completion || !keep_out)) ||
        (n_tokens > 0 && !tags))
        return ORC_ERR_ARG;
    int rc = oracle_validate(tags, offsets, n, n_tokens, completion, V);
    if (rc != ORC_OK)
        return rc;
    for (int64_t i = 0; i < n; i++) {
        int64_t lag_sum = 0, T = 0;
        for (int64_t t = offsets[i]; t < offsets[i + 1]; t++) {
            if (tags[t] == -1)
                continue;
            lag_sum += (int64_t)V - (int64_t)tags[t];
            T += 1;
        }
        int64_t wait = (int64_t)V - (int64_t)completion[i];
        if (T > 0) {
            keep_out[i] = (lag_sum <= k * T) ? 1 : 0;
            if (lag_out)
                lag_out[i] = (double)lag_sum / (double)T;
        } else {
            keep_out[i] = (wait <= k) ? 1 : 0;
            if (lag_out)
                lag_out[i] = (double)wait;
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Admission diagnostics (Sec. 4, the staleness distribution diagnostics):
 * histograms of Waiting, Generation and Effective Staleness over the
 * candidates, split into retained and rejected, plus exact integer totals.
 * Metric m of candidate i: K_wait = V - c, K_gen = S / T (0 when T = 0), and
 * K_eff = score[i] (the admission score). Bin b of metric m holds values in
 * [edges[m][b], edges[m][b+1]); values below edges[m][0] go to an underflow
 * bin and values at or above edges[m][nbins] to an overflow bin.
 * hist_out: int64 [3][2][nbins + 2], [metric][0 rejected, 1 retained][bin],
 *   bin 0 = underflow, 1..nbins, nbins + 1 = overflow.
 * totals_out: int64 [2][4], per class: count, sum of (V - c), sum S, sum T.
 * ---------------------------------------------------------------------- */
int oracle_diagnostics(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                       const int32_t *completion, int32_t V, const double *score, const uint8_t *keep,
                       const double *edges, int64_t nbins, int64_t *hist_out, int64_t *totals_out)
{
    if (n < 0 || nbins < 1 || !offsets || !edges || !hist_out || !totals_out ||
        (n > 0 && (!completion || !score || !keep)) || (n_tokens > 0 && !tags))
        return ORC_ERR_ARG;
    int rc = oracle_validate(tags, offsets, n, n_tokens, completion, V);
    if (rc != ORC_OK)
        return rc;
    int64_t nb2 = nbins + 2;
    memset(hist_out, 0, (size_t)(3 * 2 * nb2) * sizeof(int64_t));
    memset(totals_out, 0, 8 * sizeof(int64_t));
    for (int64_t i = 0; i < n; i++) {
        int64_t c = completion[i], S = 0, T = 0;
        for (int64_t t = offsets[i]; t < offsets[i + 1]; t++) {
            if (tags[t] == -1)
                continue;
            S += c - (int64_t)tags[t];
            T += 1;
        }
        double m[3];
        m[0] = (double)((int64_t)V - c);
        m[1] = (T > 0) ? (double)S / (double)T : 0.0;
        m[2] = score[i];
        int cls = keep[i] ? 1 : 0;
        for (int q = 0; q < 3; q++) {
            const double *e = edges + q * (nbins + 1);
            int64_t bin;
            if (!(m[q] >= e[0]))
                bin = 0;
            else if (m[q] >= e[nbins])
                bin = nbins + 1;
            else {
                bin = 1;
                while (!(m[q] < e[bin]))
                    bin += 1;
            }
            hist_out[(q * 2 + cls) * nb2 + bin] += 1;
        }
        int64_t *tot = totals_out + cls * 4;
        tot[0] += 1;
        tot[1] += (int64_t)V - c;
        tot[2] += S;
        tot[3] += T;
    }
    return ORC_OK;
}
