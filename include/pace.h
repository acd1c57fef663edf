/*
 * pace.h -- C ABI of the PACE pool filter step on AMD Instinct MI355X (gfx950).
 *
 * PACE (Pool-Aware Control of Effective Staleness) filters the pool of
 * completed asynchronous-RL trajectories before each trainer step:
 *
 *   pace_score    per-trajectory staleness score              Eq. (1),(2),(6)-(9)
 *   pace_budget   occupancy-driven rejection budget            Eq. (3),(4)
 *   pace_select   reject exactly `budget` highest scores       Sec. 3.1, Algorithm 1
 *   pace_compact  pack the survivors' token spans              Algorithm 1 (batch B_j)
 *   pace_validate check the data preconditions of Lemma 1     Sec. 2, Lemma 1
 *   pace_filter_step  all four steps above in one call        Algorithm 1
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pool layout (CSR over tokens): trajectory i owns tokens
 *   [offsets[i], offsets[i+1]) of every per-token column. offsets has n_traj+1
 *   int64 entries, offsets[0] = 0, non-decreasing, offsets[n_traj] = n_tokens.
 * - Per-token version tags (int32): the behavior policy version v_t that
 *   generated the token; -1 marks a non-generated token (tool output in a
 *   multi-turn rollout). Masked tokens are not response tokens of Eq. (1): they
 *   count neither in T nor in the staleness sums, but compaction copies them.
 * - Pointers are DEVICE pointers unless marked [host]. Every device call is
 *   enqueued on `stream` (a hipStream_t passed as void*, NULL = null stream)
 *   and returns without synchronising. Nothing is allocated or freed inside a
 *   call; the caller owns every buffer, including the workspace, and no
 *   pointer is retained after a call returns. Inputs and outputs must not
 *   overlap.
 * - Argument errors the host can see (null required pointers, negative or
 *   oversized counts, bad parameters, misaligned or short workspace) return
 *   an error code before anything is enqueued and nothing is written.
 * - Data preconditions (monotone offsets, -1 <= tag <= c_i, 0 <= c_i <= V,
 *   sorted window) are NOT checked by the fast path: violating them gives
 *   unspecified (but memory-safe, in-bounds) results. pace_validate checks
 *   them on the device.
 * - A failed kernel launch returns PACE_ERR_HIP.
 * - Every result is a deterministic function of the inputs: identical bits
 *   run to run and for any stream.
 * - No call keeps state from one call to the next, apart from the per-thread
 *   timers that the measurement hook pace_time_next_kernel arms for the
 *   following device call only.
 * - Workspace: at least pace_workspace_bytes() bytes, 256-byte aligned. Its
 *   contents need no initialisation and are scratch between calls; calls
 *   sharing one workspace must be ordered (same stream).
 */
#ifndef PACE_H
#define PACE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PACE_OK 0
#define PACE_ERR_INVALID_ARG (-1)
#define PACE_ERR_WORKSPACE (-2)
#define PACE_ERR_PRECONDITION (-3)
#define PACE_ERR_HIP (-4)
#define PACE_ERR_SCRATCH_LIMIT (-5) /* pace_filter_step_noalloc: pool beyond the fixed scratch */

/* Bits of the device error word written by pace_validate. */
#define PACE_BAD_OFFSETS 0x1    /* offsets[0] != 0, decreasing, or offsets[n] != n_tokens */
#define PACE_BAD_COMPLETION 0x2 /* some c_i < 0 or c_i > current_version */
#define PACE_BAD_TAG 0x4        /* some tag < -1, or tag > c_i of its trajectory */
#define PACE_BAD_WINDOW 0x8     /* prefix window not ascending, or holds NaN */
#define PACE_BAD_GROUPS 0x10    /* group offsets not 0 .. n_traj non-decreasing (pace_validate_groups) */

/* Controller parameters (host struct).
 *   w_wait     w_1 of Eq. (6): 1 for Effective and Raw Staleness, 0 for the
 *              generation-only variant (Sec. 3.2). Finite, >= 0.
 *   gamma      sharpening exponent of Eq. (9); integer in [1,4] (4 by default,
 *              App. B). window_n^gamma must stay below 2^53.
 *   window_min minimum number of prefix-window observations before the
 *              prefix weight applies (32, App. B); below it F = 1. >= 0.
 *   beta       EMA coefficient of Eq. (4), in [0,1) (0 by default).
 *   r_max      maximum rejection budget, in [0,1] (0.9, App. B). */
typedef struct pace_params {
    double w_wait;
    int32_t gamma;
    int32_t window_min;
    double beta;
    double r_max;
} pace_params;

/* Fills *p with the defaults above (w_wait 1, gamma 4, window_min 32, beta 0,
 * r_max 0.9). */
void pace_default_params(pace_params *p);

/* Workspace sizes. `which` selects the call: */
#define PACE_WS_SCORE 0
#define PACE_WS_SELECT 1
#define PACE_WS_COMPACT 2
#define PACE_WS_FILTER_STEP 3
/* Writes to *bytes_out [host] the workspace that call needs for a pool of
 * n_traj trajectories and n_tokens tokens. Returns PACE_ERR_INVALID_ARG for
 * negative sizes or an unknown `which`. */
int pace_workspace_bytes(int which, int64_t n_traj, int64_t n_tokens, size_t *bytes_out);

/* pace_score -- per-trajectory effective-staleness score (Sec. 2, Sec. 3.2).
 *
 * For trajectory i with completion version c_i = completion[i], consumed at
 * the current version j = current_version:
 *   T_i    = number of tokens with tag != -1                   (Eq. (1))
 *   S_i    = sum over those tokens of (c_i - tag)             (Eq. (2), K_gen = S_i/T_i)
 *   K_wait = j - c_i                                           (Eq. (2))
 *   F_i    = phi_gamma(q_i), q_i = #{w in window : w <= s_i} / W  (Eq. (8),(9))
 *   M_i    = w_wait * K_wait + F_i * K_gen                     (Eq. (6),(7))
 * evaluated as K_gen = (double)S_i / (double)T_i (0 when T_i = 0),
 * F_i = (double)a^g / (double)(a^g + (W-a)^g), and
 * M_i = (w_wait*K_wait) + (F_i*K_gen), each operation an IEEE binary64
 * round-to-nearest step, never fused.
 * F_i = 1 (PACE Raw Staleness) when prefix_score is NULL, when prefix_score[i]
 * is NaN (no prefix score: the rollout was never interrupted), or when
 * window_n < max(params->window_min, 1).
 *
 * tags          int32 [n_tokens], 16-byte aligned for the vector path
 * offsets       int64 [n_traj+1]
 * completion    int32 [n_traj]
 * current_version  j; must be < 2^31 - 1
 * prefix_score  double [n_traj] or NULL
 * window_sorted double [window_n], ascending, or NULL when window_n = 0
 * params        [host] controller parameters (NULL = defaults)
 * score_out     double [n_traj]  (required)
 * gen_sum_out   int64 [n_traj]   S_i, or NULL
 * gen_count_out int64 [n_traj]   T_i, or NULL
 * A single trajectory may hold at most 2^32 - 1 tokens. */
int pace_score(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
               const int32_t *completion, int32_t current_version,
               const double *prefix_score, const double *window_sorted, int64_t window_n,
               const pace_params *params, double *score_out, int64_t *gen_sum_out,
               int64_t *gen_count_out, void *workspace, size_t workspace_bytes, void *stream);

/* pace_budget -- rejection budget from pool occupancy (Sec. 3.1). Host only.
 *   r_j    = clip((N - N^tar) / max(N,1), 0, 1)                Eq. (3)
 *   r_hat  = beta * r_hat_prev + (1 - beta) * r_j              Eq. (4)
 *   budget = 0 if N <= N^tar, else min(rint(min(r_hat, r_max) * N), N - N^tar)
 * (rint rounds half to even). occupancy N >= 0, capacity N^tar >= 0.
 * r_hat_inout [host] holds r_hat_{j-1} on entry (finite, >= 0; 0 at the first
 * step) and r_hat_j on return. budget_out [host]. */
int pace_budget(int64_t occupancy, int64_t capacity, const pace_params *params,
                double *r_hat_inout, int64_t *budget_out);

/* pace_select -- reject exactly `budget` trajectories (Sec. 3.1, Algorithm 1).
 * The rejected set is the first `budget` ids in the order (score descending,
 * id ascending): trajectories with higher scores go first and equal scores
 * reject the lower id first. -0.0 and +0.0 are equal. NaN scores violate the
 * precondition (pace_score never produces them); they order above +inf.
 * score          double [n_traj]
 * budget         0 <= budget <= n_traj (n_traj < 2^31)
 * keep_out       uint8 [n_traj]: 1 = kept, 0 = rejected
 * reject_ids_out int32 [budget]: rejected ids, ascending (may be NULL when
 *                budget = 0) */
int pace_select(const double *score, int64_t n_traj, int64_t budget, uint8_t *keep_out,
                int32_t *reject_ids_out, void *workspace, size_t workspace_bytes, void *stream);

/* pace_compact -- pack the kept trajectories into the training batch
 * (Algorithm 1). Kept trajectories stay in pool order; for every payload
 * column the kept spans are concatenated (masked tokens included).
 * offsets           int64 [n_traj+1]
 * keep              uint8 [n_traj] (nonzero = kept)
 * n_cols            0..8 payload columns, each n_tokens elements of
 *                   elem_bytes[c] in {1,2,4,8} bytes
 * cols_in, cols_out [host] arrays of n_cols device pointers; each output
 *                   column must hold n_tokens elements (the upper bound, so no
 *                   host sync is needed to size it). 16-byte aligned columns
 *                   take the vector path.
 * elem_bytes        [host] int32 [n_cols]
 * offsets_out       int64 [n_traj+1]: entries 0..n_kept hold the packed CSR
 * kept_ids_out      int32 [n_traj]:   entries 0..n_kept-1 hold the kept ids
 * n_kept_tokens_out int64 [1] device scalar: offsets_out[n_kept] */
int pace_compact(const int64_t *offsets, int64_t n_traj, int64_t n_tokens, const uint8_t *keep,
                 int n_cols, const void *const *cols_in, const int32_t *elem_bytes,
                 void *const *cols_out, int64_t *offsets_out, int32_t *kept_ids_out,
                 int64_t *n_kept_tokens_out, void *workspace, size_t workspace_bytes,
                 void *stream);

/* pace_validate -- device check of the data preconditions of Lemma 1
 * (v_t <= c(tau) <= j) and of the CSR layout. Writes the OR of the
 * PACE_BAD_* bits that apply to *err_word_out (int32 device scalar; 0 = all
 * preconditions hold). window_sorted may be NULL (window_n = 0). */
int pace_validate(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                  const int32_t *completion, int32_t current_version,
                  const double *window_sorted, int64_t window_n, int32_t *err_word_out,
                  void *stream);

/* pace_filter_step -- one whole trainer-side filter step (Algorithm 1):
 * pace_budget on the host, then pace_score, pace_select and pace_compact on
 * the device, with the same arguments and results as those four calls made
 * in sequence (every output is bit-identical to theirs). The device work is
 * four dependent launches instead of six: the rank kernel also writes the
 * per-block partials the compaction needs, and the compaction writes the
 * rejected ids. Pools of 8192 < n_traj <= 262144 select across the whole
 * device (a level-0 histogram, then a kernel that finds the cut and writes
 * the keep flags and partials: five launches); larger pools run the separate
 * calls' kernels.
 *
 * occupancy, capacity, r_hat_inout, budget_out: as pace_budget ([host]).
 * score_out, gen_sum_out, gen_count_out: as pace_score (gen_* may be NULL).
 * keep_out, reject_ids_out: as pace_select (reject_ids_out holds at least
 *   *budget_out entries; n_traj entries always suffice).
 * n_cols .. n_kept_tokens_out: as pace_compact.
 * workspace: pace_workspace_bytes(PACE_WS_FILTER_STEP, ...) bytes.
 * On an argument error nothing is enqueued and *r_hat_inout is unchanged. */
int pace_filter_step(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                     const int32_t *completion, int32_t current_version,
                     const double *prefix_score, const double *window_sorted, int64_t window_n,
                     int64_t occupancy, int64_t capacity, const pace_params *params,
                     double *r_hat_inout, int64_t *budget_out, double *score_out,
                     int64_t *gen_sum_out, int64_t *gen_count_out, uint8_t *keep_out,
                     int32_t *reject_ids_out, int n_cols, const void *const *cols_in,
                     const int32_t *elem_bytes, void *const *cols_out, int64_t *offsets_out,
                     int32_t *kept_ids_out, int64_t *n_kept_tokens_out, void *workspace,
                     size_t workspace_bytes, void *stream);

/* pace_filter_step_noalloc -- pace_filter_step for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same arguments, results and kernels,
 * with no workspace argument. The workspace is instead a fixed array of
 * PACE_NOALLOC_SCRATCH_BYTES bytes in device memory, one per device, which the
 * library holds from its load until the process ends; the call allocates and
 * frees nothing. The array of the device current on the calling thread is
 * used, so `stream` must belong to that device.
 * Limit: the pool's workspace, pace_workspace_bytes(PACE_WS_FILTER_STEP,
 * n_traj, n_tokens), must fit in the array (for example 4096 trajectories of
 * up to ~1.8e9 tokens, or 65536 trajectories of up to ~1.6e9 tokens); a larger
 * pool returns PACE_ERR_SCRATCH_LIMIT after the argument checks, before
 * anything is enqueued.
 * Every call on one device shares that device's array: calls that may overlap
 * on one device (different streams, or threads) race and must be ordered by
 * the caller. No call relies on what an earlier call left in the array. */
#define PACE_NOALLOC_SCRATCH_BYTES (16u << 20)
int pace_filter_step_noalloc(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                             const int32_t *completion, int32_t current_version,
                             const double *prefix_score, const double *window_sorted, int64_t window_n,
                             int64_t occupancy, int64_t capacity, const pace_params *params,
                             double *r_hat_inout, int64_t *budget_out, double *score_out,
                             int64_t *gen_sum_out, int64_t *gen_count_out, uint8_t *keep_out,
                             int32_t *reject_ids_out, int n_cols, const void *const *cols_in,
                             const int32_t *elem_bytes, void *const *cols_out, int64_t *offsets_out,
                             int32_t *kept_ids_out, int64_t *n_kept_tokens_out, void *stream);

/* ---- Group-level admission (Appendix B) ------------------------------------
 * The full method aggregates by the mean within prompt groups; its score
 * window and diagnostics count groups. Consecutive trajectories form prompt
 * groups: group g holds trajectories [group_offsets[g], group_offsets[g+1]).
 * group_offsets: int64 [n_groups + 1] device array, expected to start at 0,
 * never decrease and end at n_traj (pace_validate_groups checks this; the
 * other calls clamp every group offset to [0, n_traj], so malformed offsets
 * give unspecified results but no out-of-bounds access). */

/* pace_group_score -- the score of each group: the mean of its members'
 * scores, added in member order and divided once by the member count. An
 * empty group scores 0.
 * score: f64 [n_traj] (pace_score output); group_score_out: f64 [n_groups]. */
int pace_group_score(const double *score, int64_t n_traj, const int64_t *group_offsets, int64_t n_groups,
                     double *group_score_out, void *stream);

/* pace_group_expand -- trajectory keep flags from group keep flags: every
 * member of group g gets (group_keep[g] != 0). keep_out: u8 [n_traj]; with
 * well-formed group offsets every entry is written. */
int pace_group_expand(const int64_t *group_offsets, int64_t n_groups, int64_t n_traj,
                      const uint8_t *group_keep, uint8_t *keep_out, void *stream);

/* pace_validate_groups -- writes PACE_BAD_GROUPS to *err_word_out (int32
 * device scalar) when the group offsets are malformed, else 0. */
int pace_validate_groups(const int64_t *group_offsets, int64_t n_groups, int64_t n_traj,
                         int32_t *err_word_out, void *stream);

/* pace_group_filter_step -- one filter step with prompt groups as the
 * admission unit: pace_score, pace_group_score, pace_budget over groups
 * (occupancy and capacity count groups), pace_select over the group scores
 * (exactly *budget_out groups rejected, first in the order (group score desc,
 * group id asc)), pace_group_expand and pace_compact, with the results of
 * those calls made in sequence.
 * group_score_out: f64 [n_groups]; group_keep_out: u8 [n_groups];
 * reject_group_ids_out: int32, at least *budget_out entries (n_groups always
 * suffice), ascending; keep_out: u8 [n_traj] (the expanded flags).
 * Other arguments as pace_filter_step. workspace:
 * pace_workspace_bytes(PACE_WS_FILTER_STEP, max(n_traj, n_groups), n_tokens)
 * bytes. Argument errors (including a budget above n_groups) return before
 * anything is enqueued, with *r_hat_inout unchanged. */
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
                           void *workspace, size_t workspace_bytes, void *stream);

/* ---- The streaming admission rule (Sec. 3.1, Algorithm 1) ------------------
 * pace_stream_admit -- one step of the paper's rule as written: the cutoff
 * kappa is the (1 - rate)-quantile of a sliding window of recently observed
 * scores, rate = min(r_hat, params->r_max); candidates are drawn in pool order,
 * a candidate scoring above kappa is rejected, the others are retained, until
 * batch_size are retained or the pool is exhausted. The realised number of
 * rejections varies (pace_select instead rejects exactly a budget).
 * Readings: kappa is fixed for the step from the window as it stood before
 * the draw, and is the lower empirical quantile, the ceil(p * cnt)-th
 * smallest of the cnt window entries with p = 1 - rate evaluated in binary64;
 * with fewer than params->window_min entries, or rate 0, nothing is rejected
 * (kappa = +inf); every drawn candidate's score then enters the window, in
 * draw order, the oldest entries giving way once the window is full.
 *
 * score: f64 [n_traj] (pace_score output; must not hold NaN).
 * r_hat: [host] smoothed rejection rate (pace_budget's r_hat).
 * batch_size: candidates to retain (>= 0).
 * window_ring: f64 [window_cap] device ring of observed scores, and
 * window_state: int64 [2] device {head, count}: the next slot to write and the
 *   number of valid entries (the count entries before head, cyclically).
 *   A fresh window is {0, 0}. Both are updated in place. 1 <= window_cap <= 1024.
 * status_out: u8 [n_traj]: 0 drawn and rejected, 1 drawn and retained,
 *   2 not drawn (stays in the pool). keep_out: u8 [n_traj], 1 = retained
 *   (pass it to pace_compact to build the batch).
 * reject_ids_out: int32, the rejected ids ascending (n_traj entries suffice).
 * kappa_out: f64 device scalar. counts_out: int64 [3] device: drawn,
 *   retained, rejected.
 * Two kernels: the cutoff, over ceil(window_cap / 16) workgroups, writes
 * kappa_out, which the draw (one workgroup) then reads; no workspace. */
int pace_stream_admit(const double *score, int64_t n_traj, double r_hat, const pace_params *params,
                      int64_t batch_size, double *window_ring, int64_t window_cap, int64_t *window_state,
                      uint8_t *status_out, uint8_t *keep_out, int32_t *reject_ids_out, double *kappa_out,
                      int64_t *counts_out, void *stream);

/* pace_stream_step -- one whole trainer step under the streaming rule:
 * pace_budget on the host (r_hat carried in *r_hat_inout), then pace_score,
 * pace_stream_admit and pace_compact of the retained batch on the device,
 * with the results of those calls made in sequence. Arguments as in those
 * calls; workspace: pace_workspace_bytes(PACE_WS_FILTER_STEP, n_traj,
 * n_tokens) bytes. Argument errors return before anything is enqueued, with
 * *r_hat_inout unchanged. */
int pace_stream_step(const int32_t *tags, const int64_t *offsets, int64_t n_traj, int64_t n_tokens,
                     const int32_t *completion, int32_t current_version, const double *prefix_score,
                     const double *window_sorted, int64_t window_n, int64_t occupancy, int64_t capacity,
                     const pace_params *params, double *r_hat_inout, int64_t batch_size,
                     double *window_ring, int64_t window_cap, int64_t *window_state, double *score_out,
                     int64_t *gen_sum_out, int64_t *gen_count_out, uint8_t *status_out, uint8_t *keep_out,
                     int32_t *reject_ids_out, double *kappa_out, int64_t *counts_out, int n_cols,
                     const void *const *cols_in, const int32_t *elem_bytes, void *const *cols_out,
                     int64_t *offsets_out, int32_t *kept_ids_out, int64_t *n_kept_tokens_out,
                     void *workspace, size_t workspace_bytes, void *stream);

/* pace_prefix_score -- Prefix Forgetting Score (Eq. (5), Sec. 3.2): for each
 * rescored prefix, the mean absolute difference between the rescoring
 * policy's log-probabilities and the behaviour log-probabilities recorded at
 * generation, over the prefix's response tokens (Appendix B: only the first
 * `cap` of them count -- 1024 for math, 2048 for tool use -- and a prefix
 * needs at least `min_tokens` (32) of them, else it has no score).
 * lp_new, lp_behavior: f32 [n_tokens], packed prefixes; prefix i holds tokens
 *   [prefix_offsets[i], prefix_offsets[i+1]) (int64 [n+1], expected 0 ..
 *   n_tokens non-decreasing; clamped on the device).
 * tags: int32 [n_tokens] or NULL; a token tagged -1 is not a response token.
 * s_pre_out: f64 [n]; NaN for a prefix without a score (pace_score then
 *   applies no prefix weight, F = 1). Each term is formed in binary64 from the
 *   two f32 values; the terms are added in a fixed tree order (bit-identical
 *   run to run), which can differ from a sequential sum by a relative
 *   (cap + 2) * 2^-53 at most. */
int pace_prefix_score(const float *lp_new, const float *lp_behavior, const int32_t *tags,
                      const int64_t *prefix_offsets, int64_t n, int64_t n_tokens, int64_t cap,
                      int64_t min_tokens, double *s_pre_out, void *stream);

/* pace_stale_k -- the Stale-k admission rule (Sec. 2): a trajectory is
 * admitted iff its policy lag, Eq. (1) (the mean over response tokens of
 * j - v_t), is at most k. Exact: by Lemma 1 the lag is (S + (j - c) T) / T,
 * compared as integers. A trajectory without response tokens (T = 0) has lag
 * j - c.
 * gen_sum, gen_count: int64 [n_traj] (pace_score's S and T); completion:
 * int32 [n_traj]; current_version: j. k: 0 <= k < 2^31.
 * keep_out: u8 [n_traj], 1 = admitted; lag_out: f64 [n_traj] or NULL. */
int pace_stale_k(const int64_t *gen_sum, const int64_t *gen_count, const int32_t *completion,
                 int32_t current_version, int64_t n_traj, int64_t k, uint8_t *keep_out, double *lag_out,
                 void *stream);

/* pace_diagnostics -- the admission diagnostics of Sec. 4: histograms of
 * Waiting (K_wait = j - c), Generation (K_gen = S / T, 0 when T = 0) and
 * Effective Staleness (the admission score) over the candidates, split into
 * rejected (keep 0) and retained (keep != 0), and exact totals per class.
 * score: f64 [n_traj]; gen_sum, gen_count: int64 [n_traj]; keep: u8 [n_traj].
 * edges: f64 [3][nbins + 1] device, ascending per metric (K_wait, K_gen,
 *   K_eff); 1 <= nbins <= 1024. Bin b holds [edges[b], edges[b+1]).
 * hist_out: int64 [3][2][nbins + 2]: [metric][0 rejected, 1 retained][bin],
 *   bin 0 below the first edge, nbins + 1 at or above the last.
 * totals_out: int64 [2][4]: per class, count, sum of (j - c), sum S, sum T.
 * Four workgroups (one per metric, one for the totals); outputs are
 * overwritten, not accumulated. */
int pace_diagnostics(const double *score, const int64_t *gen_sum, const int64_t *gen_count,
                     const int32_t *completion, int32_t current_version, const uint8_t *keep, int64_t n_traj,
                     const double *edges, int nbins, int64_t *hist_out, int64_t *totals_out, void *stream);

/* pace_time_next_kernel -- measurement hook, not part of the method.
 * Arms a one-shot timer for one phase of the device work of the NEXT call
 * made from the calling host thread to an entry point that enqueues device
 * work (every call above except pace_default_params, pace_workspace_bytes,
 * pace_budget and pace_strerror): that call launches its first kernel of the
 * phase with hipExtLaunchKernel and the two events, so that
 * hipEventElapsedTime(start, stop) afterwards gives that kernel's own
 * execution time. When that call returns, every timer armed on the thread is
 * dropped, used or not: a timer never reaches a later call.
 * The armed timers are the library's only state between calls: a per-thread
 * table of at most PACE_PHASE_COUNT event pairs, empty except between
 * pace_time_next_kernel and the return of the next device call on that
 * thread. Calls on other threads never see it.
 * phase: PACE_PHASE_REDUCE (token reduction of pace_score), PACE_PHASE_FINALIZE
 *   (score finalisation), PACE_PHASE_SELECT (the rank kernel, the
 *   single-workgroup select of the largest pools, the streaming draw, or in
 *   pace_group_filter_step the rank over groups),
 *   PACE_PHASE_COMPACT (the compaction copy kernel), PACE_PHASE_PREFIX (the
 *   Prefix Forgetting Score kernel), PACE_PHASE_AUX (the single kernel of
 *   pace_group_score, pace_group_expand, pace_stale_k or pace_diagnostics,
 *   the window-cutoff kernel of the streaming rule, or in
 *   pace_group_filter_step the kernel that expands the group flags),
 *   PACE_PHASE_CLASSIFY
 *   (pools above 8192 trajectories: the kernel that finds the rejection cut
 *   and writes the keep flags; PACE_PHASE_SELECT then times the level-0
 *   histogram of that cut search).
 * start_event, stop_event: hipEvent_t handles created by the caller with
 *   timing enabled; both NULL disarms the phase. The caller keeps ownership.
 * Returns PACE_ERR_INVALID_ARG for an unknown phase or one NULL event. */
#define PACE_PHASE_REDUCE 0
#define PACE_PHASE_FINALIZE 1
#define PACE_PHASE_SELECT 2
#define PACE_PHASE_COMPACT 3
#define PACE_PHASE_PREFIX 4
#define PACE_PHASE_AUX 5
#define PACE_PHASE_CLASSIFY 6
#define PACE_PHASE_COUNT 7
int pace_time_next_kernel(int phase, void *start_event, void *stop_event);

/* Static description of an error code. */
const char *pace_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* PACE_H */
