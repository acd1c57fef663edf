// pace_filter_step: the whole filter step (Algorithm 1, trainer side) on
// one stream, every phase spread over the whole device:
//
//   1. score_reduce   (score.hip)    every tag read once, per-chunk pieces
//   2. score_finalize (score.hip)    one thread per trajectory: the score
//   3. rank           (select.hip)   exact rank by counting -> keep flags,
//                                    plus per-block kept counts, kept tokens
//                                    and piece counts
//   4. compact_piece  (compact.hip)  one workgroup per block writes the packed
//                                    offsets, kept ids and rejected ids; one
//                                    per piece of a kept span copies it
//
// The same results as pace_score, pace_budget, pace_select and pace_compact
// called in sequence, in four launches instead of six. Pools beyond the rank
// kernel's limit (8192 trajectories) take the selection spread over the chip
// instead of the rank (select_wide.hip: the finalize also writes per-group
// key extremes and clears the level-0 histogram, then cut_hist, and classify,
// where every workgroup finds the cut and writes keep flags, the partials of
// blocks of 64 trajectories and their group sums) and compact_wide (an even
// merge-path split of the packed output); pools beyond that path's limit use
// the separate calls' kernels.
#include "device_util.hpp"
#include "kernels.hpp"

namespace pace {

size_t filter_step_ws_bytes(int64_t n, int64_t n_tokens) {
    return align256(score_ws_bytes(n, n_tokens)) + align256(compact_ws_bytes(n, n_tokens)) +
           align256(select_ws_bytes(n));
}

hipError_t launch_filter_step(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                              const int32_t *completion, int32_t V, const double *prefix,
                              const double *window, int64_t W, bool use_prefix, double w_wait,
                              int gamma, int64_t budget, double *score, int64_t *gen_sum,
                              int64_t *gen_count, uint8_t *keep, int32_t *reject_ids,
                              const CompactCols &cols, int n_cols, int64_t *offsets_out,
                              int32_t *kept_ids, int64_t *n_kept_tokens, void *ws, bool vec_ok,
                              hipStream_t stream) {
    char *p = (char *)ws;
    const ScoreWorkspace sws = score_ws_carve(p, n, n_tokens);
    p += align256(score_ws_bytes(n, n_tokens));
    void *cws_base = p;
    p += align256(compact_ws_bytes(n, n_tokens));
    void *sel_ws = p;

    const bool rank_path = n <= kRankMaxN && compact_piece_ok(n, n_tokens);
    const bool wide_path = !rank_path && compact_wide_ok(n, n_tokens);
    const WideWs ww = wide_ws_carve(sel_ws, n);
    int64_t chunk_len = 0;
    hipError_t e = launch_score_reduce(tags, offsets, n, n_tokens, V, sws, vec_ok, stream, &chunk_len);
    if (e != hipSuccess) return e;
    e = launch_score_finalize(offsets, n, n_tokens, completion, V, prefix, window, W, use_prefix,
                              w_wait, gamma, chunk_len, score, gen_sum, gen_count, sws, stream,
                              wide_path ? ww.mmin : nullptr, wide_path ? ww.mmax : nullptr,
                              wide_path ? ww.hist : nullptr);
    if (e != hipSuccess) return e;
    if (wide_path) {
        const CompactWs cw = compact_ws_carve(cws_base, n, n_tokens);
        e = launch_wide_cut(score, n, budget, ww, stream);
        if (e != hipSuccess) return e;
        e = launch_classify(score, offsets, n, n_tokens, budget, ww, keep, cw.parts, stream);
        if (e != hipSuccess) return e;
        const int64_t n_kept = n - (budget < n ? budget : n);
        return launch_compact_pieces(offsets, n, n_tokens, keep, cw.parts, cols, n_cols, offsets_out,
                                     kept_ids, n_kept_tokens, reject_ids, budget, n_kept, stream, kWideBlock,
                                     true);
    }
    if (rank_path) {
        const CompactWs cw = compact_ws_carve(cws_base, n, n_tokens);
        e = launch_rank(score, n, budget, keep, offsets, n_tokens, cw.parts, stream);
        if (e != hipSuccess) return e;
        // The rank rejects exactly min(budget, n) trajectories.
        const int64_t n_kept = n - (budget < n ? budget : n);
        return launch_compact_pieces(offsets, n, n_tokens, keep, cw.parts, cols, n_cols, offsets_out,
                                     kept_ids, n_kept_tokens, reject_ids, budget, n_kept, stream);
    }
    e = launch_select(score, n, budget, keep, reject_ids, sel_ws, stream);
    if (e != hipSuccess) return e;
    return launch_compact(offsets, n, n_tokens, keep, cols, n_cols, offsets_out, kept_ids,
                          n_kept_tokens, cws_base, stream);
}

}  // namespace pace
