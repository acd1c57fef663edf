// Group-level admission for gfx950 (Appendix B: the full method aggregates
// scores by the mean within prompt groups, and its score window and
// diagnostics count groups). Consecutive trajectories form prompt groups:
// group g holds trajectories [group_offsets[g], group_offsets[g+1]). A group
// is scored by the mean of its members' scores, budgeted, selected and
// compacted as one unit. Group offsets are clamped to [0, n] on the device,
// so malformed ones give unspecified results but no out-of-bounds access.
#include "../../include/pace.h"
#include "device_util.hpp"
#include "group_math.hpp"
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
    out[g] = group_mean(score, n, go, g);
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

// After the rank over groups, in the group filter step: workgroup w writes
// the keep flags of trajectories [1024 w, 1024 w + 1024) (their group's
// flag), the compaction's partials of the kPieceBlock-trajectory blocks among
// them, and the rejected ids among groups [1024 w, 1024 w + 1024), ascending
// (at most `budget` of them, as pace_select writes them). A trajectory's
// group is the last group whose first member is at or before it; wave 0
// finds that of the workgroup's first trajectory, the next kAdmStage group
// offsets are staged in LDS, and every thread searches them (the global
// offsets when its group lies beyond).
// kWide: the partials of blocks of kWideBlock trajectories (one wave) and
// their sums per workgroup (one group of kGroupBlocks blocks), the two
// levels the merge-path compaction reads; else blocks of kPieceBlock.
constexpr int kAdmT = 1024;
constexpr int kAdmStage = 2048;
static_assert(kAdmT == kWideBlock * kGroupBlocks, "a workgroup is one group of wide blocks");
template <bool kWide>
__global__ __launch_bounds__(kAdmT) void group_admit_kernel(const int64_t *__restrict__ go, int64_t ng, int64_t n,
                                                           const uint8_t *__restrict__ gkeep,
                                                           const int64_t *__restrict__ off, int64_t NT,
                                                           uint8_t *__restrict__ keep, PieceParts parts,
                                                           int32_t *__restrict__ reject_gids, int64_t budget) {
    __shared__ int64_t s_go[kAdmStage + 1];
    __shared__ int64_t s_gs;
    __shared__ uint32_t wsum[kAdmT / kWave];
    __shared__ int64_t wlen[kAdmT / kWave];
    const int t = threadIdx.x, lane = lane_id();
    const int64_t a = (int64_t)blockIdx.x * kAdmT;
    const int64_t i = a + t;

    // Loads that need no search: the trajectory's span, the rejected-group
    // flags before this workgroup's groups (strided) and its own group flag.
    int64_t span = 0;
    if (i < n) {
        const int64_t lo = clamp64(off[i], 0, NT), hi = clamp64(off[i + 1], 0, NT);
        span = hi > lo ? hi - lo : 0;
    }
    const int64_t a_g = a < ng ? a : ng;
    uint32_t before = 0;
    for (int64_t k = t; k < a_g; k += kAdmT) before += gkeep[k] == 0 ? 1u : 0u;
    const int64_t gr = a + t;
    const bool rej = gr < ng && gkeep[gr] == 0;

    // The group of trajectory a, then the staged group offsets.
    if (ng > 0 && a < n && t < kWave) {
        int64_t gs = wave_last_le(go, ng - 1, a);
        gs = gs < 0 ? 0 : gs;
        if (t == 0) s_gs = gs;
    }
    // Rejected ids: rej | (strided count << 11) in one block sum (the
    // workgroup holds at most 1024 rejected groups: 11 bits).
    uint32_t tot;
    const uint32_t ex = block_excl_sum_u32<kAdmT / kWave>((rej ? 1u : 0u) | (before << 11), tot, wsum);
    if (rej && reject_gids) {
        const int64_t pos = (int64_t)(tot >> 11) + (int64_t)(ex & 2047u);
        if (pos < budget) reject_gids[pos] = (int32_t)gr;
    }
    if (ng == 0 || a >= n) return;            // no trajectory here (block-uniform)
    const int64_t gs = s_gs;
    const int64_t m = (ng - gs < kAdmStage) ? ng - gs : kAdmStage;   // s_go[0..m] = go[gs..gs+m]
    for (int64_t k = t; k <= m; k += kAdmT) s_go[k] = go[gs + k];
    __syncthreads();

    bool kept = false;
    if (i < n) {
        // last k in [0, m) with s_go[k] <= i (s_go[0] <= a <= i for well-formed offsets)
        int64_t lo = 0, hi = m;
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) >> 1;
            if (s_go[mid] <= i) lo = mid; else hi = mid;
        }
        int64_t g = gs + lo;
        if (m < ng - gs && s_go[m] <= i) {    // beyond the staged offsets: search the rest
            int64_t l2 = gs + m, h2 = ng;
            while (h2 - l2 > 1) {
                const int64_t mid = (l2 + h2) >> 1;
                if (go[mid] <= i) l2 = mid; else h2 = mid;
            }
            g = l2;
        }
        kept = gkeep[g] != 0;
        keep[i] = kept ? 1 : 0;
    }

    const int64_t len = kept ? span : 0;
    if constexpr (kWide) {
        // A wave is a block of kWideBlock trajectories; the workgroup is
        // their group.
        static_assert(kWideBlock == kWave, "a wide block is one wave");
        const uint32_t c = (uint32_t)__popcll(ballot(kept));
        const int64_t l = wave_sum_i64(len);
        const int w = t / kWave;
        const int64_t b = i / kWideBlock;
        if (lane == 0) {
            if (b * kWideBlock < n) {
                parts.cnt[b] = (int32_t)c;
                parts.len[b] = l;
            }
            wsum[w] = c;
            wlen[w] = l;
        }
        __syncthreads();
        if (t == 0) {
            uint32_t gc = 0;
            int64_t gl = 0;
            for (int k = 0; k < kAdmT / kWave; ++k) {
                gc += wsum[k];
                gl += wlen[k];
            }
            parts.gcnt[blockIdx.x] = (int32_t)gc;
            parts.glen[blockIdx.x] = gl;
        }
    } else {
        // Rows of 16 lanes are blocks of kPieceBlock trajectories.
        static_assert(kPieceBlock == 16 && kAdmT % kPieceBlock == 0, "a block is one row of 16 lanes");
        const int64_t l_row = row_incl_scan_i64(len);
        const uint32_t p_row = row_incl_scan_u32((uint32_t)((len + kPieceLen - 1) / kPieceLen));
        const uint32_t c_row = (uint32_t)__popcll((ballot(kept) >> (lane & ~15)) & 0xffffull);
        const int64_t b = i / kPieceBlock;
        if ((lane & 15) == 15 && b * kPieceBlock < n) {
            parts.cnt[b] = (int32_t)c_row;
            parts.len[b] = l_row;
            parts.pcs[b] = (int32_t)p_row;
        }
    }
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

hipError_t launch_group_admit(const int64_t *group_offsets, int64_t ng, int64_t n, const uint8_t *group_keep,
                              const int64_t *offsets, int64_t n_tokens, uint8_t *keep, const PieceParts &parts,
                              int32_t *reject_group_ids, int64_t budget, bool wide, hipStream_t stream) {
    const int64_t items = n > ng ? n : ng;
    const int64_t wgs = items > 0 ? (items + kAdmT - 1) / kAdmT : 0;
    if (wgs == 0) return hipSuccess;
    if (wide)
        return launch(kPhaseAux, group_admit_kernel<true>, dim3((unsigned)wgs), dim3(kAdmT), stream, group_offsets,
                      ng, n, group_keep, offsets, n_tokens, keep, parts, reject_group_ids, budget);
    return launch(kPhaseAux, group_admit_kernel<false>, dim3((unsigned)wgs), dim3(kAdmT), stream, group_offsets, ng,
                  n, group_keep, offsets, n_tokens, keep, parts, reject_group_ids, budget);
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
    const bool pieces = compact_piece_ok(n, n_tokens);
    if (ng <= kRankMaxN && (pieces || compact_wide_ok(n, n_tokens))) {
        // Group scores inside the rank over groups; one kernel for the
        // members' flags, the compaction's partials (blocks of 16, or of 64
        // with group sums for the merge-path compaction) and the rejected ids.
        const CompactWs cw = compact_ws_carve(cws, N, n_tokens);
        if ((ng + kRankQ - 1) / kRankQ * n <= kGroupRankLoads) {
            e = launch_group_rank(score, n, group_offsets, ng, budget, group_score, group_keep, stream);
        } else {
            // Every rank workgroup re-forming every mean would read the
            // scores ng / kRankQ times over: form them once.
            e = launch_group_score(score, n, group_offsets, ng, group_score, stream);
            if (e == hipSuccess)
                e = launch_rank(group_score, ng, budget, group_keep, nullptr, 0, PieceParts{}, stream);
        }
        if (e != hipSuccess) return e;
        e = launch_group_admit(group_offsets, ng, n, group_keep, offsets, n_tokens, keep, cw.parts,
                               reject_group_ids, budget, !pieces, stream);
        if (e != hipSuccess) return e;
        return launch_compact_pieces(offsets, n, n_tokens, keep, cw.parts, cols, n_cols, offsets_out, kept_ids,
                                     n_kept_tokens, nullptr, 0, n, stream, pieces ? kPieceBlock : kWideBlock);
    }
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
