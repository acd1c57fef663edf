// Internal launch interface between the C ABI (pace_abi.cpp) and the gfx950
// kernels. Not part of the public ABI.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <tuple>

namespace pace {

// Waves the device keeps resident for the streaming kernels (CUs x 16).
int64_t resident_waves();

// ---- launches with optional per-kernel timing ------------------------------
// The phases a caller may time (pace_time_next_kernel). When a timer is armed
// for a phase on the calling host thread, that phase's next kernel is
// launched with hipExtLaunchKernel and the two events, which then bracket
// the kernel's own execution; the timer is consumed by that launch.
enum TimedPhase : int { kPhaseReduce = 0, kPhaseFinalize = 1, kPhaseSelect = 2, kPhaseCompact = 3,
                        kPhasePrefix = 4, kPhaseAux = 5, kPhaseClassify = 6, kPhaseCount = 7 };
bool take_phase_timer(int phase, hipEvent_t *start, hipEvent_t *stop);

template <typename... P, typename... A>
hipError_t launch(int phase, void (*kernel)(P...), dim3 grid, dim3 block, hipStream_t stream, A... a) {
    static_assert(sizeof...(P) == sizeof...(A), "kernel argument count");
    hipEvent_t t0 = nullptr, t1 = nullptr;
    if (phase >= 0 && take_phase_timer(phase, &t0, &t1)) {
        std::tuple<P...> held{static_cast<P>(a)...};
        void *argv[sizeof...(P)];
        std::apply([&argv](auto &...x) {
            int k = 0;
            ((argv[k++] = (void *)&x), ...);
        }, held);
        return hipExtLaunchKernel((const void *)kernel, grid, block, argv, 0, stream, t0, t1, 0);
    }
    kernel<<<grid, block, 0, stream>>>(static_cast<P>(a)...);
    return hipGetLastError();
}

// ---- score: segmented reduction over token chunks --------------------------
// Waves per CU the reduction is sized for (its register use, at most 128
// VGPRs, keeps that many resident; 32 per CU would force spills and was
// measured much slower).
constexpr int kReduceWavesPerCU = 16;
// One wave reduces one chunk of consecutive tokens; the chunk length is a
// multiple of kScoreChunkAlign (one 256-token window, 1 KiB of tags) chosen so
// that the chunks fill the device once, and at least kScoreChunkMin (which
// bounds the number of chunks, and so the carry arrays, by n_tokens / 2048).
// A coarser alignment would leave waves idle: 52.1M tokens over 4096 waves is
// 12,721 per wave, which 2048-token alignment rounds to 14,336 (3636 chunks).
constexpr int64_t kScoreChunkAlign = 256;
constexpr int64_t kScoreChunkMin = 2048;
// Largest prefix window staged in LDS by the finalize kernel.
constexpr int64_t kWindowLdsMax = 4096;

inline int64_t score_chunk_len(int64_t n_tokens, int64_t waves) {
    int64_t per = (n_tokens + waves - 1) / (waves > 0 ? waves : 1);
    per = (per + kScoreChunkAlign - 1) / kScoreChunkAlign * kScoreChunkAlign;
    return per > kScoreChunkMin ? per : kScoreChunkMin;
}
// Upper bound on the chunk count for any device (the chunk is never shorter
// than kScoreChunkMin).
inline int64_t score_max_chunks(int64_t n_tokens) {
    return (n_tokens + kScoreChunkMin - 1) / kScoreChunkMin;
}

struct ScoreWorkspace {
    uint64_t *part_sum;   // [n]   sum of (tag+1) over generated tokens of the piece that starts the segment
    int64_t *part_cnt;    // [n]   generated-token count of that piece
    uint64_t *carry_sum;  // [chunks] piece of the segment that straddles the chunk start
    int64_t *carry_cnt;   // [chunks]
};

size_t score_ws_bytes(int64_t n, int64_t n_tokens);
ScoreWorkspace score_ws_carve(void *ws, int64_t n, int64_t n_tokens);

hipError_t launch_score_reduce(const int32_t *tags, const int64_t *offsets, int64_t n,
                               int64_t n_tokens, int32_t V, const ScoreWorkspace &ws, bool vec_ok,
                               hipStream_t stream, int64_t *chunk_len_out);
// With mmin/mmax non-null, also writes the smallest and largest score key
// of each group of kFinGroup trajectories (the wide selection's range) and
// clears hist0 (2^kCutBits words, the wide selection's level-0 histogram).
constexpr int kFinGroup = 128;
hipError_t launch_score_finalize(const int64_t *offsets, int64_t n, int64_t n_tokens,
                                 const int32_t *completion, int32_t V, const double *prefix,
                                 const double *window, int64_t W, bool use_prefix, double w_wait,
                                 int gamma, int64_t chunk_len, double *score, int64_t *gen_sum,
                                 int64_t *gen_count, const ScoreWorkspace &ws, hipStream_t stream,
                                 uint64_t *mmin = nullptr, uint64_t *mmax = nullptr,
                                 uint32_t *hist0 = nullptr);
hipError_t launch_score(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                        const int32_t *completion, int32_t V, const double *prefix,
                        const double *window, int64_t W, bool use_prefix, double w_wait, int gamma,
                        double *score, int64_t *gen_sum, int64_t *gen_count,
                        const ScoreWorkspace &ws, bool vec_ok, hipStream_t stream);

// ---- select ----------------------------------------------------------------
constexpr int kSelectThreads = 1024;
constexpr int kSelectMaxItems = 16;   // keys held in registers per thread
// Pools up to this size are selected by the multi-workgroup rank-by-counting
// kernel; larger pools by the single-workgroup radix select.
constexpr int64_t kRankMaxN = 8192;
// ---- compaction by pieces: block partials ----------------------------------
// Consecutive trajectories form blocks of kPieceBlock; a kept span of len
// tokens is cut into ceil(len / kPieceLen) pieces. Per block: kept count,
// kept tokens and pieces (lengths from offsets clamped to [0, n_tokens]).
constexpr int kPieceBlock = 16;
constexpr int64_t kPieceLen = 16384;
constexpr int64_t kPieceMaxN = 8192;   // at most 512 blocks
struct PieceParts {
    int32_t *cnt;
    int64_t *len;
    int32_t *pcs;      // blocks of kPieceBlock only
    int32_t *gcnt;     // wide blocks only: per group of kGroupBlocks blocks, the sums of cnt and len
    int64_t *glen;
};
inline int64_t piece_blocks(int64_t n) { return (n + kPieceBlock - 1) / kPieceBlock; }

// ---- selection spread over the chip (pools beyond kRankMaxN) ----------------
// The rejection cut: mode 0 rejects nothing, 1 everything, 2 every key >= key,
// 3 every key > key and the ids <= id among those with key == key.
struct CutRec {
    int64_t mode;
    uint64_t key;
    int64_t id;
    int64_t pad;
};
constexpr int kWideBlock = 64;          // trajectories per compaction block on the wide path
constexpr int kGroupBlocks = 16;        // wide blocks per group of the two-level block partials
constexpr int64_t kWideHistMax = 64;    // histogram workgroups
constexpr int64_t kWideMaxN = 262144;   // limit of the wide selection and compaction
constexpr int kWideMaxGroups = (int)(kWideMaxN / (kWideBlock * kGroupBlocks));
inline int64_t wide_groups(int64_t n) { return (n + kWideBlock * kGroupBlocks - 1) / (kWideBlock * kGroupBlocks); }
constexpr int kCutBits = 11;           // level-0 digits of the cut search: 2^kCutBits bins
struct WideWs {
    CutRec *cut;
    uint64_t *range;
    uint64_t *mmin, *mmax;   // [n_mm] per group of kFinGroup trajectories
    uint32_t *hist;          // [2^kCutBits] level-0 histogram, cleared by the kernel writing mmin/mmax
    uint16_t *digit;         // [n] level-0 digit of each trajectory
    PieceParts parts;        // [n / kWideBlock] partials when no compaction workspace is at hand
    int64_t n_mm;
};
int64_t wide_hist_wgs(int64_t n);
size_t wide_select_ws_bytes(int64_t n);
WideWs wide_ws_carve(void *ws, int64_t n);
hipError_t launch_key_minmax(const double *score, int64_t n, const WideWs &w, hipStream_t stream);
// The level-0 digits and histogram of the cut search (after the kernel that
// writes mmin/mmax and clears hist).
hipError_t launch_wide_cut(const double *score, int64_t n, int64_t budget, const WideWs &w, hipStream_t stream);

// keep[i] <- 0 for the `budget` first trajectories in (score desc, id asc).
// With parts.cnt non-null, also writes the block partials of the keep flags.
// Group means of pace_group_score formed inside the rank over groups (at
// most kRankMaxN groups): group scores and group keep flags in one launch.
// Every rank workgroup (one per kRankQ groups) reads all member scores, so
// the group step uses it while ceil(ng / kRankQ) * n stays within
// kGroupRankLoads, and a separate pass of group means before the rank beyond.
constexpr int kRankQ = 16;              // targets per rank workgroup
constexpr int64_t kGroupRankLoads = (int64_t)1 << 21;
hipError_t launch_group_rank(const double *score, int64_t n, const int64_t *group_offsets, int64_t ng,
                             int64_t budget, double *group_score, uint8_t *group_keep, hipStream_t stream);
hipError_t launch_rank(const double *score, int64_t n, int64_t budget, uint8_t *keep,
                       const int64_t *offsets, int64_t n_tokens, const PieceParts &parts,
                       hipStream_t stream);
size_t select_ws_bytes(int64_t n);
// Every workgroup finds the cut of the `budget` highest from the level-0
// histogram and digits, then classifies its trajectories (keep flags, block
// partials; offsets may be null: keep flags and kept counts only); w.cut
// receives the cut.
hipError_t launch_classify(const double *score, const int64_t *offsets, int64_t n, int64_t n_tokens,
                           int64_t budget, const WideWs &w, uint8_t *keep, const PieceParts &parts,
                           hipStream_t stream);
hipError_t launch_emit_rejects_wide(const uint8_t *keep, int64_t n, const int32_t *kept_cnt, int64_t budget,
                                    int32_t *reject_ids, hipStream_t stream);
hipError_t launch_select(const double *score, int64_t n, int64_t budget, uint8_t *keep,
                         int32_t *reject_ids, void *ws, hipStream_t stream);

// ---- compact ---------------------------------------------------------------
constexpr int kMaxCols = 8;
// Output chunk (elements) handled by one wave of the copy kernel.
constexpr int64_t kCopyChunk = 4096;

struct CompactCols {
    const void *in[kMaxCols];
    void *out[kMaxCols];
    int32_t elem[kMaxCols];
    int32_t vec[kMaxCols];   // 1 when both pointers are 16-byte aligned
};

struct CompactWs {
    int64_t *hdr;          // [0] kept trajectories, [1] min(kept tokens, n_tokens)
    int64_t *kept_src;     // [n] source start of each kept span
    int32_t *chunk_first;  // [map_capacity] kept span covering each output chunk's first element
    PieceParts parts;      // [piece_blocks(n)] block partials (piece path)
};
int64_t map_capacity(int64_t n_tokens);
CompactWs compact_ws_carve(void *ws, int64_t n, int64_t n_tokens);
size_t compact_ws_bytes(int64_t n, int64_t n_tokens);
hipError_t launch_compact_copy(const CompactCols &cols, int n_cols, int64_t n_tokens,
                               const int64_t *offsets_out, const CompactWs &w, hipStream_t stream);
// Piece path (at most kPieceMaxN trajectories): one workgroup per block
// writes that block's packed offsets, kept ids and rejected ids; one
// workgroup per piece copies it. reject_ids may be NULL; when given, the ids
// with keep == 0 go there in ascending order (at most `budget` of them).
// The block partials come from the rank kernel or from launch_compact_partials.
// max_kept bounds the number of kept trajectories (n when unknown); the grid
// holds max_kept + n_tokens / kPieceLen piece workgroups.
bool compact_piece_ok(int64_t n, int64_t n_tokens);
// Blocks of kWideBlock trajectories: pools of up to kWideMaxN.
bool compact_wide_ok(int64_t n, int64_t n_tokens);
hipError_t launch_compact_partials(const int64_t *offsets, int64_t n, int64_t n_tokens,
                                   const uint8_t *keep, const PieceParts &parts, hipStream_t stream,
                                   int blk = kPieceBlock);
// blk: trajectories per block of the partials (kPieceBlock or kWideBlock).
// copy = false launches the block workgroups only (rejected ids; no columns).
hipError_t launch_compact_pieces(const int64_t *offsets, int64_t n, int64_t n_tokens, const uint8_t *keep,
                                 const PieceParts &parts, const CompactCols &cols, int n_cols,
                                 int64_t *offsets_out, int32_t *kept_ids, int64_t *n_kept_tokens,
                                 int32_t *reject_ids, int64_t budget, int64_t max_kept,
                                 hipStream_t stream, int blk = kPieceBlock, bool copy = true);
hipError_t launch_compact(const int64_t *offsets, int64_t n, int64_t n_tokens, const uint8_t *keep,
                          const CompactCols &cols, int n_cols, int64_t *offsets_out,
                          int32_t *kept_ids, int64_t *n_kept_tokens, void *ws, hipStream_t stream);

// ---- whole filter step (fused middle kernel) --------------------------------
size_t filter_step_ws_bytes(int64_t n, int64_t n_tokens);
hipError_t launch_filter_step(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                              const int32_t *completion, int32_t V, const double *prefix,
                              const double *window, int64_t W, bool use_prefix, double w_wait,
                              int gamma, int64_t budget, double *score, int64_t *gen_sum,
                              int64_t *gen_count, uint8_t *keep, int32_t *reject_ids,
                              const CompactCols &cols, int n_cols, int64_t *offsets_out,
                              int32_t *kept_ids, int64_t *n_kept_tokens, void *ws, bool vec_ok,
                              hipStream_t stream);

// ---- group-level admission ---------------------------------------------------
hipError_t launch_group_score(const double *score, int64_t n, const int64_t *group_offsets, int64_t ng,
                              double *group_score, hipStream_t stream);
hipError_t launch_group_expand(const int64_t *group_offsets, int64_t ng, int64_t n, const uint8_t *group_keep,
                               uint8_t *keep, hipStream_t stream);
hipError_t launch_group_validate(const int64_t *group_offsets, int64_t ng, int64_t n, int32_t *err,
                                 hipStream_t stream);
// pace_group_filter_step's device work; ws is a filter-step workspace.
hipError_t launch_group_filter_step(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                                    const int32_t *completion, int32_t V, const double *prefix,
                                    const double *window, int64_t W, bool use_prefix, double w_wait,
                                    int gamma, const int64_t *group_offsets, int64_t ng, int64_t budget,
                                    double *score, int64_t *gen_sum, int64_t *gen_count,
                                    double *group_score, uint8_t *group_keep, int32_t *reject_group_ids,
                                    uint8_t *keep, const CompactCols &cols, int n_cols,
                                    int64_t *offsets_out, int32_t *kept_ids, int64_t *n_kept_tokens,
                                    void *ws, bool vec_ok, hipStream_t stream);

// ---- streaming admission rule ------------------------------------------------
constexpr int64_t kStreamWindowMax = 1024;   // largest score window (ring entries)
// With offsets and parts.cnt non-null, the draw also writes the compaction's
// block partials of its keep flags (offsets clamped to [0, n_tokens]).
hipError_t launch_stream_admit(const double *score, int64_t n, double rate, int64_t window_min, int64_t B,
                               double *ring, int64_t cap, int64_t *state, uint8_t *status, uint8_t *keep,
                               int32_t *reject_ids, double *kappa, int64_t *counts, const int64_t *offsets,
                               int64_t n_tokens, const PieceParts &parts, hipStream_t stream);

// ---- Prefix Forgetting Score --------------------------------------------------
hipError_t launch_prefix_score(const float *lp_new, const float *lp_beh, const int32_t *tags,
                               const int64_t *prefix_offsets, int64_t n, int64_t n_tokens, int64_t cap,
                               int64_t min_tokens, double *s_pre, hipStream_t stream);

// ---- Stale-k admission and diagnostics ----------------------------------------
constexpr int kDiagBinsMax = 1024;
hipError_t launch_stale_k(const int64_t *S, const int64_t *T, const int32_t *completion, int32_t V, int64_t n,
                          int64_t k, uint8_t *keep, double *lag, hipStream_t stream);
hipError_t launch_diagnostics(const double *score, const int64_t *S, const int64_t *T, const int32_t *completion,
                              int32_t V, const uint8_t *keep, int64_t n, const double *edges, int nbins,
                              int64_t *hist, int64_t *totals, hipStream_t stream);

// ---- validate --------------------------------------------------------------
hipError_t launch_validate(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                           const int32_t *completion, int32_t V, const double *window, int64_t W,
                           int32_t *err_word, hipStream_t stream);

// Device address of the current device's fixed scratch array
// (PACE_NOALLOC_SCRATCH_BYTES bytes, 256-byte aligned), looked up once per
// device.
hipError_t noalloc_scratch(void **out);

inline size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace pace
