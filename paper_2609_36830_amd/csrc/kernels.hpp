// Internal launch interface between the C ABI (pace_abi.cpp) and the gfx950
// kernels. Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pace {

// ---- score: segmented reduction over token chunks --------------------------
// One wave reduces one chunk of kScoreChunk consecutive tokens.
constexpr int64_t kScoreChunk = 8192;
// Largest prefix window staged in LDS by the finalize kernel.
constexpr int64_t kWindowLdsMax = 4096;

inline int64_t score_chunks(int64_t n_tokens) { return (n_tokens + kScoreChunk - 1) / kScoreChunk; }

struct ScoreWorkspace {
    uint64_t *part_sum;   // [n]   sum of (tag+1) over generated tokens of the piece that starts the segment
    int64_t *part_cnt;    // [n]   generated-token count of that piece
    uint64_t *carry_sum;  // [chunks] piece of the segment that straddles the chunk start
    int64_t *carry_cnt;   // [chunks]
};

size_t score_ws_bytes(int64_t n, int64_t n_tokens);
ScoreWorkspace score_ws_carve(void *ws, int64_t n, int64_t n_tokens);

hipError_t launch_score(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                        const int32_t *completion, int32_t V, const double *prefix,
                        const double *window, int64_t W, bool use_prefix, double w_wait, int gamma,
                        double *score, int64_t *gen_sum, int64_t *gen_count,
                        const ScoreWorkspace &ws, bool vec_ok, hipStream_t stream);

// ---- select ----------------------------------------------------------------
constexpr int kSelectThreads = 1024;
constexpr int kSelectMaxItems = 16;   // keys held in registers per thread
size_t select_ws_bytes(int64_t n);
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

size_t compact_ws_bytes(int64_t n, int64_t n_tokens);
hipError_t launch_compact(const int64_t *offsets, int64_t n, int64_t n_tokens, const uint8_t *keep,
                          const CompactCols &cols, int n_cols, int64_t *offsets_out,
                          int32_t *kept_ids, int64_t *n_kept_tokens, void *ws, hipStream_t stream);

// ---- validate --------------------------------------------------------------
hipError_t launch_validate(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                           const int32_t *completion, int32_t V, const double *window, int64_t W,
                           int32_t *err_word, hipStream_t stream);

inline size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace pace
