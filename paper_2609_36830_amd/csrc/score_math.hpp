// Per-trajectory score of the PACE filter (Sec. 2, Sec. 3.2), as the
// finalize kernel forms it from the reduction's pieces.
//
//   T      generated (tag != -1) tokens                        Eq. (1)
//   S      sum over them of (c - tag) = c T - sum(tag), exact   Eq. (2)
//   K_wait = V - c,  K_gen = S / T (0 when T = 0)               Eq. (2)
//   F      = a^g / (a^g + (W - a)^g), a = #{w <= s_pre}         Eq. (8), (9)
//   M      = (w_wait * K_wait) + (F * K_gen)                    Eq. (6), (7)
// Every floating-point operation is one IEEE binary64 round-to-nearest step
// in this order (contraction is off for every translation unit).
#pragma once

#include "device_util.hpp"

#pragma clang fp contract(off)

namespace pace {

struct TrajScore {
    int64_t S, T;
    double score;
};

// The reduce kernel leaves, per trajectory, the sum of (tag + 1) and the
// generated-token count of the piece in the chunk holding its first token
// (part_*) and of the piece in every later chunk it covers (carry_*).
struct TrajPieces {
    uint64_t sp;   // sum of (tag + 1) over generated tokens
    int64_t T;     // generated tokens
};

// Chunk holding token position p >= 0. The chunk length is a multiple of
// kScoreChunkAlign = 2^8, so p / chunk_len = (p >> 8) / (chunk_len >> 8);
// with narrow (every position below 2^40) that is a 32-bit division.
__device__ __forceinline__ int64_t chunk_of(int64_t p, int64_t chunk_len, bool narrow) {
    static_assert(kScoreChunkAlign == 256, "chunk lengths are multiples of 2^8");
    if (narrow) return (int64_t)((uint32_t)(p >> 8) / (uint32_t)(chunk_len >> 8));
    return p / chunk_len;
}

// Pieces of trajectory i covering tokens [lo, hi): its part and the carries
// of chunks lo / chunk_len + 1 .. (hi - 1) / chunk_len. The first kCarryBatch
// carries are loaded together (one round trip); longer spans loop.
constexpr int kCarryBatch = 4;
__device__ __forceinline__ TrajPieces gather_pieces(
    int64_t i, int64_t lo, int64_t hi, const uint64_t *__restrict__ part_sum,
    const int64_t *__restrict__ part_cnt, const uint64_t *__restrict__ carry_sum,
    const int64_t *__restrict__ carry_cnt, int64_t chunk_len, bool narrow) {
    TrajPieces p{0, 0};
    if (hi > lo) {
        p.sp = part_sum[i];
        p.T = part_cnt[i];
        const int64_t first = chunk_of(lo, chunk_len, narrow) + 1;
        const int64_t last = chunk_of(hi - 1, chunk_len, narrow);
        uint64_t cs[kCarryBatch];
        int64_t cc[kCarryBatch];
#pragma unroll
        for (int u = 0; u < kCarryBatch; ++u) {
            const bool in = first + u <= last;
            cs[u] = in ? carry_sum[first + u] : 0;
            cc[u] = in ? carry_cnt[first + u] : 0;
        }
#pragma unroll
        for (int u = 0; u < kCarryBatch; ++u) {
            p.sp += cs[u];
            p.T += cc[u];
        }
        for (int64_t ch = first + kCarryBatch; ch <= last; ++ch) {
            p.sp += carry_sum[ch];
            p.T += carry_cnt[ch];
        }
    }
    return p;
}

// Score of one trajectory from its pieces.
__device__ __forceinline__ TrajScore score_from_pieces(
    TrajPieces pc, int64_t c, int32_t V, bool use_prefix, double s_pre, const double *win, int64_t W,
    double w_wait, int gamma) {
    const uint64_t sp = pc.sp;
    const int64_t T = pc.T;
    // sp = sum(tag) + T over generated tokens
    const int64_t sum_tag = (int64_t)(sp - (uint64_t)T);
    TrajScore r;
    r.T = T;
    r.S = c * T - sum_tag;
    const double k_wait = (double)((int64_t)V - c);
    const double k_gen = (T > 0) ? (double)r.S / (double)T : 0.0;
    double F = 1.0;
    if (use_prefix && !__builtin_isnan(s_pre)) {
        int64_t a_lo = 0, a_hi = W;          // count of window entries <= s_pre
        while (a_lo < a_hi) {
            const int64_t mid = (a_lo + a_hi) >> 1;
            if (win[mid] <= s_pre) a_lo = mid + 1; else a_hi = mid;
        }
        int64_t A = 1, B = 1;
        for (int g = 0; g < gamma; ++g) {
            A *= a_lo;
            B *= (W - a_lo);
        }
        F = (double)A / (double)(A + B);
    }
    const double wait_term = w_wait * k_wait;
    const double gen_term = F * k_gen;
    r.score = wait_term + gen_term;
    return r;
}

}  // namespace pace
