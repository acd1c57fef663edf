// pace_score kernels for gfx950.
//
// Step 1 (score_reduce): every per-token version tag is read exactly once.
// The token array is cut into equal chunks of consecutive tokens, one per
// wave64, sized so that every resident wave gets exactly one (a multiple of
// 2048 tokens); a chunk is read as 16-byte vectors, 8 per lane in flight, the
// first batch issued before the trajectory search. (Plain loads on purpose:
// they leave the tags in the last-level cache, where the compaction re-reads
// the kept spans.) The wave
// walks the trajectory boundaries that fall inside its chunk and keeps, per
// lane, the running piece sum of (tag + 1) over generated tokens (masked
// tags, -1, add 0) and the generated-token count. When a trajectory ends the
// wave reduces the piece across lanes and holds it in a lane until the chunk
// is done, then stores every held piece at once:
//   - the piece of a trajectory that starts inside this chunk goes to
//     part_{sum,cnt}[trajectory] (exactly one chunk holds each start);
//   - the piece of the trajectory that straddles the chunk start goes to
//     carry_{sum,cnt}[chunk] (at most one per chunk).
// No atomics, no zero-filled workspace, and the combine order is fixed, so
// the integer results are bit-identical run to run.
//
// Step 2 (score_finalize): one thread per trajectory adds its carries, forms
// S_i = c_i T_i - sum(tag) exactly in int64 and evaluates the score of
// Eq. (6)-(9) in binary64 with a fixed operation order (no contraction).
#include "device_util.hpp"
#include "kernels.hpp"
#include "score_math.hpp"

#pragma clang fp contract(off)

namespace pace {

namespace {

constexpr int kVec = 4;                       // tags per lane per window
constexpr int kWin = kWave * kVec;            // 256 tokens per wave window
constexpr int kUnroll = 8;                    // windows per super-window
constexpr int kSub = 4;                       // windows per fast-path / walk block
constexpr int kWavesPerBlock = 4;
static_assert(kScoreChunkAlign % (kWin * kUnroll) == 0, "chunk must be a multiple of the super-window");

// Lane k caches clamp(off[base + k], 0, NT); reads of increasing indices only.
struct BoundCache {
    int64_t base;
    int64_t val;
    __device__ __forceinline__ void load(const int64_t *__restrict__ off, int64_t n, int64_t NT, int64_t b) {
        base = b;
        int64_t idx = b + lane_id();
        val = (idx <= n) ? clamp64(off[idx], 0, NT) : NT;
    }
    __device__ __forceinline__ int64_t get(const int64_t *__restrict__ off, int64_t n, int64_t NT, int64_t i) {
        if (i < base || i - base >= kWave) load(off, n, NT, i);
        return readlane_i64(val, (int)(i - base));
    }
};

// Tags are >= -1, so (tag + 1) summed is the tags' sum plus 4 (mod 2^32; the
// true partial stays below 2^32), and a tag is masked exactly when its sign
// bit is set.
__device__ __forceinline__ void add_all(const int4 &v, uint32_t &s, uint32_t &c) {
    const uint32_t x0 = (uint32_t)v.x, x1 = (uint32_t)v.y, x2 = (uint32_t)v.z, x3 = (uint32_t)v.w;
    s += x0 + x1 + x2 + x3 + 4u;
    c += 4u - ((x0 >> 31) + (x1 >> 31) + (x2 >> 31) + (x3 >> 31));
}

__device__ __forceinline__ void add_all_wide(const int4 &v, uint64_t &s, uint32_t &c) {
    uint32_t u0 = (uint32_t)v.x + 1u, u1 = (uint32_t)v.y + 1u;
    uint32_t u2 = (uint32_t)v.z + 1u, u3 = (uint32_t)v.w + 1u;
    s += (uint64_t)u0 + (uint64_t)u1 + (uint64_t)u2 + (uint64_t)u3;
    c += (u0 != 0u) + (u1 != 0u) + (u2 != 0u) + (u3 != 0u);
}

// Elements of this lane's vector (relative positions r0 .. r0 + 3) that lie
// in [rlo, rlo + rlen).
__device__ __forceinline__ void add_range(const int4 &v, uint32_t r0, uint32_t rlo, uint32_t rlen,
                                          uint64_t &s, uint32_t &c) {
    const int x[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (r0 + (uint32_t)e - rlo < rlen) {
            const uint32_t u = (uint32_t)x[e] + 1u;
            s += u;
            c += (u != 0u);
        }
    }
}

template <bool kVecLoad, int U>
__device__ __forceinline__ void load_super(const int32_t *__restrict__ tags, int64_t pos, int64_t ce,
                                           int lane, int4 (&v)[U]) {
#pragma unroll
    for (int k = 0; k < U; ++k) {
        const int64_t q = pos + (int64_t)k * kWin + (int64_t)lane * kVec;
        if (kVecLoad && q + kVec <= ce) {
            v[k] = *reinterpret_cast<const int4 *>(tags + q);
        } else {
            v[k] = make_int4(-1, -1, -1, -1);      // past the end: masked, adds nothing
            if (q < ce) v[k].x = tags[q];
            if (q + 1 < ce) v[k].y = tags[q + 1];
            if (q + 2 < ce) v[k].z = tags[q + 2];
            if (q + 3 < ce) v[k].w = tags[q + 3];
        }
    }
}

// kNarrow: every tag + 1 < 2^24, so a lane's 32 tags of one super-window sum
// below 2^29 in 32 bits before widening.
template <bool kNarrow, bool kVecLoad, int U = kUnroll>
__global__ __launch_bounds__(256) void score_reduce_kernel(
    const int32_t *__restrict__ tags, const int64_t *__restrict__ off, int64_t n, int64_t NT,
    int64_t chunk_len, int64_t n_chunks, uint64_t *__restrict__ part_sum,
    int64_t *__restrict__ part_cnt, uint64_t *__restrict__ carry_sum,
    int64_t *__restrict__ carry_cnt) {
    const int lane = lane_id();
    const int64_t chunk = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x / kWave);
    if (chunk >= n_chunks) return;
    const int64_t cs = chunk * chunk_len;
    const int64_t ce = (cs + chunk_len < NT) ? cs + chunk_len : NT;

    // The first super-window's loads do not depend on the trajectory search:
    // issue them first so the search latency hides under them.
    constexpr int64_t kSuper = (int64_t)kWin * U;
    int4 va[U];
    load_super<kVecLoad>(tags, cs, ce, lane, va);

    // Trajectory that contains the chunk's first token. First guess: the
    // 64 offsets around the position the token would have if all
    // trajectories were equally long (one round of loads, which also fills
    // the bound cache); if the answer is not inside that window, a 64-ary
    // search over all offsets.
    BoundCache bc;
    int64_t s;
    {
        const int64_t guess = NT > 0 ? (int64_t)((double)cs / (double)NT * (double)n) : 0;
        const int64_t top = (n + 1 > kWave) ? n + 1 - kWave : 0;
        const int64_t base = guess - kWave / 2 < 0 ? 0 : (guess - kWave / 2 > top ? top : guess - kWave / 2);
        const int64_t idx = base + lane;
        const int64_t raw = (idx <= n) ? off[idx] : INT64_MAX;
        const uint64_t m = ballot(idx <= n && raw <= cs);
        const bool lo_ok = base == 0 || (m & 1ull);
        const bool hi_ok = base + kWave > n || !(m >> (kWave - 1));
        if (lo_ok && hi_ok) {
            s = base + (int64_t)__popcll(m) - 1;
            bc.base = base;
            bc.val = (idx <= n) ? clamp64(raw, 0, NT) : NT;
        } else {
            s = wave_last_le(off, n, cs);
            bc.base = INT64_MIN / 2;          // empty: the first get() loads
            bc.val = 0;
        }
    }
    int64_t cur, cur_end;
    bool valid = false, pending = false, carry_piece = false;
    if (s < 0) {                 // only for malformed offsets: tokens before offsets[0]
        cur = -1;
        cur_end = bc.get(off, n, NT, 0);
    } else if (s >= n) {         // tokens at or past offsets[n]
        cur = n;
        cur_end = INT64_MAX;
    } else {
        cur = s;
        const int64_t cur_start = bc.get(off, n, NT, s);
        cur_end = bc.get(off, n, NT, s + 1);
        valid = true;
        pending = true;
        carry_piece = cur_start < cs;
    }

    uint64_t acc_s = 0;
    uint32_t acc_c = 0;

    // Finished pieces wait in registers, the k-th in lane k, and are stored
    // after the last super-window: a store in mid-stream would hold up the
    // next loads (the vector memory counter covers stores too). Past 64
    // pieces a chunk stores directly.
    int n_held = 0;                     // wave-uniform
    uint64_t held_s = 0;
    int64_t held_c = 0, held_at = 0;    // held_at: trajectory, or -1 for the carry
    auto store_piece = [&](int64_t at, uint64_t ts, int64_t tc) {
        if (at < 0) {
            carry_sum[chunk] = ts;
            carry_cnt[chunk] = tc;
        } else {
            part_sum[at] = ts;
            part_cnt[at] = tc;
        }
    };
    auto flush = [&]() {
        const uint64_t ts = wave_sum_u64(acc_s);
        const int64_t tc = (int64_t)wave_sum_u64((uint64_t)acc_c);
        const int64_t at = carry_piece ? -1 : cur;
        if (n_held < kWave) {
            if (lane == n_held) {
                held_s = ts;
                held_c = tc;
                held_at = at;
            }
            ++n_held;
        } else if (lane == 0) {
            store_piece(at, ts, tc);
        }
        acc_s = 0;
        acc_c = 0;
    };

    // Boundary walk over the kSub vectors at vb (tokens [bpos, bend)): walk
    // the trajectory ends in order; for each trajectory piece every lane adds
    // its tags whose positions fall in the piece.
    auto walk = [&](int4 *vb, int64_t bpos, int64_t bend) {
        int64_t lo = bpos;
        while (true) {
            const int64_t hi = cur_end < bend ? cur_end : bend;
            if (valid && hi > lo) {
                // Keep the per-tag work inside this loop: hoisted out of it,
                // it would hold every tag's (tag + 1) live at once.
#pragma unroll
                for (int k = 0; k < kSub; ++k)
                    asm volatile("" : "+v"(vb[k].x), "+v"(vb[k].y), "+v"(vb[k].z), "+v"(vb[k].w));
                // Positions relative to the block fit in 32 bits.
                const uint32_t rlo = (uint32_t)(lo - bpos), rlen = (uint32_t)(hi - lo);
                uint64_t ps = 0;
                uint32_t pc = 0;
#pragma unroll
                for (int k = 0; k < kSub; ++k)
                    add_range(vb[k], (uint32_t)(k * kWin + lane * kVec), rlo, rlen, ps, pc);
                acc_s += ps;
                acc_c += pc;
            }
            if (cur_end > bend) break;            // trajectory continues past this block
            if (pending) flush();                 // trajectory `cur` ends at cur_end
            lo = cur_end;
            ++cur;
            while (cur < n && bc.get(off, n, NT, cur + 1) <= lo) ++cur;   // skip empty ones
            carry_piece = false;
            if (cur >= n) {
                valid = false;
                pending = false;
                cur_end = INT64_MAX;
            } else {
                valid = true;
                cur_end = bc.get(off, n, NT, cur + 1);
                pending = lo < ce;
            }
            if (lo >= bend) break;
        }
    };

    // Adds the kSub vectors at vb (all inside trajectory `cur`).
    auto add_block = [&](const int4 *vb) {
        if (kNarrow) {
            uint32_t s32 = 0, c32 = 0;
#pragma unroll
            for (int k = 0; k < kSub; ++k) add_all(vb[k], s32, c32);
            acc_s += s32;
            acc_c += c32;
        } else {
#pragma unroll
            for (int k = 0; k < kSub; ++k) add_all_wide(vb[k], acc_s, acc_c);
        }
    };

    // Adds the super-window at `pos` (held in v) to the running pieces: whole
    // blocks of kSub vectors inside trajectory `cur` take the fast path, a
    // block holding a trajectory end is walked.
    auto process = [&](int4 (&v)[U], int64_t pos) {
#pragma unroll
        for (int h = 0; h < U / kSub; ++h) {
            const int64_t bpos = pos + (int64_t)h * kSub * kWin;
            if (bpos >= ce) break;
            const int64_t bend = (bpos + kSub * kWin < ce) ? bpos + kSub * kWin : ce;
            if (valid && cur_end >= bend) add_block(v + h * kSub);
            else walk(v + h * kSub, bpos, bend);
        }
    };

    for (int64_t pos = cs; pos < ce; pos += kSuper) {
        if (pos != cs) load_super<kVecLoad>(tags, pos, ce, lane, va);
        process(va, pos);
    }
    if (pending) flush();
    if (lane < n_held) store_piece(held_at, held_s, held_c);
}

// Finalize workgroup size: small, so the few thousand trajectories of a pool
// spread over many CUs.
constexpr int kFinT = kFinGroup;

// kMinMax: the workgroup also writes the smallest and largest score key of
// its trajectories (mmin, mmax), the range the wide selection histograms.
template <bool kWinLds, bool kMinMax>
__global__ __launch_bounds__(kFinT) void score_finalize_kernel(
    const int64_t *__restrict__ off, int64_t n, int64_t NT, const int32_t *__restrict__ completion,
    int32_t V, const double *__restrict__ prefix, const double *__restrict__ window, int64_t W,
    int use_prefix, double w_wait, int gamma, int64_t chunk_len, ScoreWorkspace ws,
    double *__restrict__ score, int64_t *__restrict__ gen_sum, int64_t *__restrict__ gen_count,
    uint64_t *__restrict__ mmin, uint64_t *__restrict__ mmax) {
    __shared__ double win_lds[kWinLds ? kWindowLdsMax : 1];
    const bool narrow = (NT >> 11) < ((int64_t)1 << 32);   // token positions below 2^43
    // The trajectory's own loads go first (they do not wait for the window),
    // then the window is staged; every thread reaches the barrier.
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool in = i < n;
    int64_t lo = 0, hi = 0;
    int32_t c = 0;
    double s_pre = 0.0;
    if (in) {
        lo = clamp64(off[i], 0, NT);
        hi = clamp64(off[i + 1], 0, NT);
        c = completion[i];
        if (use_prefix) s_pre = prefix[i];
    }
    const TrajPieces pc = in ? gather_pieces(i, lo, hi, ws.part_sum, ws.part_cnt, ws.carry_sum, ws.carry_cnt,
                                             chunk_len, narrow)
                             : TrajPieces{0, 0};
    if (kWinLds && use_prefix) {
        const int w_n = (int)W;                  // W <= kWindowLdsMax here
#pragma unroll 4
        for (int k = (int)threadIdx.x; k < w_n; k += kFinT) win_lds[k] = window[k];
        __syncthreads();
    }
    if (!kMinMax && !in) return;
    uint64_t key = 0;
    if (in) {
        const TrajScore r = score_from_pieces(pc, c, V, use_prefix != 0, s_pre, kWinLds ? win_lds : window, W,
                                              w_wait, gamma);
        score[i] = r.score;
        if (gen_sum) gen_sum[i] = r.S;
        if (gen_count) gen_count[i] = r.T;
        key = score_key(r.score);
    }
    if constexpr (kMinMax) {
        __shared__ uint64_t wl[kFinT / kWave], wh[kFinT / kWave];
        const uint64_t lo = wave_min_u64(in ? key : ~0ull), hi = wave_max_u64(key);
        if (lane_id() == 0) {
            wl[threadIdx.x / kWave] = lo;
            wh[threadIdx.x / kWave] = hi;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            uint64_t a = ~0ull, b = 0;
            for (int w = 0; w < kFinT / kWave; ++w) {
                a = wl[w] < a ? wl[w] : a;
                b = wh[w] > b ? wh[w] : b;
            }
            mmin[blockIdx.x] = a;
            mmax[blockIdx.x] = b;
        }
    }
}

}  // namespace

size_t score_ws_bytes(int64_t n, int64_t n_tokens) {
    const int64_t ch = score_max_chunks(n_tokens);
    return align256((size_t)n * 8) * 2 + align256((size_t)ch * 8) * 2 + 256;
}

ScoreWorkspace score_ws_carve(void *ws, int64_t n, int64_t n_tokens) {
    const int64_t ch = score_max_chunks(n_tokens);
    char *p = (char *)ws;
    ScoreWorkspace w;
    w.part_sum = (uint64_t *)p;  p += align256((size_t)n * 8);
    w.part_cnt = (int64_t *)p;   p += align256((size_t)n * 8);
    w.carry_sum = (uint64_t *)p; p += align256((size_t)ch * 8);
    w.carry_cnt = (int64_t *)p;
    return w;
}

hipError_t launch_score_reduce(const int32_t *tags, const int64_t *offsets, int64_t n,
                               int64_t n_tokens, int32_t V, const ScoreWorkspace &ws, bool vec_ok,
                               hipStream_t stream, int64_t *chunk_len_out) {
    // One contiguous, equal token range per resident wave: a single balanced
    // round with no tail of late workgroups.
    const int64_t chunk_len = score_chunk_len(n_tokens, resident_waves() / 16 * kReduceWavesPerCU);
    *chunk_len_out = chunk_len;
    const int64_t ch = n_tokens > 0 ? (n_tokens + chunk_len - 1) / chunk_len : 0;
    if (n == 0 || ch == 0) return hipSuccess;
    const unsigned grid = (unsigned)((ch + kWavesPerBlock - 1) / kWavesPerBlock);
    const bool narrow = (int64_t)V < (1 << 24) - 1;
#define PACE_REDUCE(NARROW, VEC)                                                            \
    return launch(kPhaseReduce, score_reduce_kernel<NARROW, VEC>, dim3(grid), dim3(256), stream, \
                  tags, offsets, n, n_tokens, chunk_len, ch, ws.part_sum, ws.part_cnt,         \
                  ws.carry_sum, ws.carry_cnt)
    if (narrow && vec_ok) PACE_REDUCE(true, true);
    if (narrow) PACE_REDUCE(true, false);
    if (vec_ok) PACE_REDUCE(false, true);
    PACE_REDUCE(false, false);
#undef PACE_REDUCE
}

hipError_t launch_score_finalize(const int64_t *offsets, int64_t n, int64_t n_tokens,
                                 const int32_t *completion, int32_t V, const double *prefix,
                                 const double *window, int64_t W, bool use_prefix, double w_wait,
                                 int gamma, int64_t chunk_len, double *score, int64_t *gen_sum,
                                 int64_t *gen_count, const ScoreWorkspace &ws, hipStream_t stream,
                                 uint64_t *mmin, uint64_t *mmax) {
    if (n == 0) return hipSuccess;
    const unsigned grid = (unsigned)((n + kFinT - 1) / kFinT);
    const bool win_lds = use_prefix && W <= kWindowLdsMax;
#define PACE_FIN(WIN, MM)                                                                                    \
    return launch(kPhaseFinalize, score_finalize_kernel<WIN, MM>, dim3(grid), dim3(kFinT), stream, offsets, n, \
                  n_tokens, completion, V, prefix, window, W, use_prefix ? 1 : 0, w_wait, gamma, chunk_len, ws,   \
                  score, gen_sum, gen_count, mmin, mmax)
    if (mmin) {
        if (win_lds) PACE_FIN(true, true);
        PACE_FIN(false, true);
    }
    if (win_lds) PACE_FIN(true, false);
    PACE_FIN(false, false);
#undef PACE_FIN
}

hipError_t launch_score(const int32_t *tags, const int64_t *offsets, int64_t n, int64_t n_tokens,
                        const int32_t *completion, int32_t V, const double *prefix,
                        const double *window, int64_t W, bool use_prefix, double w_wait, int gamma,
                        double *score, int64_t *gen_sum, int64_t *gen_count,
                        const ScoreWorkspace &ws, bool vec_ok, hipStream_t stream) {
    int64_t chunk_len = 0;
    hipError_t e = launch_score_reduce(tags, offsets, n, n_tokens, V, ws, vec_ok, stream, &chunk_len);
    if (e != hipSuccess) return e;
    return launch_score_finalize(offsets, n, n_tokens, completion, V, prefix, window, W, use_prefix,
                                 w_wait, gamma, chunk_len, score, gen_sum, gen_count, ws, stream);
}

}  // namespace pace
