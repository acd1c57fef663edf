// pace_score kernels for gfx950.
//
// Step 1 (score_reduce): every per-token version tag is read exactly once.
// The token array is cut into equal chunks of consecutive tokens, one per
// wave64, sized so that every resident wave gets exactly one (a multiple of
// 256 tokens, at least 2048); a chunk is read as 16-byte vectors, 8 per lane
// in flight, the first batch issued before the trajectory search. (Plain loads on purpose:
// they leave the tags in the last-level cache, where the compaction re-reads
// the kept spans.) Let G(p) be the sum of (tag + 1) over the generated tokens
// of [chunk start, p) (masked tags, -1, add 0) and their count. The wave holds
// 64 trajectory offsets, one per lane, and ends with G at each of them
// (clamped to the chunk); a trajectory's piece in the chunk is then the
// difference of two neighbouring lanes:
//   - a block of 1024 tokens without an offset inside is added per lane;
//   - a block with offsets writes the window-local exclusive prefixes of its
//     four 256-token windows to LDS (one wave scan per window and quantity),
//     and each lane whose offset falls in the block reads its G there, so
//     the cost does not grow with the number of trajectories in the block.
// The piece of a trajectory that starts inside this chunk goes to
// part_{sum,cnt}[trajectory] (exactly one chunk holds each start); the piece
// of the trajectory that straddles the chunk start goes to
// carry_{sum,cnt}[chunk] (at most one per chunk).
// No atomics, no zero-filled workspace, and the combine order is fixed, so
// the integer results are bit-identical run to run.
//
// Step 2 (score_finalize): one thread per trajectory adds its carries, forms
// S_i = c_i T_i - sum(tag) exactly in int64 and evaluates the score of
// Eq. (6)-(9) in binary64 with a fixed operation order (no contraction).
#include <type_traits>

#include "device_util.hpp"
#include "kernels.hpp"
#include "score_math.hpp"

#pragma clang fp contract(off)

namespace pace {

namespace {

constexpr int kVec = 4;                       // tags per lane per window
constexpr int kWin = kWave * kVec;            // 256 tokens per wave window
constexpr int kUnroll = 8;                    // windows per super-window
constexpr int kSub = 4;                       // windows per block of the fast path
constexpr int kWavesPerBlock = 4;
static_assert(kScoreChunkAlign % kWin == 0, "a chunk is whole windows");

// Arithmetic of the reduction, chosen from V (tags are at most V):
//   kPacked  every tag + 1 < 2^15: an element is q = (tag + 1) * 2^9 +
//            [tag != -1], so that a window's 256 elements sum below 2^32 with
//            the count in the low 9 bits; one 32-bit scan gives both prefixes,
//            and a lane's running sums are kept as sum * 2^24 + count in 64
//            bits (one wave reduction for both);
//   kNarrow  every tag + 1 < 2^24: 32-bit window sums, counts separate;
//   kWide    64-bit sums.
enum ReduceMode : int { kPacked = 0, kNarrow = 1, kWideTags = 2 };

// Window-local exclusive prefixes of one window per wave, for the trajectory
// boundaries inside it: sums (with the packed count), and for the other modes
// the counts (at most 255 before a window's last position, so one byte).
template <int kMode>
struct WinPrefix {
    using S = typename std::conditional<kMode == kWideTags, uint64_t, uint32_t>::type;
    S s[kWavesPerBlock][kWin];
    uint8_t c[kWavesPerBlock][kMode == kPacked ? 4 : kWin];
};

__device__ __forceinline__ uint32_t wave_incl_add(uint32_t v) { return wave_incl_scan_u32(v); }
__device__ __forceinline__ uint64_t wave_incl_add(uint64_t v) { return (uint64_t)wave_incl_scan_i64((int64_t)v); }

// The next lane's value (lane 63 gets lane 0's).
__device__ __forceinline__ int64_t from_next_lane(int64_t v) {
    const int a = ((lane_id() + 1) & (kWave - 1)) << 2;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(a, (int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(a, (int)(uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

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

// Packed element: (x + 1) * 2^9 + 1 for a tag x >= 0, 0 for x = -1.
__device__ __forceinline__ uint32_t packed(int x) {
    return ((uint32_t)x << 9) + 513u + (uint32_t)(x >> 31);
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

template <int kMode, bool kVecLoad, int U = kUnroll>
__global__ __launch_bounds__(256) void score_reduce_kernel(
    const int32_t *__restrict__ tags, const int64_t *__restrict__ off, int64_t n, int64_t NT,
    int64_t chunk_len, int64_t n_chunks, uint64_t *__restrict__ part_sum,
    int64_t *__restrict__ part_cnt, uint64_t *__restrict__ carry_sum,
    int64_t *__restrict__ carry_cnt) {
    using PS = typename WinPrefix<kMode>::S;
    __shared__ WinPrefix<kMode> lds;
    const int lane = lane_id();
    const int wv = threadIdx.x / kWave;
    const int64_t chunk = (int64_t)blockIdx.x * kWavesPerBlock + wv;
    if (chunk >= n_chunks) return;
    const int64_t cs = chunk * chunk_len;
    const int64_t ce = (cs + chunk_len < NT) ? cs + chunk_len : NT;
    PS *__restrict__ pre_s = lds.s[wv];
    uint8_t *__restrict__ pre_c = lds.c[wv];

    // The first super-window's loads do not depend on the trajectory search:
    // issue them first so the search latency hides under them.
    constexpr int64_t kSuper = (int64_t)kWin * U;
    int4 va[U];
    load_super<kVecLoad>(tags, cs, ce, lane, va);

    // Boundary window: lane k holds B = offsets[bb + k] clamped to [0, NT]
    // (NT past offsets[n]), the start of trajectory bb + k and the end of
    // trajectory bb + k - 1; the window covers trajectories bb .. bb + 62.
    // First guess: the 64 offsets around the index the chunk would start at
    // if all trajectories were equally long; if the trajectory holding the
    // chunk's first token is not among them, a 64-ary search over all
    // offsets and one more load.
    int64_t bb, B;
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
            bb = base;
            B = (idx <= n) ? clamp64(raw, 0, NT) : NT;
        } else {
            const int64_t s = wave_last_le(off, n, cs);
            bb = s < 0 ? 0 : s;
            const int64_t i2 = bb + lane;
            B = (i2 <= n) ? clamp64(off[i2], 0, NT) : NT;
        }
    }
    // The next boundary window, loaded ahead when the chunk may reach it.
    int64_t nB = NT;
    bool nB_ok = false;
    auto load_next = [&]() {
        const int64_t i2 = bb + (kWave - 1) + lane;
        nB = (i2 <= n) ? clamp64(off[i2], 0, NT) : NT;
        nB_ok = true;
    };
    auto want_next = [&]() { return !nB_ok && bb + (kWave - 1) < n && readlane_i64(B, kWave - 1) < ce; };
    if (want_next()) load_next();

    // G(p): sum of (tag + 1) over generated tokens and their count in
    // [cs, p). Lane k ends with G(clamp(B, cs, ce)), so a trajectory's piece
    // in this chunk is the difference of two neighbouring lanes.
    uint64_t Gs = 0;
    int64_t Gc = 0;
    uint64_t Ws = 0;             // G at the current window's start, less what acc_* still hold
    int64_t Wc = 0;
    uint64_t acc_s = 0;          // per-lane sums of windows without a boundary (kPacked: sum * 2^24 + count)
    uint32_t acc_c = 0;
    bool dirty = false;
    auto sync = [&]() {
        if (dirty) {
            if constexpr (kMode == kPacked) {
                const uint64_t t = wave_sum_u64(acc_s);
                Ws += t >> 24;
                Wc += (int64_t)(t & 0xffffffull);
            } else {
                Ws += wave_sum_u64(acc_s);
                Wc += (int64_t)wave_sum_u64((uint64_t)acc_c);
            }
            acc_s = 0;
            acc_c = 0;
            dirty = false;
        }
    };
    // Adds nv vectors (a window or a block without boundaries) per lane.
    auto add_vecs = [&](const int4 *vb, int nv) {
        if constexpr (kMode == kWideTags) {
            for (int k = 0; k < nv; ++k) add_all_wide(vb[k], acc_s, acc_c);
        } else {
            uint32_t s32 = 0, c32 = 0;             // below 2^28 for up to 16 tags per lane
            for (int k = 0; k < nv; ++k) add_all(vb[k], s32, c32);
            if constexpr (kMode == kPacked) {
                acc_s += ((uint64_t)s32 << 24) + c32;
            } else {
                acc_s += s32;
                acc_c += c32;
            }
        }
        dirty = true;
    };
    // Smallest boundary still ahead (wave-uniform).
    int64_t next_b;
    {
        const uint64_t m = ballot(B > cs);
        next_b = m ? readlane_i64(B, __ffsll((long long)m) - 1) : INT64_MAX;
    }

    // Pieces of the window's trajectories (lane k: trajectory bb + k):
    // at = trajectory for a piece that starts in this chunk, -1 for the piece
    // that straddles the chunk start, -2 for none. The first window finished
    // mid-chunk waits in held_* and is stored after the last super-window (a
    // store in mid-stream would hold up the next loads: one counter covers
    // loads and stores).
    int64_t held_at = -2, held_c = 0;
    uint64_t held_s = 0;
    auto store_piece = [&](int64_t at, uint64_t ps, int64_t pc) {
        if (at >= 0) {
            part_sum[at] = ps;
            part_cnt[at] = pc;
        } else if (at == -1) {
            carry_sum[chunk] = ps;
            carry_cnt[chunk] = pc;
        }
    };
    auto pieces = [&](int64_t &at, uint64_t &ps, int64_t &pc) {
        const int64_t B1 = from_next_lane(B);
        ps = (uint64_t)from_next_lane((int64_t)Gs) - Gs;
        pc = from_next_lane(Gc) - Gc;
        const int64_t j = bb + lane;
        const bool has = lane < kWave - 1 && j < n && B1 > B && B < ce && B1 > cs;
        at = !has ? -2 : (B >= cs ? j : -1);
    };
    // Every boundary of the window lies before the current window's end:
    // keep its pieces and move to the next window.
    auto next_window = [&]() {
        int64_t at, pc;
        uint64_t ps;
        pieces(at, ps, pc);
        if (held_at != -2) store_piece(held_at, held_s, held_c);
        held_at = at;
        held_s = ps;
        held_c = pc;
        const uint64_t g_s = (uint64_t)readlane_i64((int64_t)Gs, kWave - 1);
        const int64_t g_c = readlane_i64(Gc, kWave - 1);
        if (!nB_ok) load_next();
        bb += kWave - 1;
        B = nB;
        nB_ok = false;
        Gs = lane == 0 ? g_s : 0ull;
        Gc = lane == 0 ? g_c : 0;
    };

    // A window [w, w_end) holding boundaries: its exclusive prefixes into
    // LDS, then every lane whose boundary falls in the window reads its G.
    auto event_window = [&](const int4 &v, int64_t w, int64_t w_end) {
        sync();
        uint64_t tot_s;
        int64_t tot_c;
        PS *ds = pre_s + lane * kVec;
        if constexpr (kMode == kPacked) {
            const uint32_t q0 = packed(v.x), q1 = packed(v.y), q2 = packed(v.z), q3 = packed(v.w);
            const uint32_t p1 = q0, p2 = p1 + q1, p3 = p2 + q2, p4 = p3 + q3;
            const uint32_t is = wave_incl_scan_u32(p4);
            const uint32_t es = is - p4;
            ds[0] = es;
            ds[1] = es + p1;
            ds[2] = es + p2;
            ds[3] = es + p3;
            const uint32_t t = (uint32_t)__builtin_amdgcn_readlane((int)is, kWave - 1);
            tot_s = t >> 9;
            tot_c = t & 511u;
        } else {
            const uint32_t u0 = (uint32_t)v.x + 1u, u1 = (uint32_t)v.y + 1u;
            const uint32_t u2 = (uint32_t)v.z + 1u, u3 = (uint32_t)v.w + 1u;
            const PS p1 = (PS)u0, p2 = p1 + (PS)u1, p3 = p2 + (PS)u2, p4 = p3 + (PS)u3;
            const uint32_t c1 = (u0 != 0u), c2 = c1 + (u1 != 0u), c3 = c2 + (u2 != 0u), c4 = c3 + (u3 != 0u);
            const PS is = wave_incl_add(p4);
            const uint32_t ic = wave_incl_scan_u32(c4);
            const PS es = is - p4;
            const uint32_t ec = ic - c4;
            ds[0] = es;
            ds[1] = es + p1;
            ds[2] = es + p2;
            ds[3] = es + p3;
            *reinterpret_cast<uint32_t *>(pre_c + lane * kVec) =
                ec | ((ec + c1) << 8) | ((ec + c2) << 16) | ((ec + c3) << 24);
            if constexpr (kMode == kNarrow) {
                tot_s = (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)is, kWave - 1);
            } else {
                tot_s = (uint64_t)readlane_i64((int64_t)is, kWave - 1);
            }
            tot_c = (int64_t)(uint32_t)__builtin_amdgcn_readlane((int)ic, kWave - 1);
        }
        while (true) {
            if (B >= w && B < w_end) {
                const int q = (int)(B - w);
                if constexpr (kMode == kPacked) {
                    const uint32_t p = (uint32_t)pre_s[q];
                    Gs = Ws + (p >> 9);
                    Gc = Wc + (int64_t)(p & 511u);
                } else {
                    Gs = Ws + (uint64_t)pre_s[q];
                    Gc = Wc + (int64_t)pre_c[q];
                }
            }
            const uint64_t m = ballot(B >= w_end);
            if (m) {
                next_b = readlane_i64(B, __ffsll((long long)m) - 1);
                break;
            }
            if (bb + (kWave - 1) >= n) {          // no trajectory after this window
                next_b = INT64_MAX;
                break;
            }
            next_window();
        }
        Ws += tot_s;
        Wc += tot_c;
    };

    // Adds block h of the super-window in v (kSub windows from bpos): a block
    // without boundaries is added per lane; in a block with boundaries each
    // window without one is added per lane, the others go to event_window.
    auto process_block = [&](int4 (&v)[U], int64_t bpos, int h) {
        if (bpos >= ce) return;
        const int64_t bend = (bpos + kSub * kWin < ce) ? bpos + kSub * kWin : ce;
        if (next_b >= bend) {
            add_vecs(v + h * kSub, kSub);
            return;
        }
#pragma unroll
        for (int k = 0; k < kSub; ++k) {
            const int64_t w = bpos + (int64_t)k * kWin;
            if (w >= ce) break;
            const int64_t w_end = (w + kWin < ce) ? w + kWin : ce;
            if (next_b >= w_end) add_vecs(v + h * kSub + k, 1);
            else event_window(v[h * kSub + k], w, w_end);
        }
    };

    auto load_half = [&](int64_t p, int half) {
#pragma unroll
        for (int k = 0; k < kSub; ++k) {
            const int64_t q = p + (int64_t)k * kWin + (int64_t)lane * kVec;
            int4 &x = va[half * kSub + k];
            if (kVecLoad && q + kVec <= ce) {
                x = *reinterpret_cast<const int4 *>(tags + q);
            } else {
                x = make_int4(-1, -1, -1, -1);
                if (q < ce) x.x = tags[q];
                if (q + 1 < ce) x.y = tags[q + 1];
                if (q + 2 < ce) x.z = tags[q + 2];
                if (q + 3 < ce) x.w = tags[q + 3];
            }
        }
    };
    // Each half of the next super-window is loaded as soon as the same half
    // of this one has been added, so loads stay queued while the other half
    // is processed.
    for (int64_t pos = cs; pos < ce; pos += kSuper) {
        process_block(va, pos, 0);
        if (pos + kSuper < ce) {
            if (want_next()) load_next();
            load_half(pos + kSuper, 0);
        }
        process_block(va, pos + kSub * kWin, 1);
        if (pos + kSuper + kSub * kWin < ce) load_half(pos + kSuper + kSub * kWin, 1);
    }
    sync();
    if (B >= ce) {
        Gs = Ws;
        Gc = Wc;
    }
    int64_t at, pc;
    uint64_t ps;
    pieces(at, ps, pc);
    store_piece(at, ps, pc);
    store_piece(held_at, held_s, held_c);
}

// Finalize workgroup size: small, so the few thousand trajectories of a pool
// spread over many CUs.
constexpr int kFinT = kFinGroup;

// kMinMax: the workgroup also writes the smallest and largest score key of
// its trajectories (mmin, mmax), the range the wide selection histograms;
// workgroup 0 clears that selection's level-0 histogram (hist0).
template <bool kWinLds, bool kMinMax>
__global__ __launch_bounds__(kFinT) void score_finalize_kernel(
    const int64_t *__restrict__ off, int64_t n, int64_t NT, const int32_t *__restrict__ completion,
    int32_t V, const double *__restrict__ prefix, const double *__restrict__ window, int64_t W,
    int use_prefix, double w_wait, int gamma, int64_t chunk_len, ScoreWorkspace ws,
    double *__restrict__ score, int64_t *__restrict__ gen_sum, int64_t *__restrict__ gen_count,
    uint64_t *__restrict__ mmin, uint64_t *__restrict__ mmax, uint32_t *__restrict__ hist0) {
    __shared__ double win_lds[kWinLds ? kWindowLdsMax : 1];
    const bool narrow = (NT >> 8) < ((int64_t)1 << 32);    // token positions below 2^40
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
        if (blockIdx.x == 0)
            for (int b = threadIdx.x; b < (1 << kCutBits); b += kFinT) hist0[b] = 0u;
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
    // Tags are at most V (a precondition): tag + 1 <= V + 1.
    const int mode = (int64_t)V < (1 << 15) - 1 ? kPacked : ((int64_t)V < (1 << 24) - 1 ? kNarrow : kWideTags);
#define PACE_REDUCE(MODE, VEC)                                                              \
    return launch(kPhaseReduce, score_reduce_kernel<MODE, VEC>, dim3(grid), dim3(256), stream, \
                  tags, offsets, n, n_tokens, chunk_len, ch, ws.part_sum, ws.part_cnt,         \
                  ws.carry_sum, ws.carry_cnt)
    if (mode == kPacked && vec_ok) PACE_REDUCE(kPacked, true);
    if (mode == kPacked) PACE_REDUCE(kPacked, false);
    if (mode == kNarrow && vec_ok) PACE_REDUCE(kNarrow, true);
    if (mode == kNarrow) PACE_REDUCE(kNarrow, false);
    if (vec_ok) PACE_REDUCE(kWideTags, true);
    PACE_REDUCE(kWideTags, false);
#undef PACE_REDUCE
}

hipError_t launch_score_finalize(const int64_t *offsets, int64_t n, int64_t n_tokens,
                                 const int32_t *completion, int32_t V, const double *prefix,
                                 const double *window, int64_t W, bool use_prefix, double w_wait,
                                 int gamma, int64_t chunk_len, double *score, int64_t *gen_sum,
                                 int64_t *gen_count, const ScoreWorkspace &ws, hipStream_t stream,
                                 uint64_t *mmin, uint64_t *mmax, uint32_t *hist0) {
    if (n == 0) return hipSuccess;
    const unsigned grid = (unsigned)((n + kFinT - 1) / kFinT);
    const bool win_lds = use_prefix && W <= kWindowLdsMax;
#define PACE_FIN(WIN, MM)                                                                                    \
    return launch(kPhaseFinalize, score_finalize_kernel<WIN, MM>, dim3(grid), dim3(kFinT), stream, offsets, n, \
                  n_tokens, completion, V, prefix, window, W, use_prefix ? 1 : 0, w_wait, gamma, chunk_len, ws,   \
                  score, gen_sum, gen_count, mmin, mmax, hist0)
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
