// The streaming admission rule for gfx950 (Sec. 3.1, Algorithm 1): the
// cutoff kappa is the (1 - r_hat)-quantile of a sliding window of recently
// observed scores; the trainer draws candidates in pool order, rejects those
// scoring above kappa and retains the rest until the batch is full.
//
// Two kernels:
//   1. stream_kappa: kappa is the ceil(p * cnt)-th smallest of the cnt window
//      entries, p = 1 - rate (the lower empirical quantile), or +inf with
//      fewer than window_min entries or a rate of 0. Each workgroup ranks
//      kKQ entries against the whole window (one entry per thread) in the
//      total order (score key, position), so exactly one entry has rank
//      k - 1 and exactly one thread writes kappa; spread over the chip, the
//      cnt^2 comparisons cost a few microseconds (about twenty on a single
//      workgroup);
//   2. stream_admit, one workgroup of 1024 threads:
//      a. the draw needs no sequential walk: candidate i is drawn iff fewer
//         than batch_size candidates before it are retained, so one ordered
//         count of the retained flags (block scans over tiles of the pool)
//         gives every candidate's status, the rejected ids in order (i minus
//         the retained before i) and the draw length;
//      b. the drawn scores enter the ring in draw order (only the last `cap`
//         of them can survive), and the ring state is advanced;
//      c. given the offsets (the fused step), the compaction's block partials
//         of the keep flags are written as well.
#include "device_util.hpp"
#include "kernels.hpp"
#include "select_block.hpp"

#pragma clang fp contract(off)

namespace pace {

namespace {

constexpr int kST = 1024;
constexpr int kSNW = kST / kWave;
constexpr int kSItems = 8;
constexpr int64_t kSTile = (int64_t)kST * kSItems;

constexpr int kKQ = 16;    // window entries ranked per workgroup

__global__ __launch_bounds__(kST) void stream_kappa_kernel(const double *__restrict__ ring, int64_t cap,
                                                           const int64_t *__restrict__ state, double rate,
                                                           int64_t window_min, double *__restrict__ kappa_out) {
    static_assert(kStreamWindowMax <= kST, "one window entry per thread");
    __shared__ uint32_t part[kSNW][kKQ / 4];
    const int t = threadIdx.x, lane = lane_id(), wave = t / kWave;
    const int64_t head = clamp64(state[0], 0, cap - 1);
    const int64_t cnt = clamp64(state[1], 0, cap);
    if (!(cnt >= window_min && cnt > 0 && rate > 0.0)) {
        if (blockIdx.x == 0 && t == 0) *kappa_out = __builtin_inf();
        return;
    }
    const int64_t u0 = (int64_t)blockIdx.x * kKQ;
    if (u0 >= cnt) return;                          // the whole workgroup
    // Window entry u (0 = oldest): the cnt most recent entries end just
    // before head.
    auto at = [&](int64_t u) {
        const int64_t x = head - cnt + u;           // in [-cap, cap)
        return x < 0 ? x + cap : x;
    };
    const bool mine = t < cnt;
    const uint64_t ky = score_key(ring[at(mine ? t : cnt - 1)]);
    const uint64_t kq_lane = score_key(ring[at(min(u0 + (lane < kKQ ? lane : 0), cnt - 1))]);
    // Entries before query q in (key, position) order, one bit per thread,
    // packed four queries per word (a wave's count fits 8 bits).
    uint32_t packed[kKQ / 4] = {};
#pragma unroll
    for (int q = 0; q < kKQ; ++q) {
        const uint64_t kq = (uint64_t)readlane_i64((int64_t)kq_lane, q);
        const uint32_t before = (uint32_t)(mine & ((ky < kq) | ((ky == kq) & ((int64_t)t < u0 + q))));
        packed[q / 4] += before << (8 * (q % 4));
    }
#pragma unroll
    for (int w = 0; w < kKQ / 4; ++w) {
        const uint32_t sum = (uint32_t)readlane_i32((int32_t)wave_incl_scan_u32(packed[w]), kWave - 1);
        if (lane == 0) part[wave][w] = sum;
    }
    __syncthreads();
    if (t < kKQ) {
        uint32_t r = 0;
#pragma unroll
        for (int v = 0; v < kSNW; ++v) r += (part[v][t / 4] >> (8 * (t % 4))) & 0xffu;
        const double p = 1.0 - rate;
        int64_t k = (int64_t)ceil(p * (double)cnt);
        if (k < 1) k = 1;
        const int64_t u = u0 + t;
        if (u < cnt && (int64_t)r == k - 1) *kappa_out = ring[at(u)];
    }
}

__device__ __forceinline__ int64_t shfl_xor_i64(int64_t v, int m) {
    const int lo = __shfl_xor((int)(uint32_t)v, m, kWave);
    const int hi = __shfl_xor((int)(uint32_t)((uint64_t)v >> 32), m, kWave);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// kParts: also writes the compaction's block partials of the keep flags
// (kept count, kept tokens, pieces per block of kPieceBlock trajectories,
// lengths from offsets clamped to [0, NT]); a block is two adjacent threads.
template <bool kParts>
__global__ __launch_bounds__(kST) void stream_admit_kernel(
    const double *__restrict__ score, int64_t n, int64_t B,
    double *__restrict__ ring, int64_t cap, int64_t *__restrict__ state, uint8_t *__restrict__ status,
    uint8_t *__restrict__ keep, int32_t *__restrict__ reject_ids, const double *__restrict__ kappa_in,
    int64_t *__restrict__ counts, const int64_t *__restrict__ off, int64_t NT, PieceParts parts, bool vec) {
    static_assert(2 * kSItems == kPieceBlock && kSTile % kPieceBlock == 0, "a block is two threads' items");
    __shared__ uint32_t wsum[kSNW];
    __shared__ int64_t s_state[2];
    const int t = threadIdx.x;
    // The first tile's scores, the cutoff and the ring state are loaded
    // together (a slot past the end reads the last score and is dropped).
    double sc[kSItems];
    int64_t ob[kSItems + 1];                   // clamped offsets of this thread's items (kParts)
    // A wave whose items all lie in the pool reads each thread's run as
    // 16-byte vectors (vec: both arrays 16-byte aligned); element loads,
    // clamped to the pool, otherwise. (One element per load, the lanes 64
    // bytes apart, would leave the single CU bound on address processing.)
    const int wave = __builtin_amdgcn_readfirstlane(t / kWave);
    auto load_tile = [&](int64_t base) {
        const int64_t i0 = base + (int64_t)t * kSItems;
        const bool full = vec && base + (int64_t)(wave + 1) * kWave * kSItems <= n;
        if (full) {
#pragma unroll
            for (int j = 0; j < kSItems / 2; ++j) {
                const double2 v = *reinterpret_cast<const double2 *>(score + i0 + 2 * j);
                sc[2 * j] = v.x;
                sc[2 * j + 1] = v.y;
            }
            if constexpr (kParts) {
#pragma unroll
                for (int j = 0; j < kSItems / 2; ++j) {
                    const longlong2 v = *reinterpret_cast<const longlong2 *>(off + i0 + 2 * j);
                    ob[2 * j] = clamp64(v.x, 0, NT);
                    ob[2 * j + 1] = clamp64(v.y, 0, NT);
                }
                ob[kSItems] = clamp64(off[i0 + kSItems], 0, NT);     // i0 + kSItems <= n
            }
        } else {
#pragma unroll
            for (int q = 0; q < kSItems; ++q) sc[q] = score[min(i0 + q, n - 1)];
            if constexpr (kParts) {
#pragma unroll
                for (int q = 0; q <= kSItems; ++q) ob[q] = clamp64(off[min(i0 + q, n)], 0, NT);
            }
        }
    };
    if (n > 0) load_tile(0);
    if (t == 0) {
        s_state[0] = state[0];
        s_state[1] = state[1];
    }
    const double kappa = *kappa_in;            // written by stream_kappa
    __syncthreads();
    const int64_t head = clamp64(s_state[0], 0, cap - 1);
    const int64_t cnt = clamp64(s_state[1], 0, cap);

    // a. The draw.
    int64_t run_ret = 0, drawn = 0;
    for (int64_t base = 0; base < n; base += kSTile) {
        const int64_t i0 = base + (int64_t)t * kSItems;
        bool in[kSItems], ret[kSItems];
        uint32_t c = 0;
        if (base > 0) load_tile(base);
#pragma unroll
        for (int q = 0; q < kSItems; ++q) {
            in[q] = i0 + q < n;
            ret[q] = in[q] && !(sc[q] > kappa);
            c += ret[q] ? 1u : 0u;
        }
        uint32_t tot;
        const uint32_t before = block_excl_sum_u32<kSNW>(c, tot, wsum);
        int64_t rb = run_ret + before;          // retained before item i0 + q
        uint32_t d = 0;
        uint32_t k_cnt = 0, k_pcs = 0;
        int64_t k_len = 0;
#pragma unroll
        for (int q = 0; q < kSItems; ++q) {
            if (!in[q]) continue;
            const int64_t i = i0 + q;
            const bool is_drawn = rb < B;
            uint8_t st = 2;
            if (is_drawn) {
                st = ret[q] ? 1 : 0;
                if (!ret[q]) reject_ids[i - rb] = (int32_t)i;
                d += 1;
            }
            status[i] = st;
            keep[i] = st == 1 ? 1 : 0;
            rb += ret[q] ? 1 : 0;
            if constexpr (kParts) {
                if (st == 1) {
                    const int64_t len = ob[q + 1] > ob[q] ? ob[q + 1] - ob[q] : 0;
                    k_cnt += 1;
                    k_len += len;
                    k_pcs += (uint32_t)((len + kPieceLen - 1) / kPieceLen);
                }
            }
        }
        if constexpr (kParts) {
            const uint32_t c2 = k_cnt + (uint32_t)__shfl_xor((int)k_cnt, 1, kWave);
            const uint32_t p2 = k_pcs + (uint32_t)__shfl_xor((int)k_pcs, 1, kWave);
            const int64_t l2 = k_len + shfl_xor_i64(k_len, 1);
            const int64_t b0 = base + (int64_t)(t & ~1) * kSItems;     // the block's first trajectory
            if ((t & 1) == 0 && b0 < n) {
                const int64_t blk = b0 / kPieceBlock;
                parts.cnt[blk] = (int32_t)c2;
                parts.len[blk] = l2;
                parts.pcs[blk] = (int32_t)p2;
            }
        }
        uint32_t dtot;
        (void)block_excl_sum_u32<kSNW>(d, dtot, wsum);
        drawn += dtot;
        run_ret += tot;
    }
    const int64_t retained = run_ret < B ? run_ret : B;

    // b. The window takes the drawn scores, oldest first.
    const int64_t first = drawn > cap ? drawn - cap : 0;
    for (int64_t u = first + t; u < drawn; u += kST) ring[(head + u) % cap] = score[u];
    if (t == 0) {
        state[0] = (head + drawn) % cap;
        state[1] = (cnt + drawn < cap) ? cnt + drawn : cap;
        counts[0] = drawn;
        counts[1] = retained;
        counts[2] = drawn - retained;
    }
}

}  // namespace

hipError_t launch_stream_admit(const double *score, int64_t n, double rate, int64_t window_min, int64_t B,
                               double *ring, int64_t cap, int64_t *state, uint8_t *status, uint8_t *keep,
                               int32_t *reject_ids, double *kappa, int64_t *counts, const int64_t *offsets,
                               int64_t n_tokens, const PieceParts &parts, hipStream_t stream) {
    hipError_t e = launch(kPhaseAux, stream_kappa_kernel, dim3((unsigned)((cap + kKQ - 1) / kKQ)), dim3(kST), stream,
                          ring, cap, state, rate, window_min, kappa);
    if (e != hipSuccess) return e;
    const bool with_parts = offsets && parts.cnt;
    const bool vec = ((uintptr_t)score & 15) == 0 && (!with_parts || ((uintptr_t)offsets & 15) == 0);
    if (with_parts)
        return launch(kPhaseSelect, stream_admit_kernel<true>, dim3(1), dim3(kST), stream, score, n, B, ring, cap,
                      state, status, keep, reject_ids, (const double *)kappa, counts, offsets, n_tokens, parts, vec);
    return launch(kPhaseSelect, stream_admit_kernel<false>, dim3(1), dim3(kST), stream, score, n, B, ring, cap,
                  state, status, keep, reject_ids, (const double *)kappa, counts, offsets, n_tokens, parts, vec);
}

}  // namespace pace
