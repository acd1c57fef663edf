// pace_select kernel for gfx950: reject exactly `budget` trajectories, the
// first ones in the order (score descending, id ascending) -- the quantile
// rejection rule of Sec. 3.1 taken over the current pool with an exact count.
//
// One workgroup of 1024 threads (16 waves). Each score becomes a 64-bit key
// whose unsigned order is the score order (sign-magnitude flip; -0 -> +0).
// Pools of up to 16384 trajectories keep their keys in registers and use the
// adaptive radix selection of select_block.hpp. Larger pools use the strided
// kernel below: an MSB-first radix select with 8-bit digits finds the
// budget-th largest key K (each pass histograms the digit of the keys still
// tied with the prefix found so far; a 256-bin suffix scan over four waves
// picks the bin that holds the cut; the search stops early when the cut falls
// on a bin boundary). Keys above K are rejected; among keys equal to K the
// lowest ids are rejected, found with a block-wide ordered count (ballot +
// popcount per wave). Rejected ids are written in ascending order by a second
// ordered count.
#include "device_util.hpp"
#include "kernels.hpp"
#include "group_math.hpp"
#include "select_block.hpp"

namespace pace {

namespace {

constexpr int kT = kSelectThreads;
constexpr int kNW = kT / kWave;   // 16 waves


// Exclusive count of `f` over the block in thread order; *total = block sum.
__device__ __forceinline__ uint32_t block_excl_count(bool f, uint32_t &total, uint32_t *wsum) {
    const uint64_t m = ballot(f);
    const uint32_t in_wave = (uint32_t)__popcll(m & lanes_below());
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) wsum[w] = (uint32_t)__popcll(m);
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < kNW; ++k) {
        const uint32_t x = wsum[k];
        tot += x;
        before += (k < w) ? x : 0u;
    }
    __syncthreads();
    total = tot;
    return before + in_wave;
}

// Strided layout, any n < 2^31 when kItems == 0 (keys staged in the
// workspace). Used for pools larger than the register-resident kernel holds.
template <int kItems>
__global__ __launch_bounds__(kT) void select_strided_kernel(const double *__restrict__ score, int64_t n,
                                                    int64_t budget, uint8_t *__restrict__ keep,
                                                    int32_t *__restrict__ reject_ids,
                                                    uint64_t *__restrict__ wkeys) {
    const int tid = threadIdx.x;
    const int64_t n_items = kItems ? kItems : (n + kT - 1) / kT;
    uint64_t kr[kItems ? kItems : 1];

    __shared__ uint32_t hist[256];
    __shared__ uint32_t wsum[kNW];
    __shared__ uint32_t sel_digit, sel_before, sel_cnt;

    // Load scores as keys.
    if (kItems) {
#pragma unroll
        for (int it = 0; it < (kItems ? kItems : 1); ++it) {
            const int64_t i = (int64_t)it * kT + tid;
            kr[it] = (i < n) ? score_key(score[i]) : 0ull;
        }
    } else {
        for (int64_t it = 0; it < n_items; ++it) {
            const int64_t i = it * kT + tid;
            if (i < n) wkeys[i] = score_key(score[i]);
        }
    }
    auto key_at = [&](int64_t it) -> uint64_t {
        if (kItems) return kr[it];
        return wkeys[it * kT + tid];
    };

    // Cut: mode 0 rejects nothing (budget 0), 1 everything (budget n),
    // 2 every key >= kcut (the cut is a digit-bin boundary), 3 every key > kcut
    // plus the first need_tie ids whose key equals kcut.
    int mode = (budget == 0) ? 0 : (budget >= n ? 1 : 3);
    uint64_t kcut = 0;
    int64_t need_tie = 0;
    if (mode == 3) {
        uint64_t prefix = 0, mask = 0;
        int64_t need = budget;
        for (int shift = 56; shift >= 0; shift -= 8) {
            if (tid < 256) hist[tid] = 0u;
            __syncthreads();
#pragma unroll
            for (int64_t it = 0; it < (kItems ? kItems : n_items); ++it) {
                const int64_t i = it * kT + tid;
                if (i < n) {
                    const uint64_t k = key_at(it);
                    if (((k ^ prefix) & mask) == 0ull) atomicAdd(&hist[(k >> shift) & 255u], 1u);
                }
            }
            __syncthreads();
            // Suffix sums over digits 255..0: thread t holds digit 255 - t.
            uint32_t h = 0, inc = 0;
            if (tid < 256) {
                h = hist[255 - tid];
                inc = wave_incl_scan_u32(h);
                if (lane_id() == kWave - 1) wsum[tid / kWave] = inc;
            }
            __syncthreads();
            if (tid < 256) {
                for (int w = 0; w < tid / kWave; ++w) inc += wsum[w];
                const uint32_t before = inc - h;          // keys with a larger digit
                if ((int64_t)before < need && (int64_t)inc >= need) {
                    sel_digit = 255u - (uint32_t)tid;
                    sel_before = before;
                    sel_cnt = h;
                }
            }
            __syncthreads();
            need -= (int64_t)sel_before;
            prefix |= (uint64_t)sel_digit << shift;
            mask |= 0xFFull << shift;
            if (need == (int64_t)sel_cnt) {   // the whole bin is rejected
                mode = 2;                     // prefix has zero low bits
                break;
            }
        }
        kcut = prefix;
        if (mode == 3) need_tie = need;
    }

    // Classify in id order and emit keep flags and ascending reject ids.
    int64_t tie_base = 0, rej_base = 0;
#pragma unroll
    for (int64_t it = 0; it < n_items; ++it) {
        const int64_t i = it * kT + tid;
        const bool in = i < n;
        const uint64_t k = in ? key_at(it) : 0ull;
        bool rej;
        if (mode == 3) {
            const bool eq = in && (k == kcut);
            uint32_t tot;
            const uint32_t r = block_excl_count(eq, tot, wsum);
            rej = in && ((k > kcut) || (eq && tie_base + (int64_t)r < need_tie));
            tie_base += tot;
        } else {
            rej = in && (mode == 1 || (mode == 2 && k >= kcut));
        }
        uint32_t tot2;
        const uint32_t pos = block_excl_count(rej, tot2, wsum);
        if (in) {
            keep[i] = rej ? 0 : 1;
            if (rej && rej_base + (int64_t)pos < budget) reject_ids[rej_base + pos] = (int32_t)i;
        }
        rej_base += tot2;
    }
}


// Register-resident selection for n <= 1024*kItems: thread t holds
// trajectories [t*kItems, (t+1)*kItems) (see select_block.hpp), then one
// ordered count places the rejected ids in ascending order.
template <int kItems>
__global__ __launch_bounds__(kT) void select_reg_kernel(const double *__restrict__ score, int64_t n,
                                                        int64_t budget, uint8_t *__restrict__ keep,
                                                        int32_t *__restrict__ reject_ids) {
    __shared__ SelectSmem sm;
    const int64_t base = (int64_t)threadIdx.x * kItems;
    uint64_t k[kItems];
#pragma unroll
    for (int q = 0; q < kItems; ++q) k[q] = score_key((base + q < n) ? score[base + q] : 0.0);
    select_smem_init(sm);
    bool rej[kItems];
    select_block<kItems>(k, base, n, budget, rej, sm);
    uint32_t nrej = 0;
#pragma unroll
    for (int q = 0; q < kItems; ++q) nrej += rej[q] ? 1u : 0u;
    uint32_t tot;
    uint32_t pos = sel_block_excl_scan(nrej, tot, sm.wsum);
#pragma unroll
    for (int q = 0; q < kItems; ++q) {
        const int64_t i = base + q;
        if (i < n) {
            keep[i] = rej[q] ? 0 : 1;
            if (rej[q]) {
                if ((int64_t)pos < budget) reject_ids[pos] = (int32_t)i;
                ++pos;
            }
        }
    }
}


// ---- rank by counting (pools of up to kRankMaxN trajectories) -------------
// rank_i = #{j : key_j > key_i} + #{j < i : key_j == key_i} is the position of
// trajectory i in the order (score desc, id asc); it is rejected iff
// rank_i < budget. Every workgroup (1024 threads) ranks the kRankQ
// trajectories of one block. A thread holds kKeys keys (j = t, t + 1024, ...)
// in registers and tests each against all kRankQ targets, whose keys every
// lane reads alike. Where all ids of a wave's key slot lie below (above) the
// targets' ids, the id tie-break is a fixed direction and one 64-bit compare
// decides; in the one slot that shares the targets' group, (key, id) is
// compared as the 96-bit word (key, 2^32 - 1 - id) by a borrow chain. No LDS
// traffic per pair; the n^2 comparisons spread over the whole device with no
// dependent rounds.
constexpr int kRankT = 1024;
constexpr int kRankMaxKeys = (int)((kRankMaxN + kRankT - 1) / kRankT);

static_assert(kRankQ == kPieceBlock, "a rank workgroup covers one partials block");

struct RankKey {
    uint32_t lo, hi, id;   // key bits 0..31, 32..63 and 2^32 - 1 - id
};

// c + 1 if (key, id) of b precedes that of a in the order (score desc, id
// asc), else c: the borrow out of a - b over the three words, added to c.
// Written as the carry chain itself (the compiler expands the equivalent C
// into compares and mask logic, four times the instructions). Each VALU that
// reads the carry a previous VALU wrote is two wait states behind it.
__device__ __forceinline__ uint32_t rank_add_beats(uint32_t c, const RankKey &a, const RankKey &b) {
    uint32_t d;
    asm("v_sub_co_u32_e32 %1, vcc, %2, %5\n\t"
        "s_nop 1\n\t"
        "v_subb_co_u32_e32 %1, vcc, %3, %6, vcc\n\t"
        "s_nop 1\n\t"
        "v_subb_co_u32_e32 %1, vcc, %4, %7, vcc\n\t"
        "s_nop 1\n\t"
        "v_addc_co_u32_e32 %0, vcc, 0, %0, vcc"
        : "+v"(c), "=&v"(d)
        : "v"(a.id), "v"(a.lo), "v"(a.hi), "v"(b.id), "v"(b.lo), "v"(b.hi)
        : "vcc");
    return c;
}

// Ranks the kRankQ targets i0 .. i0 + kRankQ - 1 of this workgroup against
// all n keys and writes their keep flags (and, with parts.cnt, the block's
// partials). v[u]: the score of item t + u * kRankT; kq_lane: in lanes
// q < kRankQ of every wave, the key of target i0 + q; span: in threads
// t < kRankQ, the clamped span length of target i0 + t.
template <int kKeys>
__device__ __forceinline__ void rank_block(const double (&v)[kKeys], uint64_t kq_lane, int64_t i0, int64_t n,
                                           int64_t budget, uint8_t *__restrict__ keep, int64_t span,
                                           const PieceParts &parts, uint32_t (*part)[kRankQ]) {
    const int t = threadIdx.x;
    // Padding keys are 0: below every target key (the smallest key of a
    // number is that of -inf, above 0), so they never count.
    uint64_t kj[kKeys];
#pragma unroll
    for (int u = 0; u < kKeys; ++u) {
        const int64_t j = t + (int64_t)u * kRankT;
        kj[u] = j < n ? score_key(v[u]) : 0ull;
    }
    uint64_t kq[kRankQ], kq_m1[kRankQ];
#pragma unroll
    for (int q = 0; q < kRankQ; ++q) {
        kq[q] = (uint64_t)readlane_i64((int64_t)kq_lane, q);
        kq_m1[q] = kq[q] - 1;
    }
    // Key slot u of this wave holds ids [64 g, 64 g + 64), g = wave + 16 u;
    // the targets all lie in group i0 / 64. For a slot in a lower group every
    // id is below every target's, so j beats q iff key_j >= key_q, that is
    // key_j > key_q - 1; in a higher group iff key_j > key_q. Only the slot
    // of the targets' own group compares (key, id) in full.
    const int64_t g_t = i0 / kWave;
    const int wave = __builtin_amdgcn_readfirstlane(t / kWave);   // uniform: keeps the tests scalar
    uint32_t cnt[kRankQ];
#pragma unroll
    for (int q = 0; q < kRankQ; ++q) cnt[q] = 0;
#pragma unroll
    for (int u = 0; u < kKeys; ++u) {
        const int64_t g = wave + (int64_t)u * (kRankT / kWave);
        if (g < g_t) {
#pragma unroll
            for (int q = 0; q < kRankQ; ++q) cnt[q] += kj[u] > kq_m1[q] ? 1u : 0u;
        } else if (g > g_t) {
#pragma unroll
            for (int q = 0; q < kRankQ; ++q) cnt[q] += kj[u] > kq[q] ? 1u : 0u;
        } else {
            const int64_t j = t + (int64_t)u * kRankT;
            const RankKey b = j < n ? RankKey{(uint32_t)kj[u], (uint32_t)(kj[u] >> 32), ~(uint32_t)j}
                                    : RankKey{0u, 0u, 0u};
#pragma unroll
            for (int q = 0; q < kRankQ; ++q) {
                const RankKey a{(uint32_t)kq[q], (uint32_t)(kq[q] >> 32), ~(uint32_t)(i0 + q)};
                cnt[q] = rank_add_beats(cnt[q], a, b);
            }
        }
    }
    // Wave sums, three counts to a word (a wave adds at most 64 * kKeys <= 512
    // per target: 10 bits), then the 16 waves' sums through LDS.
    static_assert(kWave * kRankMaxKeys < 1024, "packed wave counts fit 10 bits");
#pragma unroll
    for (int q0 = 0; q0 < kRankQ; q0 += 3) {
        uint32_t w = cnt[q0];
        if (q0 + 1 < kRankQ) w |= cnt[q0 + 1] << 10;
        if (q0 + 2 < kRankQ) w |= cnt[q0 + 2] << 20;
        w = wave_incl_scan_u32(w);
        if (lane_id() == kWave - 1) {
            part[t / kWave][q0] = w & 1023u;
            if (q0 + 1 < kRankQ) part[t / kWave][q0 + 1] = (w >> 10) & 1023u;
            if (q0 + 2 < kRankQ) part[t / kWave][q0 + 2] = w >> 20;
        }
    }
    __syncthreads();
    if (t < kWave) {   // wave 0; lanes below kRankQ own the targets
        const int64_t ii = i0 + t;
        bool kept = false;
        if (t < kRankQ && ii < n) {
            uint32_t r = 0;
#pragma unroll
            for (int k = 0; k < kRankT / kWave; ++k) r += part[k][t];
            kept = (int64_t)r >= budget;
            keep[ii] = kept ? 1 : 0;
        }
        if (parts.cnt) {
            const int64_t len = kept ? span : 0;
            const uint32_t c = (uint32_t)__popcll(ballot(kept));
            const int64_t l = wave_sum_i64(len);
            const int64_t pc = wave_sum_i64((len + kPieceLen - 1) / kPieceLen);
            if (t == 0) {
                parts.cnt[blockIdx.x] = (int32_t)c;
                parts.len[blockIdx.x] = l;
                parts.pcs[blockIdx.x] = (int32_t)pc;
            }
        }
    }
}


template <int kKeys>
__global__ __launch_bounds__(kRankT) void rank_kernel(const double *__restrict__ score, int64_t n,
                                                     int64_t budget, uint8_t *__restrict__ keep,
                                                     const int64_t *__restrict__ off, int64_t NT,
                                                     PieceParts parts) {
    __shared__ uint32_t part[kRankT / kWave][kRankQ];
    const int t = threadIdx.x;
    const int64_t i0 = (int64_t)blockIdx.x * kRankQ;
    // All loads first: this thread's keys, the targets, the block's spans.
    double v[kKeys];
#pragma unroll
    for (int u = 0; u < kKeys; ++u) {
        const int64_t j = t + (int64_t)u * kRankT;
        v[u] = j < n ? score[j] : 0.0;
    }
    // Lane q of every wave loads target q; its key is formed in the vector
    // unit and read out to scalars (a scalar-side conversion branches on
    // every target).
    const int lane = lane_id();
    const double vq = lane < kRankQ && i0 + lane < n ? score[i0 + lane] : 0.0;
    int64_t span = 0;
    if (parts.cnt && t < kRankQ && i0 + t < n) {
        const int64_t lo = clamp64(off[i0 + t], 0, NT), hi = clamp64(off[i0 + t + 1], 0, NT);
        span = hi > lo ? hi - lo : 0;
    }
    rank_block<kKeys>(v, score_key(vq), i0, n, budget, keep, span, parts, part);
}

// Prompt groups (at most kRankMaxN) in the group filter step: every
// workgroup forms all ng group means from the trajectory scores (group_mean,
// the arithmetic of pace_group_score) and ranks its kRankQ target groups
// against them, writing the targets' group scores and keep flags. Forming
// the means in every workgroup costs ng / kRankQ times the loads of one pass
// over the scores, and saves the group scores' launch.
template <int kKeys>
__global__ __launch_bounds__(kRankT) void group_rank_kernel(const double *__restrict__ score, int64_t n,
                                                           const int64_t *__restrict__ go, int64_t ng,
                                                           int64_t budget, double *__restrict__ group_score,
                                                           uint8_t *__restrict__ group_keep) {
    __shared__ uint32_t part[kRankT / kWave][kRankQ];
    __shared__ uint64_t s_key[kRankQ];
    const int t = threadIdx.x;
    const int64_t i0 = (int64_t)blockIdx.x * kRankQ;
    double v[kKeys];
#pragma unroll
    for (int u = 0; u < kKeys; ++u) {
        const int64_t g = t + (int64_t)u * kRankT;
        v[u] = 0.0;
        if (g < ng) {
            v[u] = group_mean(score, n, go, g);
            if (g >= i0 && g < i0 + kRankQ) {   // this workgroup's targets
                group_score[g] = v[u];
                s_key[g - i0] = score_key(v[u]);
            }
        }
    }
    __syncthreads();
    const int lane = lane_id();
    const uint64_t kq_lane = (lane < kRankQ && i0 + lane < ng) ? s_key[lane] : 0ull;
    rank_block<kKeys>(v, kq_lane, i0, ng, budget, group_keep, 0, PieceParts{}, part);
}

// Rejected ids in ascending order from the keep flags (n <= 1024*kItems).
template <int kItems>
__global__ __launch_bounds__(kT) void emit_rejects_kernel(const uint8_t *__restrict__ keep, int64_t n,
                                                          int64_t budget, int32_t *__restrict__ reject_ids) {
    __shared__ uint32_t wsum[kNW];
    const int64_t base = (int64_t)threadIdx.x * kItems;
    bool rej[kItems];
    uint32_t c = 0;
#pragma unroll
    for (int q = 0; q < kItems; ++q) {
        rej[q] = base + q < n && keep[base + q] == 0;
        c += rej[q] ? 1u : 0u;
    }
    uint32_t tot;
    uint32_t pos = block_excl_sum_u32<kNW>(c, tot, wsum);
#pragma unroll
    for (int q = 0; q < kItems; ++q) {
        if (rej[q]) {
            if ((int64_t)pos < budget) reject_ids[pos] = (int32_t)(base + q);
            ++pos;
        }
    }
}

}  // namespace

size_t select_ws_bytes(int64_t n) {
    const size_t strided = (n > (int64_t)kT * kSelectMaxItems) ? align256((size_t)n * 8) : 256;
    const size_t wide = wide_select_ws_bytes(n);
    return strided > wide ? strided : wide;
}

hipError_t launch_rank(const double *score, int64_t n, int64_t budget, uint8_t *keep,
                       const int64_t *offsets, int64_t n_tokens, const PieceParts &parts,
                       hipStream_t stream) {
    if (n == 0) return hipSuccess;
    if (n > kRankMaxN) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((n + kRankQ - 1) / kRankQ));
#define PACE_RANK(K) \
    return launch(kPhaseSelect, rank_kernel<K>, grid, dim3(kRankT), stream, score, n, budget, keep, offsets, \
                  n_tokens, parts)
    if (n <= kRankT) PACE_RANK(1);
    if (n <= 2 * kRankT) PACE_RANK(2);
    if (n <= 4 * kRankT) PACE_RANK(4);
    PACE_RANK(8);
#undef PACE_RANK
}

hipError_t launch_group_rank(const double *score, int64_t n, const int64_t *group_offsets, int64_t ng,
                             int64_t budget, double *group_score, uint8_t *group_keep, hipStream_t stream) {
    if (ng == 0) return hipSuccess;
    if (ng > kRankMaxN) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((ng + kRankQ - 1) / kRankQ));
#define PACE_GROUP_RANK(K) \
    return launch(kPhaseSelect, group_rank_kernel<K>, grid, dim3(kRankT), stream, score, n, group_offsets, ng, \
                  budget, group_score, group_keep)
    if (ng <= kRankT) PACE_GROUP_RANK(1);
    if (ng <= 2 * kRankT) PACE_GROUP_RANK(2);
    if (ng <= 4 * kRankT) PACE_GROUP_RANK(4);
    PACE_GROUP_RANK(8);
#undef PACE_GROUP_RANK
}

hipError_t launch_select(const double *score, int64_t n, int64_t budget, uint8_t *keep,
                         int32_t *reject_ids, void *ws, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const int64_t items = (n + kT - 1) / kT;
    if (n <= kRankMaxN) {
        hipError_t e = launch_rank(score, n, budget, keep, nullptr, 0, PieceParts{nullptr, nullptr, nullptr},
                                   stream);
        if (e != hipSuccess || budget == 0) return e;
        if (items <= 1)
            emit_rejects_kernel<1><<<1, kT, 0, stream>>>(keep, n, budget, reject_ids);
        else if (items <= 2)
            emit_rejects_kernel<2><<<1, kT, 0, stream>>>(keep, n, budget, reject_ids);
        else if (items <= 4)
            emit_rejects_kernel<4><<<1, kT, 0, stream>>>(keep, n, budget, reject_ids);
        else
            emit_rejects_kernel<8><<<1, kT, 0, stream>>>(keep, n, budget, reject_ids);
        return hipGetLastError();
    }
    if (n <= kWideMaxN) {
        // the cut over the chip, keep flags, then the rejected ids in order
        const WideWs w = wide_ws_carve(ws, n);
        hipError_t e = launch_key_minmax(score, n, w, stream);
        if (e == hipSuccess) e = launch_wide_cut(score, n, budget, w, stream);
        if (e == hipSuccess) e = launch_classify(score, nullptr, n, 0, budget, w, keep, w.parts, stream);
        if (e == hipSuccess) e = launch_emit_rejects_wide(keep, n, w.parts.cnt, budget, reject_ids, stream);
        return e;
    }
    if (items <= 16)
        return launch(kPhaseSelect, select_reg_kernel<16>, dim3(1), dim3(kT), stream, score, n, budget,
                      keep, reject_ids);
    return launch(kPhaseSelect, select_strided_kernel<0>, dim3(1), dim3(kT), stream, score, n, budget,
                  keep, reject_ids, (uint64_t *)ws);
}

}  // namespace pace
