// Exact top-`budget` selection spread over the chip, for pools beyond the
// rank kernel's size limit: the Sec. 3.1 rejection rule taken over the current
// pool as an exact count (score descending, ties to the lower trajectory id),
// as a cut that any thread can apply to any (key, id).
//
// Keys are the 64-bit order-preserving images of the binary64 scores
// (score_key). Kernels, in order:
//   key_minmax  (only when the scores do not come from the filter step's
//               finalize, which writes the same per-group minima and maxima)
//               per group of trajectories, the smallest and largest key;
//               workgroup 0 clears the level-0 histogram;
//   cut_hist    up to kWideHistMax workgroups: the global key range [lo, hi]
//               from the group extremes, then each workgroup takes the
//               level-0 digit (Level0: linear in the score when the range is
//               finite, else the top bits of key - lo; monotone in the key)
//               of every score in its slice, keeps it (16 bits per
//               trajectory) and adds its LDS histogram to the global one;
//   classify    1024-thread workgroups; each first finds the cut itself
//               (find_cut): scans the global histogram from the top for
//               the bin holding the budget-th largest key; stages that bin's
//               keys (candidates) in LDS with one pass over the digits when
//               they fit, and repeats the bin search on them with finer key
//               bins until at most kRankMax remain, which are ranked by
//               counting on (key desc, id asc). A bin rejected whole ends the
//               search early; many equal keys are ordered by id with an
//               ordered count. More candidates than LDS holds are refined by
//               histogramming the scores again from global memory.
//               Then one thread per trajectory applies the cut: keep flags,
//               per block of kWideBlock trajectories the kept count and kept
//               tokens, and their sums per group of kGroupBlocks blocks, the
//               two-level partials the wide compaction reads.
// Histograms use LDS atomics, plus one global atomic per non-empty bin and
// workgroup; the integer counts do not depend on their order.
#include "device_util.hpp"
#include "kernels.hpp"

namespace pace {

namespace {

constexpr int kHBits = kCutBits;
constexpr int kHBins = 1 << kHBits;
constexpr int kWT = 1024;                // threads of the histogram and cut workgroups
constexpr int kWW = kWT / kWave;
constexpr int kCandCap = 4096;           // candidates staged in LDS
constexpr int kMMT = kFinGroup;          // threads of a min/max workgroup (one key each)

// Bins of 2^shift keys cover [lo, hi] in at most kHBins bins.
__device__ __forceinline__ int range_shift(uint64_t lo, uint64_t hi) {
    const uint64_t span = hi - lo;
    const int L = span ? 64 - __clzll((long long)span) : 0;
    return L > kHBits ? L - kHBits : 0;
}

__device__ __forceinline__ bool cut_rejects(const CutRec &c, uint64_t k, int64_t i) {
    switch (c.mode) {
        case 0: return false;
        case 1: return true;
        case 2: return k >= c.key;
        default: return k > c.key || (k == c.key && i <= c.id);
    }
}

// The score of a key (inverse of score_key; NaN for the NaN key).
__device__ __forceinline__ double key_score(uint64_t k) {
    const uint64_t b = (k >> 63) ? (k & 0x7fffffffffffffffull) : ~k;
    return __longlong_as_double((long long)b);
}

// Level-0 digit: linear in the score over [smin, smax] when both ends and
// their difference are finite and the range is not a point (bins of equal
// score width: a score distribution spreads over many of them), else the top
// bits of key - lo (bins of equal key width, which for binary64 keys mostly
// separate exponents). Either way the digit is monotone in the key, so every
// bin holds a contiguous range of keys.
struct Level0 {
    bool linear;
    double smin, scale;
    uint64_t lo;
    int sh;
    __device__ __forceinline__ uint32_t digit(uint64_t key, double s) const {
        if (linear) {
            const double x = (s - smin) * scale;
            return x < (double)(kHBins - 1) ? (uint32_t)x : (uint32_t)(kHBins - 1);
        }
        const uint64_t d = (key - lo) >> sh;
        return d < (uint64_t)kHBins ? (uint32_t)d : (uint32_t)(kHBins - 1);
    }
};
__device__ __forceinline__ Level0 level0(uint64_t lo, uint64_t hi) {
    Level0 L;
    const double a = key_score(lo), b = key_score(hi);
    const double w = b - a;
    L.linear = __builtin_isfinite(a) && __builtin_isfinite(b) && __builtin_isfinite(w) && w > 0.0;
    L.smin = a;
    L.scale = L.linear ? (double)kHBins / w : 0.0;
    L.lo = lo;
    L.sh = range_shift(lo, hi);
    return L;
}

// Smallest and largest key of each group of kMMT scores.
// Workgroup 0 also clears the level-0 histogram.
__global__ __launch_bounds__(kMMT) void key_minmax_kernel(const double *__restrict__ score, int64_t n,
                                                          uint64_t *__restrict__ mmin, uint64_t *__restrict__ mmax,
                                                          uint32_t *__restrict__ hist0) {
    __shared__ uint64_t wl[kMMT / kWave], wh[kMMT / kWave];
    if (blockIdx.x == 0)
        for (int b = threadIdx.x; b < kHBins; b += kMMT) hist0[b] = 0u;
    const int64_t i = (int64_t)blockIdx.x * kMMT + threadIdx.x;
    const uint64_t k = i < n ? score_key(score[i]) : 0ull;
    const uint64_t lo = wave_min_u64(i < n ? k : ~0ull), hi = wave_max_u64(k);
    if (lane_id() == 0) {
        wl[threadIdx.x / kWave] = lo;
        wh[threadIdx.x / kWave] = hi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t a = ~0ull, b = 0;
        for (int w = 0; w < kMMT / kWave; ++w) {
            a = wl[w] < a ? wl[w] : a;
            b = wh[w] > b ? wh[w] : b;
        }
        mmin[blockIdx.x] = a;
        mmax[blockIdx.x] = b;
    }
}

// Each workgroup histograms the level-0 digits of its slice of the scores in
// LDS, keeps every digit (16 bits per trajectory, for the cut workgroup's
// staging pass) and adds its non-empty bins to the global histogram, which the
// kernel before it cleared.
__global__ __launch_bounds__(kWT) void cut_hist_kernel(const double *__restrict__ score, int64_t n,
                                                       const uint64_t *__restrict__ mmin,
                                                       const uint64_t *__restrict__ mmax, int64_t n_mm,
                                                       int64_t per_wg, uint32_t *__restrict__ hist,
                                                       uint16_t *__restrict__ digit, uint64_t *__restrict__ range) {
    __shared__ uint32_t h[kHBins];
    __shared__ uint64_t wl[kWW], wh[kWW];
    const int t = threadIdx.x, lane = lane_id(), wv = t / kWave;
    const int64_t i0 = (int64_t)blockIdx.x * per_wg;
    const int64_t i1 = (i0 + per_wg < n) ? i0 + per_wg : n;
    // The first scores of the slice do not depend on the range: load them first.
    double sc[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int64_t j = i0 + t + (int64_t)u * kWT;
        sc[u] = j < i1 ? score[j] : 0.0;
    }
    for (int b = t; b < kHBins; b += kWT) h[b] = 0u;
    uint64_t lo = ~0ull, hi = 0;
    for (int64_t i = t; i < n_mm; i += kWT) {
        const uint64_t a = mmin[i], b = mmax[i];
        lo = a < lo ? a : lo;
        hi = b > hi ? b : hi;
    }
    lo = wave_min_u64(lo);
    hi = wave_max_u64(hi);
    if (lane == 0) {
        wl[wv] = lo;
        wh[wv] = hi;
    }
    __syncthreads();
    lo = ~0ull;
    hi = 0;
#pragma unroll
    for (int w = 0; w < kWW; ++w) {
        lo = wl[w] < lo ? wl[w] : lo;
        hi = wh[w] > hi ? wh[w] : hi;
    }
    const Level0 L = level0(lo, hi);
    for (int64_t i = i0 + t; i < i1; i += 4 * kWT) {
        if (i != i0 + t) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t j = i + (int64_t)u * kWT;
                sc[u] = j < i1 ? score[j] : 0.0;
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t j = i + (int64_t)u * kWT;
            if (j < i1) {
                const uint32_t d = L.digit(score_key(sc[u]), sc[u]);
                atomicAdd(&h[d], 1u);
                digit[j] = (uint16_t)d;
            }
        }
    }
    __syncthreads();
    for (int b = t; b < kHBins; b += kWT)
        if (h[b] != 0u) atomicAdd(&hist[b], h[b]);
    if (blockIdx.x == 0 && t == 0) {
        range[0] = lo;
        range[1] = hi;
    }
}

// Shared memory of the cut search (one 1024-thread workgroup).
struct CutSmem {
    uint32_t h[kHBins];
    uint32_t wsum[kWW];
    uint64_t ck[kCandCap];
    uint32_t ci[kCandCap];
    uint32_t ncand;
    uint64_t s_lo, s_hi, s_key;
    int64_t s_need, s_id;
    uint32_t s_cnt, s_d;
    uint64_t wl[kWW], wh[kWW];
    CutRec cut;
};
constexpr int kRankMax = kWT / 4;        // candidates ranked by counting, four threads each

// The rejection cut of the budget highest (key, -id) from the level-0
// histogram and digits. Called by every thread of a kWT-thread workgroup; the
// result is in sm.cut after the caller's next barrier.
__device__ void find_cut(const double *__restrict__ score, int64_t n, int64_t budget,
                         const uint32_t *__restrict__ hist, const uint16_t *__restrict__ digit,
                         const uint64_t *__restrict__ range, CutSmem &sm) {
    const int t = threadIdx.x, lane = lane_id();
    if (budget <= 0 || budget >= n) {
        if (t == 0) sm.cut = CutRec{budget <= 0 ? 0 : 1, 0, 0, 0};
        return;
    }
    uint64_t lo = range[0], hi = range[1];
    int64_t need = budget;
    uint32_t cnt = 0;

    // Descending bin search over key bins of 2^sh: thread t holds the counts
    // a, b of digits kHBins - 1 - 2t and kHBins - 2 - 2t. Narrows [lo, hi] to
    // the bin that holds the need-th largest candidate.
    auto pick = [&](uint32_t a, uint32_t b, int sh) {
        uint32_t tot;
        const uint32_t ex = block_excl_sum_u32<kWW>(a + b, tot, sm.wsum);
        if ((int64_t)ex < need && need <= (int64_t)ex + a + b) {
            const bool first = need <= (int64_t)ex + a;
            const uint64_t d = first ? (uint64_t)(kHBins - 1 - 2 * t) : (uint64_t)(kHBins - 2 - 2 * t);
            const uint64_t blo = lo + (d << sh);
            const uint64_t room = hi - blo, w = (((uint64_t)1 << sh) - 1);
            sm.s_need = need - (int64_t)(first ? ex : ex + a);
            sm.s_cnt = first ? a : b;
            sm.s_lo = blo;
            sm.s_hi = blo + (room < w ? room : w);
        }
        __syncthreads();
        need = sm.s_need;
        cnt = sm.s_cnt;
        lo = sm.s_lo;
        hi = sm.s_hi;
        __syncthreads();
    };
    auto reject_bin_and_above = [&]() {
        if (t == 0) sm.cut = CutRec{2, lo, 0, 0};
    };

    // Level 0: the global histogram of the level-0 digits, from the top.
    uint32_t d0;
    {
        uint32_t tot;
        const uint32_t a = hist[kHBins - 1 - 2 * t], b = hist[kHBins - 2 - 2 * t];
        const uint32_t ex = block_excl_sum_u32<kWW>(a + b, tot, sm.wsum);
        if ((int64_t)ex < need && need <= (int64_t)ex + a + b) {
            const bool first = need <= (int64_t)ex + a;
            sm.s_d = first ? (uint32_t)(kHBins - 1 - 2 * t) : (uint32_t)(kHBins - 2 - 2 * t);
            sm.s_need = need - (int64_t)(first ? ex : ex + a);
            sm.s_cnt = first ? a : b;
        }
        if (t == 0) sm.ncand = 0u;
        __syncthreads();
        d0 = sm.s_d;
        need = sm.s_need;
        cnt = sm.s_cnt;
        __syncthreads();
    }
    // The keys of bin d0: staged in LDS when they fit (a pass over the
    // digits, then one load of each candidate's score), else only their
    // smallest and largest key. Either way [lo, hi] becomes the bin's key
    // range.
    bool staged = false;
    uint64_t kl = ~0ull, kh = 0;
    if (cnt <= (uint32_t)kCandCap) {
        constexpr int kDU = 8;                   // 16-byte digit vectors in flight per thread
        const int64_t nv = (n + 7) / 8;
        const uint32_t dd = d0 | (d0 << 16);
        for (int64_t v0 = t; v0 < nv; v0 += (int64_t)kDU * kWT) {
            uint4 dv[kDU];
#pragma unroll
            for (int u = 0; u < kDU; ++u) {
                const int64_t v = v0 + (int64_t)u * kWT;
                dv[u] = v < nv ? *reinterpret_cast<const uint4 *>(digit + v * 8) : make_uint4(~0u, ~0u, ~0u, ~0u);
            }
#pragma unroll
            for (int u = 0; u < kDU; ++u) {
                // Digits are below 2^15, so (x - 0x10001) & ~x & 0x80008000 is
                // non-zero exactly when a half of x = word ^ dd is zero (or
                // the borrow of a zero low half reaches the high one).
                const uint32_t wd[4] = {dv[u].x ^ dd, dv[u].y ^ dd, dv[u].z ^ dd, dv[u].w ^ dd};
                uint32_t any = 0;
#pragma unroll
                for (int e = 0; e < 4; ++e) any |= (wd[e] - 0x00010001u) & ~wd[e] & 0x80008000u;
                if (any != 0u) {
                    const int64_t v = v0 + (int64_t)u * kWT;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int64_t i = v * 8 + e;
                        if (i < n && ((wd[e >> 1] >> (16 * (e & 1))) & 0xffffu) == 0u) {
                            const uint32_t sl = atomicAdd(&sm.ncand, 1u);
                            if (sl < (uint32_t)kCandCap) sm.ci[sl] = (uint32_t)i;
                        }
                    }
                }
            }
        }
        __syncthreads();
        cnt = sm.ncand < (uint32_t)kCandCap ? sm.ncand : (uint32_t)kCandCap;
        for (uint32_t j = (uint32_t)t; j < cnt; j += kWT) {
            const uint64_t k = score_key(score[sm.ci[j]]);
            sm.ck[j] = k;
            kl = k < kl ? k : kl;
            kh = k > kh ? k : kh;
        }
        staged = true;
    } else {
        for (int64_t i = t; i < n; i += kWT) {
            if (digit[i] == d0) {
                const uint64_t k = score_key(score[i]);
                kl = k < kl ? k : kl;
                kh = k > kh ? k : kh;
            }
        }
    }
    kl = wave_min_u64(kl);
    kh = wave_max_u64(kh);
    if (lane == 0) {
        sm.wl[t / kWave] = kl;
        sm.wh[t / kWave] = kh;
    }
    __syncthreads();
    lo = ~0ull;
    hi = 0;
#pragma unroll
    for (int w = 0; w < kWW; ++w) {
        lo = sm.wl[w] < lo ? sm.wl[w] : lo;
        hi = sm.wh[w] > hi ? sm.wh[w] : hi;
    }
    if (need == (int64_t)cnt) {
        reject_bin_and_above();
        return;
    }

    // Finer levels until at most kRankMax candidates remain or they all share
    // one key (each level splits the key range by 2^kHBits, so six suffice).
    for (int level = 0; level < 8 && lo != hi; ++level) {
        if (!staged && cnt <= (uint32_t)kCandCap) {
            // One pass over the scores stages every key in [lo, hi].
            if (t == 0) sm.ncand = 0u;
            __syncthreads();
            for (int64_t i = t; i < n; i += 4 * kWT) {
                uint64_t k[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int64_t j = i + (int64_t)u * kWT;
                    k[u] = j < n ? score_key(score[j]) : 0ull;
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int64_t j = i + (int64_t)u * kWT;
                    const bool c = j < n && k[u] >= lo && k[u] <= hi;
                    const uint64_t m = ballot(c);
                    if (m != 0ull) {
                        const int leader = __ffsll((long long)m) - 1;
                        uint32_t base = 0;
                        if (lane == leader) base = atomicAdd(&sm.ncand, (uint32_t)__popcll(m));
                        base = (uint32_t)__builtin_amdgcn_readlane((int)base, leader);
                        const uint32_t sl = base + (uint32_t)__popcll(m & lanes_below());
                        if (c && sl < (uint32_t)kCandCap) {
                            sm.ck[sl] = k[u];
                            sm.ci[sl] = (uint32_t)j;
                        }
                    }
                }
            }
            __syncthreads();
            cnt = sm.ncand < (uint32_t)kCandCap ? sm.ncand : (uint32_t)kCandCap;
            staged = true;
        }
        if (staged && cnt <= (uint32_t)kRankMax) break;
        // histogram of the candidates' next digit
        const int sh = range_shift(lo, hi);
        for (int b = t; b < kHBins; b += kWT) sm.h[b] = 0u;
        __syncthreads();
        if (staged) {
            for (uint32_t j = (uint32_t)t; j < cnt; j += kWT) {
                const uint64_t k = sm.ck[j];
                if (k >= lo && k <= hi) atomicAdd(&sm.h[(k - lo) >> sh], 1u);
            }
        } else {
            for (int64_t i = t; i < n; i += kWT) {
                const uint64_t k = score_key(score[i]);
                if (k >= lo && k <= hi) atomicAdd(&sm.h[(k - lo) >> sh], 1u);
            }
        }
        __syncthreads();
        pick(sm.h[kHBins - 1 - 2 * t], sm.h[kHBins - 2 - 2 * t], sh);
        if (need == (int64_t)cnt) {
            reject_bin_and_above();
            return;
        }
        if (staged) {
            // keep the staged candidates that lie in the new range
            uint64_t kk[kCandCap / kWT];
            uint32_t ii[kCandCap / kWT];
            const uint32_t c_old = sm.ncand < (uint32_t)kCandCap ? sm.ncand : (uint32_t)kCandCap;
#pragma unroll
            for (int u = 0; u < kCandCap / kWT; ++u) {
                const uint32_t j = (uint32_t)t + (uint32_t)u * kWT;
                kk[u] = j < c_old ? sm.ck[j] : 0ull;
                ii[u] = j < c_old ? sm.ci[j] : 0u;
            }
            __syncthreads();
            if (t == 0) sm.ncand = 0u;
            __syncthreads();
#pragma unroll
            for (int u = 0; u < kCandCap / kWT; ++u) {
                const uint32_t j = (uint32_t)t + (uint32_t)u * kWT;
                const bool c = j < c_old && kk[u] >= lo && kk[u] <= hi;
                const uint64_t m = ballot(c);
                if (m != 0ull) {
                    const int leader = __ffsll((long long)m) - 1;
                    uint32_t base = 0;
                    if (lane == leader) base = atomicAdd(&sm.ncand, (uint32_t)__popcll(m));
                    base = (uint32_t)__builtin_amdgcn_readlane((int)base, leader);
                    if (c) {
                        const uint32_t sl = base + (uint32_t)__popcll(m & lanes_below());
                        sm.ck[sl] = kk[u];
                        sm.ci[sl] = ii[u];
                    }
                }
            }
            __syncthreads();
            cnt = sm.ncand;
        }
    }

    if (staged && cnt <= (uint32_t)kRankMax) {
        // Rank by counting: candidate j gets threads 4j .. 4j + 3, each
        // comparing it with every fourth candidate; the need-th largest
        // (key desc, id asc) has rank need - 1.
        const uint32_t j = (uint32_t)t >> 2, q = (uint32_t)t & 3u;
        uint32_t r = 0;
        uint64_t ka = 0;
        uint32_t ia = 0;
        if (j < cnt) {
            ka = sm.ck[j];
            ia = sm.ci[j];
            for (uint32_t x = q; x < cnt; x += 4) {
                const uint64_t kb = sm.ck[x];
                const uint32_t ib = sm.ci[x];
                r += (kb > ka || (kb == ka && ib < ia)) ? 1u : 0u;
            }
        }
        r += (uint32_t)__shfl_xor((int)r, 1, kWave);
        r += (uint32_t)__shfl_xor((int)r, 2, kWave);
        if (j < cnt && q == 0u && (int64_t)r == need - 1) sm.cut = CutRec{3, ka, (int64_t)ia, 0};
        return;
    }

    // Every candidate has the key lo (more of them than the ranking takes):
    // the need-th lowest id among the trajectories with that key, by an
    // ordered count over ids (thread t takes ids [t*per, (t+1)*per)).
    const int64_t per = (n + kWT - 1) / kWT;
    const int64_t j0 = (int64_t)t * per, j1 = (j0 + per < n) ? j0 + per : n;
    uint32_t c = 0;
    for (int64_t j = j0; j < j1; ++j) c += score_key(score[j]) == lo ? 1u : 0u;
    uint32_t tot;
    uint32_t before = block_excl_sum_u32<kWW>(c, tot, sm.wsum);
    if ((int64_t)before < need && need <= (int64_t)before + c) {
        for (int64_t j = j0; j < j1; ++j) {
            if (score_key(score[j]) == lo && (int64_t)(++before) == need) {
                sm.cut = CutRec{3, lo, j, 0};
                break;
            }
        }
    }
}

// One 1024-thread workgroup per 1024 trajectories: the cut (find_cut, the
// same in every workgroup), then per trajectory the keep flag, per block of
// kWideBlock trajectories (one wave) the kept count and kept tokens (spans
// clamped to [0, NT]; zero without offsets), and per workgroup (a group of
// kGroupBlocks blocks) their sums. Workgroup 0 also stores the cut.
__global__ __launch_bounds__(kWT) void classify_kernel(const double *__restrict__ score,
                                                       const int64_t *__restrict__ off, int64_t n, int64_t NT,
                                                       int64_t budget, const uint32_t *__restrict__ hist,
                                                       const uint16_t *__restrict__ digit,
                                                       const uint64_t *__restrict__ range, CutRec *__restrict__ cut,
                                                       uint8_t *__restrict__ keep, PieceParts parts) {
    static_assert(kWideBlock == kWave, "a wide block is one wave");
    __shared__ CutSmem sm;
    const int64_t i = (int64_t)blockIdx.x * kWT + threadIdx.x;
    // This thread's trajectory first: its loads do not wait for the cut.
    double sc = 0.0;
    int64_t lo = 0, hi = 0;
    if (i < n) {
        sc = score[i];
        if (off) {
            lo = clamp64(off[i], 0, NT);
            hi = clamp64(off[i + 1], 0, NT);
        }
    }
    find_cut(score, n, budget, hist, digit, range, sm);
    __syncthreads();
    const CutRec c = sm.cut;
    if (blockIdx.x == 0 && threadIdx.x == 0) *cut = c;
    bool kept = false;
    int64_t len = 0;
    if (i < n) {
        kept = !cut_rejects(c, score_key(sc), i);
        keep[i] = kept ? 1 : 0;
        len = kept && hi > lo ? hi - lo : 0;
    }
    const uint32_t kc = (uint32_t)__popcll(ballot(kept));
    const int64_t l = wave_sum_i64(len);
    const int64_t b = i / kWideBlock;
    const int w = threadIdx.x / kWave;
    static_assert(kWT == kWideBlock * kGroupBlocks, "a classify workgroup is one group of blocks");
    if (lane_id() == 0) {
        if (b * kWideBlock < n) {
            parts.cnt[b] = (int32_t)kc;
            parts.len[b] = l;
        }
        sm.wl[w] = kc;                  // the search's LDS is free again
        sm.wh[w] = (uint64_t)l;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t gc = 0;
        int64_t gl = 0;
        for (int k = 0; k < kGroupBlocks; ++k) {
            gc += (uint32_t)sm.wl[k];
            gl += (int64_t)sm.wh[k];
        }
        parts.gcnt[blockIdx.x] = (int32_t)gc;
        parts.glen[blockIdx.x] = gl;
    }
}

// Rejected ids in ascending order: one wave per block of kWideBlock
// trajectories; the rejections before the block follow from the kept counts
// of the blocks before it.
__global__ __launch_bounds__(kWave) void emit_rejects_wide_kernel(const uint8_t *__restrict__ keep, int64_t n,
                                                                  const int32_t *__restrict__ kept_cnt,
                                                                  int64_t budget, int32_t *__restrict__ reject_ids) {
    const int lane = lane_id();
    const int64_t b = blockIdx.x;
    int64_t s = 0;
    for (int64_t j = lane; j < b; j += kWave) s += kept_cnt[j];
    s = wave_sum_i64(s);
    const int64_t i = b * kWideBlock + lane;
    const bool rej = i < n && keep[i] == 0;
    const int64_t pos = b * kWideBlock - s + (int64_t)__popcll(ballot(rej) & lanes_below());
    if (rej && pos < budget) reject_ids[pos] = (int32_t)i;
}

}  // namespace

int64_t wide_hist_wgs(int64_t n) {
    const int64_t g = n / 2048;
    return g < 1 ? 1 : (g > kWideHistMax ? kWideHistMax : g);
}

size_t wide_select_ws_bytes(int64_t n) {
    const int64_t mm = (n + kMMT - 1) / kMMT;
    const int64_t nb = (n + kWideBlock - 1) / kWideBlock;
    const int64_t ng = wide_groups(n);
    return 256 + align256((size_t)mm * 8) * 2 + align256((size_t)kHBins * 4) + align256((size_t)n * 2) +
           align256((size_t)nb * 4) * 2 + align256((size_t)nb * 8) + align256((size_t)ng * 4) +
           align256((size_t)ng * 8);
}

WideWs wide_ws_carve(void *ws, int64_t n) {
    const int64_t mm = (n + kMMT - 1) / kMMT;
    char *p = (char *)ws;
    WideWs w;
    w.cut = (CutRec *)p;        p += 64;
    w.range = (uint64_t *)p;    p += 192;
    w.mmin = (uint64_t *)p;     p += align256((size_t)mm * 8);
    w.mmax = (uint64_t *)p;     p += align256((size_t)mm * 8);
    w.hist = (uint32_t *)p;     p += align256((size_t)kHBins * 4);
    w.digit = (uint16_t *)p;    p += align256((size_t)n * 2);
    const int64_t nb = (n + kWideBlock - 1) / kWideBlock;
    w.parts.cnt = (int32_t *)p; p += align256((size_t)nb * 4);
    w.parts.len = (int64_t *)p; p += align256((size_t)nb * 8);
    w.parts.pcs = (int32_t *)p; p += align256((size_t)nb * 4);
    const int64_t ng = wide_groups(n);
    w.parts.gcnt = (int32_t *)p; p += align256((size_t)ng * 4);
    w.parts.glen = (int64_t *)p;
    w.n_mm = mm;
    return w;
}

hipError_t launch_key_minmax(const double *score, int64_t n, const WideWs &w, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    return launch(kPhaseSelect, key_minmax_kernel, dim3((unsigned)w.n_mm), dim3(kMMT), stream, score, n, w.mmin,
                  w.mmax, w.hist);
}

hipError_t launch_wide_cut(const double *score, int64_t n, int64_t budget, const WideWs &w, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const int64_t g = wide_hist_wgs(n);
    const int64_t per = (n + g - 1) / g;
    return launch(kPhaseSelect, cut_hist_kernel, dim3((unsigned)g), dim3(kWT), stream, score, n, w.mmin,
                  w.mmax, w.n_mm, per, w.hist, w.digit, w.range);
}

hipError_t launch_classify(const double *score, const int64_t *offsets, int64_t n, int64_t n_tokens,
                           int64_t budget, const WideWs &w, uint8_t *keep, const PieceParts &parts,
                           hipStream_t stream) {
    if (n == 0) return hipSuccess;
    return launch(kPhaseClassify, classify_kernel, dim3((unsigned)((n + kWT - 1) / kWT)), dim3(kWT), stream,
                  score, offsets, n, n_tokens, budget, w.hist, w.digit, w.range, w.cut, keep, parts);
}

hipError_t launch_emit_rejects_wide(const uint8_t *keep, int64_t n, const int32_t *kept_cnt, int64_t budget,
                                    int32_t *reject_ids, hipStream_t stream) {
    if (n == 0 || budget == 0) return hipSuccess;
    return launch(kPhaseSelect, emit_rejects_wide_kernel, dim3((unsigned)((n + kWideBlock - 1) / kWideBlock)),
                  dim3(kWave), stream, keep, n, kept_cnt, budget, reject_ids);
}

}  // namespace pace
