// Block-wide exact top-`budget` selection for one 1024-thread workgroup
// (gfx950). Thread t holds kItems consecutive trajectories.
//
// Order: score descending, id ascending (equal scores reject the lower id
// first). Keys are the 64-bit order-preserving images of the binary64 scores
// (-0 -> +0, NaN above +inf), so unsigned key order is score order.
//
// Adaptive MSB-first radix select. The candidates are the keys that agree
// with `prefix` on the bits of `mask`; keys that disagree were decided by an
// earlier pass (rejected if (key & mask) > prefix, kept otherwise). Each pass
//   1. ORs and ANDs the candidates' keys: bits where they all agree join the
//      prefix at once, and the next digit is the 8 bits just below the
//      highest bit where they differ (so a tight cluster of scores costs no
//      more passes than a spread one);
//   2. histograms that digit in LDS (the wave's most common digits with one
//      atomic each) and lets wave 0 pick the digit bin holding the cut.
// It stops when the cut bin is rejected whole, when at most kDirect
// candidates remain (ranked pairwise by (key desc, id asc) in one wave), or
// when every candidate has the same key (ties go by an ordered count of ids).
// Scans and reductions use DPP row moves; a pass costs three barriers.
#pragma once

#include "device_util.hpp"

namespace pace {

constexpr int kSelT = 1024;
constexpr int kSelWaves = kSelT / kWave;
constexpr int kDirect = 64;

struct SelectSmem {
    uint32_t hist[2][256];
    uint32_t wsum[kSelWaves];
    uint64_t wor[kSelWaves], wand[kSelWaves];
    uint32_t sel_digit, sel_before, sel_cnt, ncand;
    uint64_t cand_key[kDirect];
    int64_t cand_id[kDirect];
    uint32_t cand_rej[kDirect];
};

__device__ __forceinline__ uint32_t sel_block_excl_scan(uint32_t v, uint32_t &total, uint32_t *wsum) {
    return block_excl_sum_u32<kSelWaves>(v, total, wsum);
}

// Clears the shared state; call once before select_block (which begins with
// a barrier).
__device__ __forceinline__ void select_smem_init(SelectSmem &sm) {
    if (threadIdx.x < 512) (&sm.hist[0][0])[threadIdx.x] = 0u;
    if (threadIdx.x == 0) sm.ncand = 0u;
}

// Bits [s, s+8) of k as a digit; s may be negative (the last digit then
// covers the low 8+s bits, shifted up).
__device__ __forceinline__ uint32_t digit_at(uint64_t k, int s) {
    return (uint32_t)((s >= 0 ? (k >> s) : (k << (-s))) & 0xFFull);
}
__device__ __forceinline__ uint64_t digit_bits(uint64_t d, int s) {
    return s >= 0 ? (d << s) : (d >> (-s));
}

// rej[q] <- trajectory base+q is rejected.
template <int kItems>
__device__ void select_block(const uint64_t (&k)[kItems], int64_t base, int64_t n, int64_t budget,
                             bool (&rej)[kItems], SelectSmem &sm) {
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int wv = tid / kWave;
    __syncthreads();
    if (budget <= 0 || budget >= n) {
#pragma unroll
        for (int q = 0; q < kItems; ++q) rej[q] = (base + q < n) && budget > 0;
        return;
    }

    // mode 2: reject (key & mask) >= prefix; 3: all candidates equal, the
    // first `need` ids are rejected; 4: pairwise-ranked candidates.
    int mode = 0;
    uint64_t prefix = 0, mask = 0;
    int64_t need = budget;
    uint32_t cnt = (uint32_t)n;
    for (int pass = 0; pass < 10; ++pass) {
        if (cnt <= (uint32_t)kDirect) {
            mode = 4;
            break;
        }
        // 1. bits on which all candidates agree
        uint64_t lor = 0, land = ~0ull;
#pragma unroll
        for (int q = 0; q < kItems; ++q) {
            if (base + q < n && ((k[q] ^ prefix) & mask) == 0ull) {
                lor |= k[q];
                land &= k[q];
            }
        }
        lor = wave_or_u64(lor);
        land = wave_and_u64(land);
        if (lane == 0) {
            sm.wor[wv] = lor;
            sm.wand[wv] = land;
        }
        __syncthreads();
        lor = 0;
        land = ~0ull;
#pragma unroll
        for (int w = 0; w < kSelWaves; ++w) {
            lor |= sm.wor[w];
            land &= sm.wand[w];
        }
        const uint64_t diff = lor ^ land;
        if (diff == 0ull) {                 // every candidate has the key lor
            prefix = lor;
            mask = ~0ull;
            mode = 3;
            break;
        }
        const int h = 63 - __clzll((long long)diff);
        const uint64_t agree = (h == 63) ? 0ull : (~0ull << (h + 1));
        prefix |= lor & agree;
        mask |= agree;
        const int s = h - 7;

        // 2. histogram of the digit below the agreed bits
        uint32_t *H = sm.hist[pass & 1];
#pragma unroll
        for (int q = 0; q < kItems; ++q) {
            bool act = base + q < n && ((k[q] ^ prefix) & mask) == 0ull;
            const uint32_t d = digit_at(k[q], s);
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const uint64_t m = ballot(act);
                if (m == 0ull) break;
                const int leader = __ffsll((long long)m) - 1;
                const uint32_t dl = (uint32_t)__builtin_amdgcn_readlane((int)d, leader);
                const uint64_t same = ballot(act && d == dl);
                if (lane == leader) atomicAdd(&H[dl], (uint32_t)__popcll(same));
                act = act && d != dl;
            }
            if (act) atomicAdd(&H[d], 1u);
        }
        __syncthreads();
        if (wv == 0) {
            // lane l owns digits 255-4l .. 252-4l (descending)
            const uint32_t h0 = H[255 - 4 * lane], h1 = H[254 - 4 * lane];
            const uint32_t h2 = H[253 - 4 * lane], h3 = H[252 - 4 * lane];
            const uint32_t t = h0 + h1 + h2 + h3;
            uint32_t bb = wave_incl_scan_u32(t) - t;      // keys with a larger digit
            const uint32_t hb[4] = {h0, h1, h2, h3};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if ((int64_t)bb < need && need <= (int64_t)bb + (int64_t)hb[j]) {
                    sm.sel_digit = 255u - 4u * (uint32_t)lane - (uint32_t)j;
                    sm.sel_before = bb;
                    sm.sel_cnt = hb[j];
                }
                bb += hb[j];
            }
        } else if (tid < kWave + 256) {
            sm.hist[(pass + 1) & 1][tid - kWave] = 0u;    // the next pass's buffer
        }
        __syncthreads();
        need -= (int64_t)sm.sel_before;
        cnt = sm.sel_cnt;
        prefix |= digit_bits(sm.sel_digit, s);
        mask |= digit_bits(0xFFull, s);
        if (need == (int64_t)cnt) {            // the whole bin is rejected
            mode = 2;
            break;
        }
    }
    if (mode == 0) mode = 4;   // not reached: ten passes fix more than 64 bits

    int slot[kItems];
    if (mode == 4) {
#pragma unroll
        for (int q = 0; q < kItems; ++q) {
            slot[q] = -1;
            if (base + q < n && ((k[q] ^ prefix) & mask) == 0ull) {
                const uint32_t sl = atomicAdd(&sm.ncand, 1u);
                if (sl < (uint32_t)kDirect) {
                    sm.cand_key[sl] = k[q];
                    sm.cand_id[sl] = base + q;
                    slot[q] = (int)sl;
                }
            }
        }
        __syncthreads();
        const uint32_t c = sm.ncand < (uint32_t)kDirect ? sm.ncand : (uint32_t)kDirect;
        if ((uint32_t)tid < c) {
            const uint64_t mk = sm.cand_key[tid];
            const int64_t mi = sm.cand_id[tid];
            uint32_t r = 0;
            for (uint32_t u = 0; u < c; ++u) {
                const uint64_t ku = sm.cand_key[u];
                r += (ku > mk || (ku == mk && sm.cand_id[u] < mi)) ? 1u : 0u;
            }
            sm.cand_rej[tid] = ((int64_t)r < need) ? 1u : 0u;
        }
        __syncthreads();
    }

    int64_t tie_rank = 0;
    if (mode == 3) {
        uint32_t eqc = 0;
#pragma unroll
        for (int q = 0; q < kItems; ++q) eqc += (base + q < n && k[q] == prefix) ? 1u : 0u;
        uint32_t t2;
        tie_rank = sel_block_excl_scan(eqc, t2, sm.wsum);
    }

#pragma unroll
    for (int q = 0; q < kItems; ++q) {
        bool r = false;
        if (base + q < n) {
            const uint64_t km = k[q] & mask;
            switch (mode) {
                case 2: r = km >= prefix; break;
                case 3:
                    if (km > prefix) r = true;
                    else if (k[q] == prefix) r = (tie_rank++ < need);
                    break;
                default:
                    r = km > prefix || (km == prefix && slot[q] >= 0 && sm.cand_rej[slot[q]] != 0u);
                    break;
            }
        }
        rej[q] = r;
    }
}

}  // namespace pace
