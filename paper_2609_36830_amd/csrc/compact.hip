// pace_compact kernels for gfx950: pack the kept trajectories' token spans
// into the training batch (Algorithm 1), survivors in pool order.
//
// Copy routine of the scan path: a wave copies a contiguous range of output
// elements. Output goes out as aligned 16-byte non-temporal vectors (64 lanes
// x 16 B = 1 KiB per wave window, four windows in flight); sources are read
// with plain loads, since the kept spans are often still in the last-level
// cache from the scoring pass. Inside one kept span the source is the
// destination shifted by a constant, so the source
// misalignment is wave-uniform: each lane loads the aligned 16 bytes under
// its window, takes the next 16 bytes from the neighbouring lane (lane 63
// loads them), and a byte funnel shift assembles the output vector. Windows
// that straddle span ends, the ragged tail and unaligned columns copy element
// by element.
//
// Piece path (n <= kPieceMaxN): consecutive trajectories form blocks of
// kPieceBlock; per block the rank kernel (or compact_partials_kernel) has
// written the kept count, kept tokens and the number of pieces of at most
// kPieceLen tokens the kept spans cut into. The copy kernel then runs one
// 256-thread workgroup per block, writing that block's packed offsets, kept
// ids and rejected ids, and piece workgroups (at most one resident round;
// each takes pieces q, q + stride, ...): the workgroup scans the block
// partials (at most 512) to find a piece's block, the 16 trajectories of the
// block to find its span, and copies the piece with 16-byte vectors, four
// loads in flight per thread (source loads dword-aligned, stores aligned and
// non-temporal). Pieces are short enough that long trajectories spread over
// many workgroups, long enough that the per-workgroup set-up is small next to
// the copy.
//
// Wide path (8192 < n <= kWideMaxN): blocks of kWideBlock trajectories with
// two-level partials, and the packed output split evenly over one resident
// round of workgroups by merge path (compact_wide_kernel below).
//
// Scan path (larger pools): one workgroup scans the flags into the packed
// offsets, kept ids, span sources and a map from each output chunk of
// kCopyChunk elements to its first span; a second kernel copies.
#include "device_util.hpp"
#include "kernels.hpp"

namespace pace {

namespace {

constexpr int kT = 1024;
constexpr int kNW = kT / kWave;

// ---------------------------------------------------------------------------
// Spans: packed offsets o(j) and source starts s(j) of kept span j
// ---------------------------------------------------------------------------
// Global arrays, lane k caching entry base + k.
struct GlobalSpans {
    const int64_t *oo;
    const int64_t *ss;
    int64_t n_kept;
    int64_t base, o, s;
    __device__ __forceinline__ void load(int64_t b) {
        base = b;
        const int64_t idx = b + lane_id();
        o = (idx <= n_kept) ? oo[idx] : INT64_MAX;
        s = (idx < n_kept) ? ss[idx] : 0;
    }
    __device__ __forceinline__ void ensure(int64_t j) {   // entries j and j + 1
        if (j < base || j + 1 - base >= kWave) load(j);
    }
    __device__ __forceinline__ int64_t O(int64_t j) const { return readlane_i64(o, (int)(j - base)); }
    __device__ __forceinline__ int64_t S(int64_t j) const { return readlane_i64(s, (int)(j - base)); }
};

template <int E> struct Elem;
template <> struct Elem<1> { using T = uint8_t; };
template <> struct Elem<2> { using T = uint16_t; };
template <> struct Elem<4> { using T = uint32_t; };
template <> struct Elem<8> { using T = uint64_t; };

// Bytes [shift, shift + 16) of the 32-byte little-endian string a|b
// (shift is wave-uniform).
__device__ __forceinline__ uint4 funnel16(const uint4 &a, const uint4 &b, int shift) {
    const uint32_t r = (uint32_t)(shift & 3);
#define AB(hi, lo) __builtin_amdgcn_alignbyte((hi), (lo), r)
    uint4 o;
    switch (shift >> 2) {
        case 0: o = make_uint4(AB(a.y, a.x), AB(a.z, a.y), AB(a.w, a.z), AB(b.x, a.w)); break;
        case 1: o = make_uint4(AB(a.z, a.y), AB(a.w, a.z), AB(b.x, a.w), AB(b.y, b.x)); break;
        case 2: o = make_uint4(AB(a.w, a.z), AB(b.x, a.w), AB(b.y, b.x), AB(b.z, b.y)); break;
        default: o = make_uint4(AB(b.x, a.w), AB(b.y, b.x), AB(b.z, b.y), AB(b.w, b.z)); break;
    }
#undef AB
    return o;
}

__device__ __forceinline__ uint4 shfl_down1(const uint4 &a) {
    uint4 b;
    b.x = (uint32_t)__shfl_down((int)a.x, 1, kWave);
    b.y = (uint32_t)__shfl_down((int)a.y, 1, kWave);
    b.z = (uint32_t)__shfl_down((int)a.z, 1, kWave);
    b.w = (uint32_t)__shfl_down((int)a.w, 1, kWave);
    return b;
}

// Copies packed elements [cs, ce) of one column; j is a kept span with
// o(j) <= cs (the last such, for well-formed input). Every access is checked
// against n_tokens, so malformed offsets stay in bounds.
template <int E, typename Spans>
__device__ void copy_range(const char *__restrict__ in, char *__restrict__ out, bool vec, Spans &sp,
                           int64_t n_kept, int64_t NT, int64_t cs, int64_t ce, int64_t j) {
    using T = typename Elem<E>::T;
    constexpr int VE = 16 / E;          // elements per lane vector
    constexpr int WE = kWave * VE;      // elements per wave window (1 KiB)
    constexpr int U = 4;                // windows per unrolled step
    const int lane = lane_id();
    const int64_t nbytes = NT * E;
    for (int64_t w = cs; w < ce; w += WE) {
        sp.ensure(j);
        while (j + 1 < n_kept && sp.O(j + 1) <= w) {
            ++j;
            sp.ensure(j);
        }
        const int64_t we = (w + WE < ce) ? w + WE : ce;
        const int64_t o_lo = sp.O(j), o_hi = sp.O(j + 1);
        const int64_t delta = sp.S(j) - o_lo;          // src element = dst element + delta
        const int shift = (int)((((delta * E) % 16) + 16) % 16);
        // lane 63's extra aligned vector after its own, for the last window
        auto tail_ok = [&](int64_t nwin) {
            const int64_t ab63 = (w + (nwin - 1) * WE + (int64_t)(kWave - 1) * VE + delta) * E - shift;
            return shift == 0 || ab63 + 32 <= nbytes;
        };
        const bool in_span = vec && o_lo <= w && w + delta >= 0;
        if (in_span && w + U * WE <= o_hi && w + U * WE <= ce && w + U * WE + delta <= NT && tail_ok(U)) {
            const int64_t ab = (w + (int64_t)lane * VE + delta) * E - shift;
            uint4 a[U], x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) a[u] = *reinterpret_cast<const uint4 *>(in + ab + u * 1024);
            if (shift != 0 && lane == kWave - 1) {
#pragma unroll
                for (int u = 0; u < U; ++u) x[u] = *reinterpret_cast<const uint4 *>(in + ab + u * 1024 + 16);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                uint4 o = a[u];
                if (shift != 0) {
                    uint4 b = shfl_down1(a[u]);
                    if (lane == kWave - 1) b = x[u];
                    o = funnel16(a[u], b, shift);
                }
                store_nt(reinterpret_cast<uint4 *>(out + (w + (int64_t)u * WE + (int64_t)lane * VE) * E), o);
            }
            w += (U - 1) * WE;
            continue;
        }
        if (in_span && w + WE <= o_hi && w + WE <= ce && w + WE + delta <= NT && tail_ok(1)) {
            const int64_t ab = (w + (int64_t)lane * VE + delta) * E - shift;
            const uint4 a = *reinterpret_cast<const uint4 *>(in + ab);
            uint4 o = a;
            if (shift != 0) {
                uint4 b = shfl_down1(a);
                if (lane == kWave - 1) b = *reinterpret_cast<const uint4 *>(in + ab + 16);
                o = funnel16(a, b, shift);
            }
            store_nt(reinterpret_cast<uint4 *>(out + (w + (int64_t)lane * VE) * E), o);
            continue;
        }
        // Element path: every span that meets [w, we).
        int64_t jj = j;
        while (true) {
            sp.ensure(jj);
            const int64_t lo = sp.O(jj), hi = sp.O(jj + 1);
            const int64_t d = sp.S(jj) - lo;
            const int64_t a = lo > w ? lo : w;
            const int64_t b = hi < we ? hi : we;
#pragma unroll
            for (int k = 0; k < VE; ++k) {
                const int64_t p = w + (int64_t)lane * VE + k;
                const int64_t src = p + d;
                if (p >= a && p < b && src >= 0 && src < NT)
                    reinterpret_cast<T *>(out)[p] = reinterpret_cast<const T *>(in)[src];
            }
            if (hi >= we || jj + 1 >= n_kept) break;
            ++jj;
        }
        j = jj;
    }
}

template <typename Spans>
__device__ __forceinline__ void copy_range_col(const CompactCols &cols, int col, Spans &sp,
                                               int64_t n_kept, int64_t NT, int64_t cs, int64_t ce,
                                               int64_t j) {
    const char *in = (const char *)cols.in[col];
    char *out = (char *)cols.out[col];
    const bool vec = cols.vec[col] != 0;
    switch (cols.elem[col]) {
        case 1: copy_range<1>(in, out, vec, sp, n_kept, NT, cs, ce, j); break;
        case 2: copy_range<2>(in, out, vec, sp, n_kept, NT, cs, ce, j); break;
        case 4: copy_range<4>(in, out, vec, sp, n_kept, NT, cs, ce, j); break;
        default: copy_range<8>(in, out, vec, sp, n_kept, NT, cs, ce, j); break;
    }
}

// ---------------------------------------------------------------------------
// Piece path
// ---------------------------------------------------------------------------
constexpr int kPT = 256;                  // threads of a piece workgroup
constexpr int kPW = kPT / kWave;          // its waves
constexpr int kCopyU = 4;                 // 16-byte loads in flight per thread in a piece copy

// Span length of trajectory i if kept (offsets clamped to [0, NT]), else 0.
// (The flag and both offsets are loaded together: one round trip.)
__device__ __forceinline__ int64_t kept_span(const int64_t *__restrict__ off, const uint8_t *__restrict__ keep,
                                             int64_t i, int64_t NT, int64_t &lo) {
    const bool k = keep[i] != 0;
    const int64_t a = off[i], b = off[i + 1];
    lo = 0;
    if (!k) return -1;
    lo = clamp64(a, 0, NT);
    const int64_t hi = clamp64(b, 0, NT);
    return hi > lo ? hi - lo : 0;
}

// One wave per block of kBlk trajectories: the block partials from the keep
// flags.
template <int kBlk>
__global__ __launch_bounds__(kWave) void compact_partials_kernel(const int64_t *__restrict__ off, int64_t n,
                                                                int64_t NT, const uint8_t *__restrict__ keep,
                                                                PieceParts parts) {
    const int lane = lane_id();
    const int64_t i = (int64_t)blockIdx.x * kBlk + lane;
    int64_t len = 0, lo;
    bool kept = false;
    if (lane < kBlk && i < n) {
        const int64_t k = kept_span(off, keep, i, NT, lo);
        kept = k >= 0;
        len = kept ? k : 0;
    }
    const uint32_t c = (uint32_t)__popcll(ballot(kept));
    const int64_t l = wave_sum_i64(len);
    const int64_t pc = wave_sum_i64((len + kPieceLen - 1) / kPieceLen);
    if (lane == 0) {
        parts.cnt[blockIdx.x] = (int32_t)c;
        parts.len[blockIdx.x] = l;
        parts.pcs[blockIdx.x] = (int32_t)pc;
    }
}

// The workgroup copies elements [d, d + m) of one column from [s, s + m).
template <int E>
__device__ __forceinline__ void copy_piece(const char *__restrict__ in, char *__restrict__ out, bool vec,
                                           int64_t d, int64_t s, int64_t m) {
    using T = typename Elem<E>::T;
    const T *src = reinterpret_cast<const T *>(in);
    T *dst = reinterpret_cast<T *>(out);
    const int t = threadIdx.x;
    const int64_t delta = s - d;
    if (E >= 4 && vec) {
        constexpr int VE = 16 / E;
        const int64_t e = d + m;
        const int64_t a0 = (d + VE - 1) / VE * VE, a1 = e / VE * VE;
        if (a0 < a1) {
            if (t < a0 - d) dst[d + t] = src[d + t + delta];
            if (t < e - a1) dst[a1 + t] = src[a1 + t + delta];
            // kCopyU loads in flight per thread, then their stores.
            const int64_t v1 = a1 / VE;
            int64_t v = a0 / VE + t;
            for (; v + (kCopyU - 1) * kPT < v1; v += kCopyU * kPT) {
                uint4 x[kCopyU];
#pragma unroll
                for (int u = 0; u < kCopyU; ++u) x[u] = load_a4(src + (v + u * kPT) * VE + delta);
#pragma unroll
                for (int u = 0; u < kCopyU; ++u) store_nt(reinterpret_cast<uint4 *>(dst + (v + u * kPT) * VE), x[u]);
            }
            for (; v < v1; v += kPT) store_nt(reinterpret_cast<uint4 *>(dst + v * VE), load_a4(src + v * VE + delta));
            return;
        }
    }
    for (int64_t p = d + t; p < d + m; p += kPT) dst[p] = src[p + delta];
}

// kBlk trajectories per block (at most a wave); thread t holds the partials
// of blocks [t*kPP, (t+1)*kPP). offsets_out, kept_ids and n_kept_tokens may
// be null (rejected ids only).
template <int kBlk, int kPP>
__global__ __launch_bounds__(kPT) void compact_piece_kernel(
    const int64_t *__restrict__ off, int64_t n, int64_t NT, const uint8_t *__restrict__ keep,
    PieceParts parts, int64_t nb, CompactCols cols, int n_cols, int64_t *__restrict__ offsets_out,
    int32_t *__restrict__ kept_ids, int64_t *__restrict__ n_kept_tokens, int32_t *__restrict__ reject_ids,
    int64_t budget) {
    constexpr int kPartsPerThread = kPP;
    static_assert(kBlk <= kWave, "a block is handled by one wave");
    __shared__ uint32_t w_cnt[kPW], w_pcs[kPW];
    __shared__ int64_t w_len[kPW];
    __shared__ int64_t sel[3];
    __shared__ int64_t piece[3];
    const int t = threadIdx.x;
    const int64_t q = blockIdx.x;
    if (t == 0) {
        sel[0] = sel[1] = sel[2] = 0;
        piece[0] = piece[1] = piece[2] = 0;   // an unmatched piece copies nothing
    }

    // 1. Exclusive prefix of the block partials; thread t holds blocks
    //    [t * kPartsPerThread, (t + 1) * kPartsPerThread).
    uint32_t c[kPartsPerThread], pc[kPartsPerThread];
    int64_t l[kPartsPerThread];
    uint32_t cs = 0, ps = 0;
    int64_t ls = 0;
#pragma unroll
    for (int k = 0; k < kPartsPerThread; ++k) {
        const int64_t b = (int64_t)t * kPartsPerThread + k;
        c[k] = b < nb ? (uint32_t)parts.cnt[b] : 0u;
        l[k] = b < nb ? parts.len[b] : 0;
        pc[k] = b < nb ? (uint32_t)parts.pcs[b] : 0u;
        cs += c[k];
        ls += l[k];
        ps += pc[k];
    }
    uint32_t tot_c, tot_p;
    int64_t tot_l;
    uint32_t cb = block_excl_sum_u32<kPW>(cs, tot_c, w_cnt);
    int64_t lb = block_excl_sum_i64<kPW>(ls, tot_l, w_len);
    uint32_t pb = block_excl_sum_u32<kPW>(ps, tot_p, w_pcs);
    if (q == 0 && t == 0 && offsets_out) {
        offsets_out[tot_c] = tot_l;
        *n_kept_tokens = tot_l;
    }

    if (q < nb) {
        // 2a. Index outputs of block q.
#pragma unroll
        for (int k = 0; k < kPartsPerThread; ++k) {
            if ((int64_t)t * kPartsPerThread + k == q) {
                sel[0] = cb;
                sel[1] = lb;
            }
            cb += c[k];
            lb += l[k];
        }
        __syncthreads();
        if (t < kWave) {
            const int64_t i = q * kBlk + t;
            const bool in = t < kBlk && i < n;
            int64_t len = 0, lo;
            bool kept = false;
            if (in) {
                const int64_t k = kept_span(off, keep, i, NT, lo);
                kept = k >= 0;
                len = kept ? k : 0;
            }
            const int64_t rank = sel[0] + (int64_t)__popcll(ballot(kept) & lanes_below());
            const int64_t dst = sel[1] + (wave_incl_scan_i64(len) - len);
            if (kept) {
                if (offsets_out) {
                    offsets_out[rank] = dst;
                    kept_ids[rank] = (int32_t)i;
                }
            } else if (in && reject_ids) {
                const int64_t rr = i - rank;       // trajectories before i that were rejected
                if (rr < budget) reject_ids[rr] = (int32_t)i;
            }
        }
        return;
    }

    // 2b. Pieces q - nb, q - nb + stride, ... (stride = piece workgroups in
    //     the grid): for each, its block, then its trajectory in the block.
    const int64_t stride = (int64_t)gridDim.x - nb;
    for (int64_t pq = q - nb; pq < (int64_t)tot_p; pq += stride) {
        __syncthreads();                       // the previous piece's reads of sel/piece are done
        if (t == 0) {
            sel[0] = sel[1] = sel[2] = 0;
            piece[0] = piece[1] = piece[2] = 0;   // an unmatched piece copies nothing
        }
        __syncthreads();
        uint32_t pbk = pb;
        int64_t lbk = lb;
#pragma unroll
        for (int k = 0; k < kPartsPerThread; ++k) {
            const int64_t b = (int64_t)t * kPartsPerThread + k;
            if (b < nb && pc[k] > 0 && (int64_t)pbk <= pq && pq < (int64_t)pbk + pc[k]) {
                sel[0] = b;
                sel[1] = pbk;
                sel[2] = lbk;
            }
            pbk += pc[k];
            lbk += l[k];
        }
        __syncthreads();
        if (t < kWave) {
            const int64_t b = sel[0];
            const int64_t i = b * kBlk + t;
            int64_t len = 0, lo = 0;
            if (t < kBlk && i < n) {
                const int64_t k = kept_span(off, keep, i, NT, lo);
                len = k > 0 ? k : 0;
            }
            const int64_t np = (len + kPieceLen - 1) / kPieceLen;
            const int64_t np_incl = wave_incl_scan_i64(np);
            const int64_t len_incl = wave_incl_scan_i64(len);
            const int64_t qq = pq - sel[1];
            if (np > 0 && np_incl - np <= qq && qq < np_incl) {
                const int64_t k = qq - (np_incl - np);
                piece[0] = sel[2] + (len_incl - len) + k * kPieceLen;
                piece[1] = lo + k * kPieceLen;
                piece[2] = (len - k * kPieceLen) < kPieceLen ? len - k * kPieceLen : kPieceLen;
            }
        }
        __syncthreads();
        const int64_t d = piece[0], s = piece[1];
        int64_t m = piece[2];
        if (d >= NT || m <= 0) continue;        // overlapping (malformed) offsets overflow the output
        if (d + m > NT) m = NT - d;
        for (int col = 0; col < n_cols; ++col) {
            const char *in = (const char *)cols.in[col];
            char *out = (char *)cols.out[col];
            const bool vec = cols.vec[col] != 0;
            switch (cols.elem[col]) {
                case 1: copy_piece<1>(in, out, vec, d, s, m); break;
                case 2: copy_piece<2>(in, out, vec, d, s, m); break;
                case 4: copy_piece<4>(in, out, vec, d, s, m); break;
                default: copy_piece<8>(in, out, vec, d, s, m); break;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Wide path: blocks of kWideBlock trajectories, the copy split by merge path
// ---------------------------------------------------------------------------
// The block partials come in two levels: per block (kept count and tokens)
// and per group of kGroupBlocks blocks (their sums), so that a workgroup
// finds any block's packed position from at most kWideMaxGroups group sums
// and the kGroupBlocks - 1 blocks before it in its group, with wave
// reductions and no scan over all blocks.
//
// The packed output is split evenly by a merge path over the cost (kept
// tokens + kBlockCost per block): workgroup q copies the kept tokens of cost
// range [q S, (q + 1) S), S = ceil(total cost / grid), which holds at most
// S / kBlockCost + 2 blocks, four blocks (one per wave) at a time. Then wave w
// of workgroup q writes the index outputs of block q + w * grid.
constexpr int64_t kBlockCost = 2048;
constexpr int kSpanT = kPT;               // spans in one copy table: four blocks of one wave each
constexpr int kSpanU = 8;                 // 16-byte loads in flight per thread in a span copy
struct SpanTable {
    int32_t start[kSpanT + 1];   // first slot of each span; [kSpanT] = slots in the table
    int64_t dst[kSpanT];         // destination of each span's first slot (bytes or elements)
    int64_t src[kSpanT];         // its source
};

// The span holding slot g: the last span whose first slot is <= g.
__device__ __forceinline__ int span_find(const SpanTable &tb, int32_t g) {
    int j = 0;
#pragma unroll
    for (int step = kSpanT / 2; step > 0; step >>= 1) j = tb.start[j + step] <= g ? j + step : j;
    return j;
}

// Thread t brings span t's range [a, b) and shift del (source - destination)
// in elements; the slots are groups of `per` elements at multiples of `per`
// inside the range, [v0, v1) the part they cover (v0 = v1 when none), so that
// [a, v0) and [v1, b) each hold fewer than `per` elements.
__device__ __forceinline__ void span_table(SpanTable &tb, uint32_t *wsum, int64_t a, int64_t b, int64_t del,
                                           int per, int64_t &v0, int64_t &v1) {
    v0 = (a + per - 1) / per * per;
    v1 = b / per * per;
    if (v1 < v0) v1 = v0;
    if (v0 > b) v0 = v1 = b;
    const uint32_t cnt = (uint32_t)((v1 - v0) / per);
    uint32_t tot;
    const uint32_t ex = block_excl_sum_u32<kPW>(cnt, tot, wsum);
    const int t = threadIdx.x;
    tb.start[t] = (int32_t)ex;
    if (t == kPT - 1) tb.start[kSpanT] = (int32_t)tot;
    tb.dst[t] = v0;
    tb.src[t] = v0 + del;
}

// Columns of 4- or 8-byte elements with 16-byte aligned pointers: the slots
// are the aligned 16-byte destination vectors (sources at least 4-byte
// aligned, one dwordx4 load each); each thread then copies the elements at
// its own range's ends (fewer than 16 bytes at each end, all loads first).
template <int E>
__device__ void copy_spans_vec(const char *__restrict__ in, char *__restrict__ out, int64_t a, int64_t b,
                               int64_t del, SpanTable &tb, uint32_t *wsum) {
    using T = typename Elem<E>::T;
    constexpr int VE = 16 / E;
    const T *src = reinterpret_cast<const T *>(in);
    T *dst = reinterpret_cast<T *>(out);
    const int t = threadIdx.x;
    __syncthreads();                           // the previous table is no longer read
    int64_t v0, v1;
    span_table(tb, wsum, a, b, del, VE, v0, v1);
    __syncthreads();
    const int32_t total = tb.start[kSpanT];
    for (int32_t g0 = t; g0 < total; g0 += kSpanU * kPT) {
        uint4 x[kSpanU];
#pragma unroll
        for (int u = 0; u < kSpanU; ++u) {
            const int32_t g = g0 + u * kPT;
            if (g < total) {
                const int j = span_find(tb, g);
                x[u] = load_a4(src + tb.src[j] + (int64_t)(g - tb.start[j]) * VE);
            }
        }
#pragma unroll
        for (int u = 0; u < kSpanU; ++u) {
            const int32_t g = g0 + u * kPT;
            if (g < total) {
                const int j = span_find(tb, g);
                store_nt(reinterpret_cast<uint4 *>(dst + tb.dst[j] + (int64_t)(g - tb.start[j]) * VE), x[u]);
            }
        }
    }
    T h[VE - 1], e[VE - 1];
#pragma unroll
    for (int k = 0; k < VE - 1; ++k) {
        if (a + k < v0) h[k] = src[a + k + del];
        if (v1 + k < b) e[k] = src[v1 + k + del];
    }
#pragma unroll
    for (int k = 0; k < VE - 1; ++k) {
        if (a + k < v0) dst[a + k] = h[k];
        if (v1 + k < b) dst[v1 + k] = e[k];
    }
}

// Any other column: one element per slot.
template <int E>
__device__ void copy_spans_elem(const char *__restrict__ in, char *__restrict__ out, int64_t a, int64_t b,
                                int64_t del, SpanTable &tb, uint32_t *wsum) {
    using T = typename Elem<E>::T;
    const T *src = reinterpret_cast<const T *>(in);
    T *dst = reinterpret_cast<T *>(out);
    const int t = threadIdx.x;
    __syncthreads();
    int64_t v0, v1;
    span_table(tb, wsum, a, b, del, 1, v0, v1);
    __syncthreads();
    const int32_t total = tb.start[kSpanT];
    for (int32_t g = t; g < total; g += kPT) {
        const int j = span_find(tb, g);
        const int64_t r = g - tb.start[j];
        dst[tb.dst[j] + r] = src[tb.src[j] + r];
    }
}

// Range [a, b) of a column, shift del, in elements.
__device__ __forceinline__ void copy_spans_col(const CompactCols &cols, int col, int64_t a, int64_t b, int64_t del,
                                               SpanTable &tb, uint32_t *wsum) {
    const char *in = (const char *)cols.in[col];
    char *out = (char *)cols.out[col];
    const bool vec = cols.vec[col] != 0;
    switch (cols.elem[col]) {
        case 1: copy_spans_elem<1>(in, out, a, b, del, tb, wsum); break;
        case 2: copy_spans_elem<2>(in, out, a, b, del, tb, wsum); break;
        case 4:
            if (vec) copy_spans_vec<4>(in, out, a, b, del, tb, wsum);
            else copy_spans_elem<4>(in, out, a, b, del, tb, wsum);
            break;
        default:
            if (vec) copy_spans_vec<8>(in, out, a, b, del, tb, wsum);
            else copy_spans_elem<8>(in, out, a, b, del, tb, wsum);
            break;
    }
}

// One workgroup of 1024 threads per kGroupBlocks blocks of kWideBlock
// trajectories (one wave each): the block partials from the keep flags and
// the group's sums.
__global__ __launch_bounds__(kWideBlock * kGroupBlocks) void compact_partials_wide_kernel(
    const int64_t *__restrict__ off, int64_t n, int64_t NT, const uint8_t *__restrict__ keep, PieceParts parts) {
    static_assert(kWideBlock == kWave, "a wide block is one wave");
    __shared__ uint32_t sc[kGroupBlocks];
    __shared__ int64_t sl[kGroupBlocks];
    const int lane = lane_id(), w = threadIdx.x / kWave;
    const int64_t b = (int64_t)blockIdx.x * kGroupBlocks + w;
    const int64_t i = b * kWideBlock + lane;
    int64_t len = 0, lo;
    bool kept = false;
    if (i < n) {
        const int64_t k = kept_span(off, keep, i, NT, lo);
        kept = k >= 0;
        len = kept ? k : 0;
    }
    const uint32_t c = (uint32_t)__popcll(ballot(kept));
    const int64_t l = wave_sum_i64(len);
    if (lane == 0) {
        if (b * kWideBlock < n) {
            parts.cnt[b] = (int32_t)c;
            parts.len[b] = l;
        }
        sc[w] = c;
        sl[w] = l;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t gc = 0;
        int64_t gl = 0;
        for (int k = 0; k < kGroupBlocks; ++k) {
            gc += sc[k];
            gl += sl[k];
        }
        parts.gcnt[blockIdx.x] = (int32_t)gc;
        parts.glen[blockIdx.x] = gl;
    }
}

// nb blocks in ng = ceil(nb / kGroupBlocks) <= kWideMaxGroups groups;
// 4 * grid >= nb. offsets_out, kept_ids and n_kept_tokens may be null
// (rejected ids only).
__global__ __launch_bounds__(kPT) void compact_wide_kernel(
    const int64_t *__restrict__ off, int64_t n, int64_t NT, const uint8_t *__restrict__ keep,
    PieceParts parts, int64_t nb, CompactCols cols, int n_cols, int64_t *__restrict__ offsets_out,
    int32_t *__restrict__ kept_ids, int64_t *__restrict__ n_kept_tokens, int32_t *__restrict__ reject_ids,
    int64_t budget) {
    static_assert(kWideBlock == kWave, "a wide block is one wave");
    static_assert(kWideMaxGroups == 4 * kWave, "group sums: four per lane of one wave");
    __shared__ int64_t s_gl[kWideMaxGroups + 1];   // kept tokens before each group; [kWideMaxGroups] = total
    __shared__ uint32_t s_gc[kWideMaxGroups + 1];  // kept trajectories before each group
    __shared__ int64_t s_cut[6];                   // b0, b1, x0, x1
    __shared__ uint32_t wsum[kPW];
    __shared__ SpanTable tb;
    const int t = threadIdx.x, w = t / kWave, lane = lane_id();
    const int64_t q = blockIdx.x, G = gridDim.x;
    const int64_t ng = (nb + kGroupBlocks - 1) / kGroupBlocks;

    // The block `b`'s kept count and tokens before it inside its group: the
    // wave's lanes below kGroupBlocks hold the group's earlier blocks.
    auto in_group = [&](int64_t b, uint32_t &c, int64_t &l) {
        const int64_t j = b / kGroupBlocks * kGroupBlocks + lane;
        c = 0u;
        l = 0;
        if (lane < kGroupBlocks && j < b) {
            c = (uint32_t)parts.cnt[j];
            l = parts.len[j];
        }
    };

    // 0. The index block of this wave: its spans and its group's earlier
    //    partials, loaded with the group sums (one round trip).
    const int64_t ib = q + (int64_t)w * G;
    int64_t i_lo = 0, i_len = -1;
    uint32_t i_c = 0u;
    int64_t i_l = 0;
    if (ib < nb) {
        const int64_t i = ib * kWideBlock + lane;
        if (i < n) {
            const uint8_t kf = keep[i];
            const int64_t a = off[i], b = off[i + 1];
            if (kf != 0) {
                i_lo = clamp64(a, 0, NT);
                const int64_t hi = clamp64(b, 0, NT);
                i_len = hi > i_lo ? hi - i_lo : 0;
            }
        }
        in_group(ib, i_c, i_l);
    }

    // 1. Exclusive prefixes of the group sums (wave 0, four groups per lane).
    if (w == 0) {
        uint32_t c4[4];
        int64_t l4[4];
        uint32_t cs = 0u;
        int64_t ls = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int64_t g = (int64_t)lane * 4 + k;
            c4[k] = g < ng ? (uint32_t)parts.gcnt[g] : 0u;
            l4[k] = g < ng ? parts.glen[g] : 0;
            cs += c4[k];
            ls += l4[k];
        }
        uint32_t ce = wave_incl_scan_u32(cs) - cs;
        int64_t le = wave_incl_scan_i64(ls) - ls;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            s_gc[lane * 4 + k] = ce;
            s_gl[lane * 4 + k] = le;
            ce += c4[k];
            le += l4[k];
        }
        if (lane == kWave - 1) {
            s_gc[kWideMaxGroups] = ce;
            s_gl[kWideMaxGroups] = le;
        }
    }
    __syncthreads();
    const int64_t tot_l = s_gl[kWideMaxGroups];

    // 2. Copy the kept tokens of cost range [q S, (q + 1) S). Wave 0 finds the
    //    blocks holding costs c0, c1 - 1 and c1: per cost, a binary search over
    //    the groups' cost starts, then lanes 16u .. 16u + 15 scan that group's
    //    block lengths (row u of the wave).
    const int64_t T = tot_l + kBlockCost * nb;
    const int64_t S = (T + G - 1) / G;
    const int64_t c0 = q * S;
    if (n_cols > 0 && nb > 0 && c0 < T) {
        const int64_t c1 = (c0 + S < T) ? c0 + S : T;
        if (w == 0) {
            const int u = lane / kGroupBlocks, r = lane % kGroupBlocks;
            const int64_t key = u == 0 ? c0 : (u == 1 ? c1 - 1 : c1);
            int64_t lo = 0, hi = ng;                // last group whose cost starts at or before key
            while (hi - lo > 1) {
                const int64_t mid = (lo + hi) / 2;
                if (s_gl[mid] + kBlockCost * kGroupBlocks * mid <= key) lo = mid;
                else hi = mid;
            }
            const int64_t j = lo * kGroupBlocks + r;
            const int64_t len = (u < 3 && j < nb) ? parts.len[j] : 0;
            const int64_t before = s_gl[lo] + (row_incl_scan_i64(len) - len);
            const int64_t cst = before + kBlockCost * j;   // cost start of block j
            const bool ok = u < 3 && j < nb && cst <= key;
            const uint64_t m = ballot(ok);
            const uint32_t row = (uint32_t)(m >> (16 * u)) & 0xffffu;
            const bool last = ok && (row >> (r + 1)) == 0u;
            if (last) {
                if (u == 0) s_cut[0] = j;
                if (u == 1) s_cut[1] = j;
                const int64_t rr = key - cst - kBlockCost;
                const int64_t x = before + (rr < 0 ? 0 : (rr > len ? len : rr));
                if (u == 0) s_cut[2] = x;
                if (u == 2) s_cut[3] = x;
            }
        }
        __syncthreads();
        const int64_t b0 = s_cut[0], b1 = s_cut[1], x0 = s_cut[2], x1 = s_cut[3];
        for (int64_t bg = b0; x0 < x1 && bg <= b1; bg += kPW) {
            // Wave w: block bg + w, lane j its trajectory j; the part of its
            // kept span inside [x0, x1).
            const int64_t b = bg + w;
            int64_t a = 0, e = 0, del = 0;
            if (b <= b1) {
                const int64_t i = b * kWideBlock + lane;
                int64_t len = 0, lo_i = 0;
                if (i < n) {
                    const int64_t k = kept_span(off, keep, i, NT, lo_i);
                    len = k > 0 ? k : 0;
                }
                uint32_t gc;
                int64_t gl;
                in_group(b, gc, gl);
                const int64_t lb = s_gl[b / kGroupBlocks] + wave_sum_i64(gl);
                const int64_t dst = lb + (wave_incl_scan_i64(len) - len);
                const int64_t s0 = dst > x0 ? dst : x0;
                const int64_t s1 = (dst + len < x1) ? dst + len : x1;
                if (s1 > s0) {
                    a = s0;
                    e = s1 < NT ? s1 : NT;             // overlapping (malformed) offsets overflow the output
                    if (a > e) a = e;
                    del = lo_i - dst;
                }
            }
            for (int col = 0; col < n_cols; ++col) copy_spans_col(cols, col, a, e, del, tb, wsum);
        }
    }

    // 3. Index outputs of block ib (after the copy: their stores would hold
    //    up the copy's first loads, one counter covering both).
    if (q == 0 && t == 0 && offsets_out) {
        offsets_out[s_gc[kWideMaxGroups]] = tot_l;
        *n_kept_tokens = tot_l;
    }
    if (ib < nb) {
        const int64_t i = ib * kWideBlock + lane;
        const bool kept = i_len >= 0;
        const int64_t len = kept ? i_len : 0;
        const int64_t g = ib / kGroupBlocks;
        const int64_t cb = (int64_t)s_gc[g] + (int64_t)wave_sum_u64((uint64_t)i_c);
        const int64_t lb = s_gl[g] + wave_sum_i64(i_l);
        const int64_t rank = cb + (int64_t)__popcll(ballot(kept) & lanes_below());
        const int64_t dst = lb + (wave_incl_scan_i64(len) - len);
        if (kept) {
            if (offsets_out) {
                offsets_out[rank] = dst;
                kept_ids[rank] = (int32_t)i;
            }
        } else if (i < n && reject_ids) {
            const int64_t rr = i - rank;           // trajectories before i that were rejected
            if (rr < budget) reject_ids[rr] = (int32_t)i;
        }
    }
}

// ---------------------------------------------------------------------------
// Scan path
// ---------------------------------------------------------------------------
// hdr[0] = n_kept, hdr[1] = min(total kept tokens, n_tokens)
__global__ __launch_bounds__(kT) void compact_scan_kernel(
    const int64_t *__restrict__ off, int64_t n, int64_t NT, const uint8_t *__restrict__ keep,
    int64_t *__restrict__ offsets_out, int32_t *__restrict__ kept_ids,
    int64_t *__restrict__ n_kept_tokens, int64_t *__restrict__ kept_src,
    int32_t *__restrict__ chunk_first, int64_t map_cap, int64_t *__restrict__ hdr) {
    __shared__ uint32_t wcnt[kNW];
    __shared__ int64_t wlen[kNW];
    int64_t run_cnt = 0, run_len = 0;
    for (int64_t base = 0; base < n; base += kT) {
        const int64_t i = base + threadIdx.x;
        const bool in = i < n;
        const bool k = in && keep[i] != 0;
        int64_t lo = 0, len = 0;
        if (k) {
            lo = clamp64(off[i], 0, NT);
            const int64_t hi = clamp64(off[i + 1], 0, NT);
            len = hi > lo ? hi - lo : 0;
        }
        uint32_t tc;
        const uint32_t r = block_excl_sum_u32<kNW>(k ? 1u : 0u, tc, wcnt);
        int64_t tl;
        const int64_t d = block_excl_sum_i64<kNW>(len, tl, wlen);
        if (k) {
            const int64_t rank = run_cnt + r;
            const int64_t dst = run_len + d;
            offsets_out[rank] = dst;
            kept_ids[rank] = (int32_t)i;
            kept_src[rank] = lo;
            int64_t end = dst + len;
            if (end > NT) end = NT;
            for (int64_t c = (dst + kCopyChunk - 1) / kCopyChunk; c * kCopyChunk < end && c < map_cap; ++c)
                chunk_first[c] = (int32_t)rank;
        }
        run_cnt += tc;
        run_len += tl;
    }
    if (threadIdx.x == 0) {
        offsets_out[run_cnt] = run_len;
        *n_kept_tokens = run_len;
        hdr[0] = run_cnt;
        hdr[1] = run_len < NT ? run_len : NT;
    }
}

__global__ __launch_bounds__(256) void compact_copy_kernel(
    CompactCols cols, const int64_t *__restrict__ oo, const int64_t *__restrict__ ss,
    const int32_t *__restrict__ chunk_first, const int64_t *__restrict__ hdr, int64_t NT) {
    const int col = blockIdx.y;
    const int64_t n_kept = hdr[0];
    const int64_t total = hdr[1];
    if (n_kept <= 0) return;
    const int64_t n_chunks = (total + kCopyChunk - 1) / kCopyChunk;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x / kWave);
    for (int64_t c = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave; c < n_chunks; c += waves) {
        const int64_t cs = c * kCopyChunk;
        const int64_t ce = (cs + kCopyChunk < total) ? cs + kCopyChunk : total;
        const int64_t j = clamp64(chunk_first[c], 0, n_kept - 1);
        GlobalSpans sp{oo, ss, n_kept, 0, 0, 0};
        sp.load(j);
        copy_range_col(cols, col, sp, n_kept, NT, cs, ce, j);
    }
}

}  // namespace

int64_t map_capacity(int64_t n_tokens) { return (n_tokens + kCopyChunk - 1) / kCopyChunk + 1; }

CompactWs compact_ws_carve(void *ws, int64_t n, int64_t n_tokens) {
    const size_t nb = (size_t)piece_blocks(n);
    char *p = (char *)ws;
    CompactWs w;
    w.hdr = (int64_t *)p;          p += 256;
    w.kept_src = (int64_t *)p;     p += align256((size_t)n * 8);
    w.chunk_first = (int32_t *)p;  p += align256((size_t)map_capacity(n_tokens) * 4);
    w.parts.cnt = (int32_t *)p;    p += align256(nb * 4);
    w.parts.len = (int64_t *)p;    p += align256(nb * 8);
    w.parts.pcs = (int32_t *)p;    p += align256(nb * 4);
    const size_t ng = (size_t)wide_groups(n);
    w.parts.gcnt = (int32_t *)p;   p += align256(ng * 4);
    w.parts.glen = (int64_t *)p;
    return w;
}

size_t compact_ws_bytes(int64_t n, int64_t n_tokens) {
    const size_t nb = (size_t)piece_blocks(n);
    const size_t ng = (size_t)wide_groups(n);
    return 256 + align256((size_t)n * 8) + align256((size_t)map_capacity(n_tokens) * 4) +
           align256(nb * 4) * 2 + align256(nb * 8) + align256(ng * 4) + align256(ng * 8);
}

bool compact_piece_ok(int64_t n, int64_t n_tokens) {
    return n <= kPieceMaxN && n_tokens / kPieceLen < ((int64_t)1 << 30);
}

bool compact_wide_ok(int64_t n, int64_t n_tokens) {
    return n <= kWideMaxN && n_tokens / kPieceLen < ((int64_t)1 << 30);
}

hipError_t launch_compact_partials(const int64_t *offsets, int64_t n, int64_t n_tokens,
                                   const uint8_t *keep, const PieceParts &parts, hipStream_t stream,
                                   int blk) {
    if (n == 0) return hipSuccess;
    if (blk == kWideBlock)
        return launch(-1, compact_partials_wide_kernel,
                      dim3((unsigned)((n + kWideBlock * kGroupBlocks - 1) / (kWideBlock * kGroupBlocks))),
                      dim3(kWideBlock * kGroupBlocks), stream, offsets, n, n_tokens, keep, parts);
    return launch(-1, compact_partials_kernel<kPieceBlock>, dim3((unsigned)piece_blocks(n)), dim3(kWave), stream,
                  offsets, n, n_tokens, keep, parts);
}

hipError_t launch_compact_pieces(const int64_t *offsets, int64_t n, int64_t n_tokens, const uint8_t *keep,
                                 const PieceParts &parts, const CompactCols &cols, int n_cols,
                                 int64_t *offsets_out, int32_t *kept_ids, int64_t *n_kept_tokens,
                                 int32_t *reject_ids, int64_t budget, int64_t max_kept,
                                 hipStream_t stream, int blk, bool copy) {
    // Block workgroups, then the piece workgroups: a kept span of len tokens
    // has at most len / kPieceLen + 1 pieces, so all kept spans together have
    // at most max_kept + n_tokens / kPieceLen.
    // Past one resident round of workgroups (8 per CU) the piece workgroups
    // loop over the pieces instead.
    const int64_t nb = (n + blk - 1) / blk;
    const int64_t kept_bound = max_kept < 0 ? 0 : (max_kept > n ? n : max_kept);
    int64_t piece_wgs = copy ? kept_bound + n_tokens / kPieceLen + 1 : 0;
    const int64_t round = resident_waves() / 16 * 8 - nb;
    if (round > 0 && piece_wgs > round) piece_wgs = round;
    if (copy && piece_wgs < 1) piece_wgs = 1;
    const int64_t grid = (nb > 0 ? nb : 1) + piece_wgs;
    const int64_t per = (nb + kPT - 1) / kPT;
#define PACE_PIECES(B, P)                                                                                      \
    return launch(kPhaseCompact, compact_piece_kernel<B, P>, dim3((unsigned)grid), dim3(kPT), stream, offsets, n, \
                  n_tokens, keep, parts, nb, cols, copy ? n_cols : 0, offsets_out, kept_ids, n_kept_tokens,      \
                  reject_ids, budget)
    if (blk == kPieceBlock) {
        if (per > 2) return hipErrorInvalidValue;
        PACE_PIECES(kPieceBlock, 2);
    }
#undef PACE_PIECES
    if (blk != kWideBlock || (nb + kGroupBlocks - 1) / kGroupBlocks > kWideMaxGroups) return hipErrorInvalidValue;
    // Every workgroup indexes up to four blocks and copies an even share of
    // the output: one resident round (four per CU) when copying.
    int64_t wgs = (nb + kPW - 1) / kPW;
    if (copy && wgs < resident_waves() / 16 * 4) wgs = resident_waves() / 16 * 4;
    if (wgs < 1) wgs = 1;
    return launch(kPhaseCompact, compact_wide_kernel, dim3((unsigned)wgs), dim3(kPT), stream, offsets, n, n_tokens,
                  keep, parts, nb, cols, copy ? n_cols : 0, offsets_out, kept_ids, n_kept_tokens, reject_ids, budget);
}

hipError_t launch_compact_copy(const CompactCols &cols, int n_cols, int64_t n_tokens,
                               const int64_t *offsets_out, const CompactWs &w, hipStream_t stream) {
    if (n_cols == 0 || n_tokens == 0) return hipSuccess;
    const int64_t max_chunks = (n_tokens + kCopyChunk - 1) / kCopyChunk;
    int64_t blocks = (max_chunks + 3) / 4;
    if (blocks > 1024) blocks = 1024;
    if (blocks < 1) blocks = 1;
    dim3 grid((unsigned)blocks, (unsigned)n_cols);
    return launch(kPhaseCompact, compact_copy_kernel, grid, dim3(256), stream, cols, offsets_out,
                  w.kept_src, w.chunk_first, w.hdr, n_tokens);
}

hipError_t launch_compact(const int64_t *offsets, int64_t n, int64_t n_tokens, const uint8_t *keep,
                          const CompactCols &cols, int n_cols, int64_t *offsets_out,
                          int32_t *kept_ids, int64_t *n_kept_tokens, void *ws, hipStream_t stream) {
    CompactWs w = compact_ws_carve(ws, n, n_tokens);
    if (compact_piece_ok(n, n_tokens) || compact_wide_ok(n, n_tokens)) {
        const int blk = compact_piece_ok(n, n_tokens) ? kPieceBlock : kWideBlock;
        hipError_t e = launch_compact_partials(offsets, n, n_tokens, keep, w.parts, stream, blk);
        if (e != hipSuccess) return e;
        return launch_compact_pieces(offsets, n, n_tokens, keep, w.parts, cols, n_cols, offsets_out,
                                     kept_ids, n_kept_tokens, nullptr, 0, n, stream, blk, true);
    }
    compact_scan_kernel<<<1, kT, 0, stream>>>(offsets, n, n_tokens, keep, offsets_out, kept_ids,
                                             n_kept_tokens, w.kept_src, w.chunk_first,
                                             map_capacity(n_tokens), w.hdr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_compact_copy(cols, n_cols, n_tokens, offsets_out, w, stream);
}

}  // namespace pace
