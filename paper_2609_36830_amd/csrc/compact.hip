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
// Wide blocks (kWideBlock = 64 trajectories, pools up to kWideMaxN): the kept
// spans of a block are mostly short, so one span per piece would leave every
// piece workgroup mostly set-up. Spans longer than kPieceLen still make
// pieces; the shorter ones of a block are copied together as segments of
// kSegLen tokens: the block's own workgroup copies the first right after its
// index outputs, piece workgroups the rest. A segment copy lays a table of
// 16-byte destination slots over its spans in LDS, so each thread keeps
// several loads in flight whatever the span lengths.
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
// flags (pieces as wide_block_pieces counts them for wide blocks).
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
    const int64_t pc = kBlk == kWideBlock
        ? wide_block_pieces(wave_sum_i64(len > kPieceLen ? (len + kPieceLen - 1) / kPieceLen : 0),
                            wave_sum_i64(len > kPieceLen ? 0 : len))
        : wave_sum_i64((len + kPieceLen - 1) / kPieceLen);
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

// The workgroup copies one segment of a wide block: lane j of wave 0 brings
// destination range [a, b) of span j (empty when span j has no part in the
// segment) and del = source - destination, in elements. The slots are, for
// columns of 4- or 8-byte elements with 16-byte aligned pointers, the aligned
// 16-byte destination vectors inside each range (in bytes; sources are at
// least 4-byte aligned), else single elements; a segment has at most kSegLen
// elements. The slots' prefix over the spans goes to LDS; each thread takes
// slots t, t + kPT, ... (kSegU loads in flight, each slot's span by a
// six-step binary search), and with vectors the lanes of wave 0 copy the few
// bytes at their range's ends.
constexpr int kSegU = 8;
struct SegTable {
    int32_t start[kWave + 1];   // first slot of each span; [kWave] = slots in the segment
    int64_t dst[kWave];         // destination of each span's first slot (bytes or elements)
    int64_t src[kWave];         // its source
};

// Span j holding slot g.
__device__ __forceinline__ int seg_find(const SegTable &tb, int32_t g) {
    int j = 0;
#pragma unroll
    for (int step = kWave / 2; step > 0; step >>= 1) j = tb.start[j + step] <= g ? j + step : j;
    return j;
}

// Builds the slot table (wave 0) from per-lane ranges [a, b) in units of
// `unit` and source shift del; slots are groups of `per` units at multiples
// of `per`, units outside them go through `edge` (called by the lane).
template <typename Edge>
__device__ __forceinline__ void seg_table(SegTable &tb, int64_t a, int64_t b, int64_t del, int per, Edge edge) {
    int64_t v0 = (a + per - 1) / per, v1 = b / per;
    if (v1 < v0) v1 = v0;
    const int32_t cnt = (int32_t)(v1 - v0);
    const int32_t incl = (int32_t)wave_incl_scan_u32((uint32_t)cnt);
    const int t = threadIdx.x;
    tb.start[t] = incl - cnt;
    if (t == kWave - 1) tb.start[kWave] = incl;
    tb.dst[t] = v0 * per;
    tb.src[t] = v0 * per + del;
    const int64_t h = cnt > 0 ? v0 * per : b;
    for (int64_t p = a; p < h; ++p) edge(p);
    if (cnt > 0)
        for (int64_t p = v1 * per; p < b; ++p) edge(p);
}

// 16-byte vector slots over byte ranges.
__device__ void copy_segment_vec(const char *__restrict__ in, char *__restrict__ out, int64_t a, int64_t b,
                                 int64_t del, SegTable &tb) {
    const int t = threadIdx.x;
    __syncthreads();                           // the previous column's table is no longer read
    if (t < kWave) seg_table(tb, a, b, del, 16, [&](int64_t p) { out[p] = in[p + del]; });
    __syncthreads();
    const int32_t total = tb.start[kWave];
    for (int32_t g0 = t; g0 < total; g0 += kSegU * kPT) {
        uint32_t jr[kSegU];                    // span << 26 | slot in span; ~0: none
        uint4 x[kSegU];
#pragma unroll
        for (int u = 0; u < kSegU; ++u) {
            const int32_t g = g0 + u * kPT;
            jr[u] = ~0u;
            if (g < total) {
                const int j = seg_find(tb, g);
                const int32_t r = g - tb.start[j];
                jr[u] = ((uint32_t)j << 26) | (uint32_t)r;
                x[u] = load_a4(in + tb.src[j] + (int64_t)r * 16);
            }
        }
#pragma unroll
        for (int u = 0; u < kSegU; ++u)
            if (jr[u] != ~0u)
                store_nt(reinterpret_cast<uint4 *>(out + tb.dst[jr[u] >> 26] + (int64_t)(jr[u] & 0x3ffffffu) * 16),
                         x[u]);
    }
}

// Single-element slots.
template <int E>
__device__ void copy_segment_elem(const char *__restrict__ in, char *__restrict__ out, int64_t a, int64_t b,
                                  int64_t del, SegTable &tb) {
    using T = typename Elem<E>::T;
    const T *src = reinterpret_cast<const T *>(in);
    T *dst = reinterpret_cast<T *>(out);
    const int t = threadIdx.x;
    __syncthreads();
    if (t < kWave) seg_table(tb, a, b, del, 1, [&](int64_t) {});
    __syncthreads();
    const int32_t total = tb.start[kWave];
    for (int32_t g = t; g < total; g += kPT) {
        const int j = seg_find(tb, g);
        const int64_t r = g - tb.start[j];
        dst[tb.dst[j] + r] = src[tb.src[j] + r];
    }
}

__device__ __forceinline__ void copy_segment_col(const CompactCols &cols, int col, int64_t a, int64_t b, int64_t del,
                                                 SegTable &tb) {
    const char *in = (const char *)cols.in[col];
    char *out = (char *)cols.out[col];
    const int E = cols.elem[col];
    if (cols.vec[col] != 0 && E >= 4) {
        copy_segment_vec(in, out, a * E, b * E, del * E, tb);
        return;
    }
    switch (E) {
        case 1: copy_segment_elem<1>(in, out, a, b, del, tb); break;
        case 2: copy_segment_elem<2>(in, out, a, b, del, tb); break;
        case 4: copy_segment_elem<4>(in, out, a, b, del, tb); break;
        default: copy_segment_elem<8>(in, out, a, b, del, tb); break;
    }
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
    // Wide block workgroups: the block's spans, loaded with the partials
    // (flag and offsets together: one round trip). len -1: rejected.
    int64_t b_lo = 0, b_len = -1;
    if constexpr (kBlk == kWideBlock) {
        const int64_t i = q * kBlk + t;
        if (q < nb && t < kWave && i < n) {
            const uint8_t kf = keep[i];
            const int64_t a = off[i], b = off[i + 1];
            if (kf != 0) {
                b_lo = clamp64(a, 0, NT);
                const int64_t hi = clamp64(b, 0, NT);
                b_len = hi > b_lo ? hi - b_lo : 0;
            }
        }
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
        int64_t a = 0, e = 0, del = 0;         // wide: span t's part of the block's first segment
        if (t < kWave) {
            const int64_t i = q * kBlk + t;
            const bool in = t < kBlk && i < n;
            int64_t len = 0, lo = 0;
            bool kept = false;
            if constexpr (kBlk == kWideBlock) {
                kept = b_len >= 0;
                len = kept ? b_len : 0;
                lo = b_lo;
            } else if (in) {
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
            if constexpr (kBlk == kWideBlock) {
                const int64_t sl = len > kPieceLen ? 0 : len;
                const int64_t f = wave_incl_scan_i64(sl) - sl;
                const int64_t fb = (f + sl < kSegLen) ? f + sl : kSegLen;
                if (fb > f) {
                    a = dst;
                    e = dst + (fb - f);
                    del = lo - dst;
                    if (e > NT) e = NT;                // overlapping (malformed) offsets overflow the output
                    if (a > e) a = e;
                }
            }
        }
        if constexpr (kBlk == kWideBlock) {
            __shared__ SegTable tb0;
            for (int col = 0; col < n_cols; ++col) copy_segment_col(cols, col, a, e, del, tb0);
        }
        return;
    }

    // 2b. Pieces q - nb, q - nb + stride, ... (stride = piece workgroups in
    //     the grid): for each, its block, then its trajectory in the block
    //     (wide blocks: a piece of a long span, or a segment of the short ones
//     after the first, which the block's workgroup copies).
    const int64_t stride = (int64_t)gridDim.x - nb;
    if constexpr (kBlk == kWideBlock) {
        __shared__ SegTable tb;
        __shared__ int sg_mode;
        // The blocks' piece and token prefixes move to LDS, so that no
        // register holds them while the pieces are copied.
        __shared__ uint32_t s_pb[kPT * kPartsPerThread + 1];
        __shared__ int64_t s_lb[kPT * kPartsPerThread];
        {
            uint32_t pbk = pb;
            int64_t lbk = lb;
#pragma unroll
            for (int k = 0; k < kPartsPerThread; ++k) {
                s_pb[t * kPartsPerThread + k] = pbk;
                s_lb[t * kPartsPerThread + k] = lbk;
                pbk += pc[k];
                lbk += l[k];
            }
            if (t == kPT - 1) s_pb[kPT * kPartsPerThread] = pbk;
        }
        for (int64_t pq = q - nb; pq < (int64_t)tot_p; pq += stride) {
            __syncthreads();                   // the previous piece's reads of sel/piece/sg_mode are done
            if (t == 0) {
                sel[0] = sel[1] = sel[2] = 0;
                piece[0] = piece[1] = piece[2] = 0;
                sg_mode = 0;
            }
            __syncthreads();
#pragma unroll
            for (int k = 0; k < kPartsPerThread; ++k) {
                const int b = t * kPartsPerThread + k;
                const uint32_t p0 = s_pb[b], p1 = s_pb[b + 1];
                if (b < nb && (int64_t)p0 <= pq && pq < (int64_t)p1) {
                    sel[0] = b;
                    sel[1] = p0;
                    sel[2] = s_lb[b];
                }
            }
            __syncthreads();
            int64_t a = 0, e = 0, del = 0;     // wave 0, lane j: span j's destination range and shift
            if (t < kWave) {
                const int64_t i = sel[0] * kBlk + t;
                int64_t len = 0, lo = 0;
                if (i < n) {
                    const int64_t k = kept_span(off, keep, i, NT, lo);
                    len = k > 0 ? k : 0;
                }
                const int64_t dst = sel[2] + (wave_incl_scan_i64(len) - len);
                const bool lng = len > kPieceLen;
                const int64_t np = lng ? (len + kPieceLen - 1) / kPieceLen : 0;
                const int64_t np_incl = wave_incl_scan_i64(np);
                const int64_t n_long = readlane_i64(np_incl, kWave - 1);
                const int64_t qq = pq - sel[1];
                if (qq < n_long) {
                    if (np > 0 && np_incl - np <= qq && qq < np_incl) {
                        const int64_t k = qq - (np_incl - np);
                        piece[0] = dst + k * kPieceLen;
                        piece[1] = lo + k * kPieceLen;
                        piece[2] = (len - k * kPieceLen) < kPieceLen ? len - k * kPieceLen : kPieceLen;
                    }
                    if (t == 0) sg_mode = 1;
                } else {
                    const int64_t sl = lng ? 0 : len;
                    const int64_t f = wave_incl_scan_i64(sl) - sl;     // span's start among the short tokens
                    const int64_t s0 = (qq - n_long + 1) * kSegLen, s1 = s0 + kSegLen;
                    const int64_t fa = f > s0 ? f : s0, fb = (f + sl < s1) ? f + sl : s1;
                    if (fb > fa) {
                        a = dst + (fa - f);
                        e = dst + (fb - f);
                        del = lo - dst;
                        if (e > NT) e = NT;            // overlapping (malformed) offsets overflow the output
                        if (a > e) a = e;
                    }
                    if (t == 0) sg_mode = 2;
                }
            }
            __syncthreads();
            const int mode = sg_mode;
            if (mode == 2) {
                for (int col = 0; col < n_cols; ++col) copy_segment_col(cols, col, a, e, del, tb);
                continue;
            }
            const int64_t d = piece[0], s = piece[1];
            int64_t m = piece[2];
            if (mode != 1 || d >= NT || m <= 0) continue;
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
        return;
    }
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
    w.parts.pcs = (int32_t *)p;
    return w;
}

size_t compact_ws_bytes(int64_t n, int64_t n_tokens) {
    const size_t nb = (size_t)piece_blocks(n);
    return 256 + align256((size_t)n * 8) + align256((size_t)map_capacity(n_tokens) * 4) +
           align256(nb * 4) * 2 + align256(nb * 8);
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
        return launch(-1, compact_partials_kernel<kWideBlock>, dim3((unsigned)((n + kWideBlock - 1) / kWideBlock)),
                      dim3(kWave), stream, offsets, n, n_tokens, keep, parts);
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
    if (blk != kWideBlock || per > 16) return hipErrorInvalidValue;
    if (per <= 2) PACE_PIECES(kWideBlock, 2);
    if (per <= 4) PACE_PIECES(kWideBlock, 4);
    if (per <= 8) PACE_PIECES(kWideBlock, 8);
    PACE_PIECES(kWideBlock, 16);
#undef PACE_PIECES
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
