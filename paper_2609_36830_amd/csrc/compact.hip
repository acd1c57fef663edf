// pace_compact kernels for gfx950: pack the kept trajectories' token spans
// into the training batch (Algorithm 1), survivors in pool order.
//
// Copy routine (both paths): a wave copies a contiguous range of output
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
// Span path (n <= kSpanMaxN, n_tokens < 2^31): ONE kernel. Every 1024-thread
// workgroup (one per CU) first rebuilds the ordered scan of keep flags and
// kept lengths for the whole pool in LDS -- a few kilobytes from L2, one
// block scan -- then its waves copy equal shares of the packed batch,
// locating their first span by a search in LDS. Workgroup 0 also writes the
// packed offsets, kept ids, the kept-token count and (when asked) the
// rejected ids.
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

// LDS arrays (int32: the span path requires n_tokens < 2^31).
struct LdsSpans {
    const int32_t *kdst;   // [n_kept + 1]
    const int32_t *ksrc;   // [n_kept]
    __device__ __forceinline__ void ensure(int64_t) {}
    __device__ __forceinline__ int64_t O(int64_t j) const { return kdst[j]; }
    __device__ __forceinline__ int64_t S(int64_t j) const { return ksrc[j]; }
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
// Span path
// ---------------------------------------------------------------------------
// Last j in [0, m) with a[j] <= p (a non-decreasing, LDS), or 0.
__device__ __forceinline__ int64_t lds_last_le(const int32_t *a, int64_t m, int64_t p) {
    int64_t lo = 0, hi = m;           // answer in [lo, hi)
    while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if ((int64_t)a[mid] <= p) lo = mid; else hi = mid;
    }
    return lo;
}

template <int kItems>
__global__ __launch_bounds__(kT) void compact_span_kernel(
    const int64_t *__restrict__ off, int64_t n, int64_t NT, const uint8_t *__restrict__ keep,
    CompactCols cols, int n_cols, int64_t *__restrict__ offsets_out, int32_t *__restrict__ kept_ids,
    int64_t *__restrict__ n_kept_tokens, int32_t *__restrict__ reject_ids, int64_t budget) {
    __shared__ int32_t kdst[kItems * kT + 1];
    __shared__ int32_t ksrc[kItems * kT];
    __shared__ uint32_t wcnt[kNW], wrej[kNW];
    __shared__ int64_t wlen[kNW];
    const bool writer = blockIdx.x == 0;
    const int64_t base = (int64_t)threadIdx.x * kItems;

    // 1. Ordered scan of the keep flags and kept lengths, in every workgroup.
    int64_t o[kItems + 1];
    bool kp[kItems];
#pragma unroll
    for (int q = 0; q <= kItems; ++q) o[q] = (base + q <= n) ? clamp64(off[base + q], 0, NT) : 0;
#pragma unroll
    for (int q = 0; q < kItems; ++q) kp[q] = (base + q < n) && keep[base + q] != 0;
    uint32_t c = 0, r = 0;
    int64_t l = 0;
#pragma unroll
    for (int q = 0; q < kItems; ++q) {
        if (kp[q]) {
            c += 1;
            l += (o[q + 1] > o[q]) ? o[q + 1] - o[q] : 0;
        } else if (base + q < n) {
            r += 1;
        }
    }
    uint32_t tot_keep, tot_rej;
    int64_t tot_len;
    uint32_t rank = block_excl_sum_u32<kNW>(c, tot_keep, wcnt);
    int64_t dst = block_excl_sum_i64<kNW>(l, tot_len, wlen);
    uint32_t rpos = reject_ids ? block_excl_sum_u32<kNW>(r, tot_rej, wrej) : 0u;
#pragma unroll
    for (int q = 0; q < kItems; ++q) {
        const int64_t i = base + q;
        if (kp[q]) {
            const int64_t len = (o[q + 1] > o[q]) ? o[q + 1] - o[q] : 0;
            kdst[rank] = (int32_t)(dst < NT ? dst : NT);
            ksrc[rank] = (int32_t)o[q];
            if (writer) {
                offsets_out[rank] = dst;
                kept_ids[rank] = (int32_t)i;
            }
            ++rank;
            dst += len;
        } else if (reject_ids && writer && i < n) {
            if ((int64_t)rpos < budget) reject_ids[rpos] = (int32_t)i;
            ++rpos;
        }
    }
    if (threadIdx.x == 0) {
        kdst[tot_keep] = (int32_t)(tot_len < NT ? tot_len : NT);
        if (writer) {
            offsets_out[tot_keep] = tot_len;
            *n_kept_tokens = tot_len;
        }
    }
    __syncthreads();

    // 2. Copy: the waves of the grid split the packed batch into equal,
    //    1024-element-aligned ranges.
    const int64_t n_kept = tot_keep;
    const int64_t total = tot_len < NT ? tot_len : NT;
    if (n_kept == 0 || total == 0 || n_cols == 0) return;
    const int64_t waves = (int64_t)gridDim.x * kNW;
    int64_t per = (total + waves - 1) / waves;
    per = (per + 1023) / 1024 * 1024;
    const int64_t cs = ((int64_t)blockIdx.x * kNW + threadIdx.x / kWave) * per;
    if (cs >= total) return;
    const int64_t ce = (cs + per < total) ? cs + per : total;
    LdsSpans sp{kdst, ksrc};
    int64_t j = lds_last_le(kdst, n_kept, cs);
    while (j + 1 < n_kept && (int64_t)kdst[j + 1] <= cs) ++j;     // skip empty spans
    for (int col = 0; col < n_cols; ++col) copy_range_col(cols, col, sp, n_kept, NT, cs, ce, j);
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
    (void)n_tokens;
    char *p = (char *)ws;
    CompactWs w;
    w.hdr = (int64_t *)p;          p += 256;
    w.kept_src = (int64_t *)p;     p += align256((size_t)n * 8);
    w.chunk_first = (int32_t *)p;
    return w;
}

size_t compact_ws_bytes(int64_t n, int64_t n_tokens) {
    return 256 + align256((size_t)n * 8) + align256((size_t)map_capacity(n_tokens) * 4);
}

bool compact_span_ok(int64_t n, int64_t n_tokens) {
    return n <= kSpanMaxN && n_tokens < (int64_t)INT32_MAX;
}

hipError_t launch_compact_span(const int64_t *offsets, int64_t n, int64_t n_tokens, const uint8_t *keep,
                               const CompactCols &cols, int n_cols, int64_t *offsets_out,
                               int32_t *kept_ids, int64_t *n_kept_tokens, int32_t *reject_ids,
                               int64_t budget, hipStream_t stream) {
    // One 1024-thread workgroup per CU.
    unsigned grid = (unsigned)(resident_waves() / 16);
    if (grid < 1) grid = 1;
    const int64_t items = (n + kT - 1) / kT;
#define PACE_SPAN(K)                                                                            \
    compact_span_kernel<K><<<grid, kT, 0, stream>>>(offsets, n, n_tokens, keep, cols, n_cols,  \
        offsets_out, kept_ids, n_kept_tokens, reject_ids, budget)
    if (items <= 1) PACE_SPAN(1);
    else if (items <= 2) PACE_SPAN(2);
    else if (items <= 4) PACE_SPAN(4);
    else PACE_SPAN(8);
#undef PACE_SPAN
    return hipGetLastError();
}

hipError_t launch_compact_copy(const CompactCols &cols, int n_cols, int64_t n_tokens,
                               const int64_t *offsets_out, const CompactWs &w, hipStream_t stream) {
    if (n_cols == 0 || n_tokens == 0) return hipSuccess;
    const int64_t max_chunks = (n_tokens + kCopyChunk - 1) / kCopyChunk;
    int64_t blocks = (max_chunks + 3) / 4;
    if (blocks > 1024) blocks = 1024;
    if (blocks < 1) blocks = 1;
    dim3 grid((unsigned)blocks, (unsigned)n_cols);
    compact_copy_kernel<<<grid, 256, 0, stream>>>(cols, offsets_out, w.kept_src, w.chunk_first, w.hdr, n_tokens);
    return hipGetLastError();
}

hipError_t launch_compact(const int64_t *offsets, int64_t n, int64_t n_tokens, const uint8_t *keep,
                          const CompactCols &cols, int n_cols, int64_t *offsets_out,
                          int32_t *kept_ids, int64_t *n_kept_tokens, void *ws, hipStream_t stream) {
    if (compact_span_ok(n, n_tokens))
        return launch_compact_span(offsets, n, n_tokens, keep, cols, n_cols, offsets_out, kept_ids,
                                   n_kept_tokens, nullptr, 0, stream);
    CompactWs w = compact_ws_carve(ws, n, n_tokens);
    compact_scan_kernel<<<1, kT, 0, stream>>>(offsets, n, n_tokens, keep, offsets_out, kept_ids,
                                             n_kept_tokens, w.kept_src, w.chunk_first,
                                             map_capacity(n_tokens), w.hdr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_compact_copy(cols, n_cols, n_tokens, offsets_out, w, stream);
}

}  // namespace pace
