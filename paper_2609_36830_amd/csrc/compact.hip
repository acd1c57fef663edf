// pace_compact kernels for gfx950: pack the kept trajectories' token spans
// into the training batch (Algorithm 1), survivors in pool order.
//
// Step 1 (compact_scan, one workgroup of 1024 threads): ordered scan of the
// keep flags and kept lengths over trajectories -> offsets_out, kept_ids,
// the source start of every kept span, and a map from each output chunk of
// kCopyChunk elements to the kept span that covers its first element.
//
// Step 2 (compact_copy): one wave per output chunk (grid-stride), one
// workgroup row per payload column. Output is written in aligned 16-byte
// vectors (64 lanes x 16 B = 1 KiB per wave window). Inside one kept span the
// source is the destination shifted by a constant, so its misalignment is
// wave-uniform: each lane loads the aligned 16 bytes under its window, takes
// the next 16 bytes from the neighbouring lane (lane 63 loads them), and a
// byte funnel shift assembles the output vector. Windows that straddle span
// ends, the ragged tail, and unaligned columns copy element by element.
#include "device_util.hpp"
#include "kernels.hpp"

namespace pace {

namespace {

constexpr int kT = 1024;
constexpr int kNW = kT / kWave;

__device__ __forceinline__ uint32_t blk_excl_count(bool f, uint32_t &total, uint32_t *wsum) {
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

__device__ __forceinline__ int64_t blk_excl_sum(int64_t v, int64_t &total, int64_t *wsum) {
    const int64_t inc = wave_incl_scan_i64(v);
    const int w = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) wsum[w] = inc;
    __syncthreads();
    int64_t before = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < kNW; ++k) {
        const int64_t x = wsum[k];
        tot += x;
        before += (k < w) ? x : 0;
    }
    __syncthreads();
    total = tot;
    return before + inc - v;
}

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
        const uint32_t r = blk_excl_count(k, tc, wcnt);
        int64_t tl;
        const int64_t d = blk_excl_sum(len, tl, wlen);
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

template <int E> struct Elem;
template <> struct Elem<1> { using T = uint8_t; };
template <> struct Elem<2> { using T = uint16_t; };
template <> struct Elem<4> { using T = uint32_t; };
template <> struct Elem<8> { using T = uint64_t; };

// Lane k caches o[base + k] = offsets_out and s[base + k] = kept_src.
struct SpanCache {
    int64_t base, o, s;
    __device__ __forceinline__ void load(const int64_t *__restrict__ oo, const int64_t *__restrict__ ss,
                                         int64_t n_kept, int64_t b) {
        base = b;
        const int64_t idx = b + lane_id();
        o = (idx <= n_kept) ? oo[idx] : INT64_MAX;
        s = (idx < n_kept) ? ss[idx] : 0;
    }
    __device__ __forceinline__ void ensure(const int64_t *oo, const int64_t *ss, int64_t n_kept, int64_t j) {
        // entries j and j + 1 must be cached
        if (j < base || j + 1 - base >= kWave) load(oo, ss, n_kept, j);
    }
    __device__ __forceinline__ int64_t O(int64_t j) const { return readlane_i64(o, (int)(j - base)); }
    __device__ __forceinline__ int64_t S(int64_t j) const { return readlane_i64(s, (int)(j - base)); }
};

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

template <int E>
__device__ void copy_chunk(const char *__restrict__ in, char *__restrict__ out, bool vec,
                           const int64_t *__restrict__ oo, const int64_t *__restrict__ ss,
                           int64_t n_kept, int64_t NT, int64_t cs, int64_t ce, int64_t j) {
    using T = typename Elem<E>::T;
    constexpr int VE = 16 / E;          // elements per lane vector
    constexpr int WE = kWave * VE;      // elements per wave window (1 KiB)
    const int lane = lane_id();
    const int64_t nbytes = NT * E;
    SpanCache sc;
    sc.load(oo, ss, n_kept, j);
    for (int64_t w = cs; w < ce; w += WE) {
        sc.ensure(oo, ss, n_kept, j);
        while (j + 1 < n_kept && sc.O(j + 1) <= w) {
            ++j;
            sc.ensure(oo, ss, n_kept, j);
        }
        const int64_t we = (w + WE < ce) ? w + WE : ce;
        const int64_t o_lo = sc.O(j), o_hi = sc.O(j + 1);
        const int64_t delta = sc.S(j) - o_lo;          // src element = dst element + delta
        bool fast = vec && o_lo <= w && w + WE <= o_hi && w + WE <= ce &&
                    w + delta >= 0 && w + WE + delta <= NT;
        int shift = 0;
        if (fast) {
            shift = (int)((((delta * E) % 16) + 16) % 16);
            // lane 63 also reads the aligned vector after its own
            const int64_t ab63 = (w + (int64_t)(kWave - 1) * VE + delta) * E - shift;
            if (shift != 0 && ab63 + 32 > nbytes) fast = false;
        }
        if (fast) {
            const int64_t sb = (w + (int64_t)lane * VE + delta) * E;
            const int64_t ab = sb - shift;
            const uint4 a = *reinterpret_cast<const uint4 *>(in + ab);
            uint4 o = a;
            if (shift != 0) {
                uint4 b = shfl_down1(a);
                if (lane == kWave - 1) b = *reinterpret_cast<const uint4 *>(in + ab + 16);
                o = funnel16(a, b, shift);
            }
            *reinterpret_cast<uint4 *>(out + (w + (int64_t)lane * VE) * E) = o;
            continue;
        }
        // Element path: every span that meets [w, we).
        int64_t jj = j;
        while (true) {
            sc.ensure(oo, ss, n_kept, jj);
            const int64_t lo = sc.O(jj), hi = sc.O(jj + 1);
            const int64_t d = sc.S(jj) - lo;
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

__global__ __launch_bounds__(256) void compact_copy_kernel(
    CompactCols cols, const int64_t *__restrict__ oo, const int64_t *__restrict__ ss,
    const int32_t *__restrict__ chunk_first, const int64_t *__restrict__ hdr, int64_t NT) {
    const int col = blockIdx.y;
    const int E = cols.elem[col];
    const bool vec = cols.vec[col] != 0;
    const int64_t n_kept = hdr[0];
    const int64_t total = hdr[1];
    if (n_kept <= 0) return;
    const int64_t n_chunks = (total + kCopyChunk - 1) / kCopyChunk;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x / kWave);
    for (int64_t c = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave; c < n_chunks; c += waves) {
        const int64_t cs = c * kCopyChunk;
        const int64_t ce = (cs + kCopyChunk < total) ? cs + kCopyChunk : total;
        const int64_t j = clamp64(chunk_first[c], 0, n_kept - 1);
        const char *in = (const char *)cols.in[col];
        char *out = (char *)cols.out[col];
        switch (E) {
            case 1: copy_chunk<1>(in, out, vec, oo, ss, n_kept, NT, cs, ce, j); break;
            case 2: copy_chunk<2>(in, out, vec, oo, ss, n_kept, NT, cs, ce, j); break;
            case 4: copy_chunk<4>(in, out, vec, oo, ss, n_kept, NT, cs, ce, j); break;
            default: copy_chunk<8>(in, out, vec, oo, ss, n_kept, NT, cs, ce, j); break;
        }
    }
}

int64_t map_capacity(int64_t n_tokens) { return (n_tokens + kCopyChunk - 1) / kCopyChunk + 1; }

struct CompactWs {
    int64_t *hdr;
    int64_t *kept_src;
    int32_t *chunk_first;
};

CompactWs compact_ws_carve(void *ws, int64_t n, int64_t n_tokens) {
    char *p = (char *)ws;
    CompactWs w;
    w.hdr = (int64_t *)p;          p += 256;
    w.kept_src = (int64_t *)p;     p += align256((size_t)n * 8);
    w.chunk_first = (int32_t *)p;
    (void)n_tokens;
    return w;
}

}  // namespace

size_t compact_ws_bytes(int64_t n, int64_t n_tokens) {
    return 256 + align256((size_t)n * 8) + align256((size_t)map_capacity(n_tokens) * 4);
}

hipError_t launch_compact(const int64_t *offsets, int64_t n, int64_t n_tokens, const uint8_t *keep,
                          const CompactCols &cols, int n_cols, int64_t *offsets_out,
                          int32_t *kept_ids, int64_t *n_kept_tokens, void *ws, hipStream_t stream) {
    CompactWs w = compact_ws_carve(ws, n, n_tokens);
    compact_scan_kernel<<<1, kT, 0, stream>>>(offsets, n, n_tokens, keep, offsets_out, kept_ids,
                                             n_kept_tokens, w.kept_src, w.chunk_first,
                                             map_capacity(n_tokens), w.hdr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || n_cols == 0 || n_tokens == 0) return e;
    const int64_t max_chunks = (n_tokens + kCopyChunk - 1) / kCopyChunk;
    int64_t blocks = (max_chunks + 3) / 4;
    if (blocks > 1024) blocks = 1024;
    if (blocks < 1) blocks = 1;
    dim3 grid((unsigned)blocks, (unsigned)n_cols);
    compact_copy_kernel<<<grid, 256, 0, stream>>>(cols, offsets_out, w.kept_src, w.chunk_first, w.hdr, n_tokens);
    return hipGetLastError();
}

}  // namespace pace
