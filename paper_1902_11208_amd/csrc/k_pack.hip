// Example packing kernels (Section V-A; Algorithm 1 in Appendix B):
// placement, mask, rectangle-id map, scatter and gather.
#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

// ---------------------------------------------------------------------------
// Placement. One workgroup.
//  1. Sort keys (height ascending, width descending, original index ascending)
//     with a bitonic network in LDS: this is the bucketing by height and the
//     "widest first" candidate order inside each bucket.
//  2. One wave walks the buckets and fills rows greedily: the first remaining
//     candidate opens a row; then, while space is left, the first candidate
//     no wider than the remaining space (widths are sorted within the bucket)
//     and from there the first one not yet placed are found, each with one or
//     two ballots (a 64-way search over the sorted keys; a bit per position,
//     64 per lane, marks the placed ones). A row closes when nothing fits and
//     is flushed when its bucket runs empty. Coordinates are assigned as rows
//     are made.
// Key layout: [63:42] height, [41:21] (2^21-1-width), [20:0] index.
// ---------------------------------------------------------------------------
constexpr int PLACE_THREADS = 1024;

__global__ void __launch_bounds__(PLACE_THREADS)
k_pack_place(int n, int npow2, int canvas_w, const int32_t* __restrict__ hw, int32_t* __restrict__ out) {
    extern __shared__ unsigned long long smem_keys[];
    unsigned long long* keys = smem_keys;  // npow2
    const int tid = threadIdx.x;
    for (int i = tid; i < npow2; i += PLACE_THREADS) {
        unsigned long long k = ~0ull;
        if (i < n) {
            unsigned long long h = (unsigned long long)hw[i];
            unsigned long long w = (unsigned long long)hw[n + i];
            k = (h << 42) | (((1ull << 21) - 1 - w) << 21) | (unsigned long long)i;
        }
        keys[i] = k;
    }
    __syncthreads();
    for (int size = 2; size <= npow2; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int t = tid; t < npow2 / 2; t += PLACE_THREADS) {
                int lo = 2 * t - (t & (stride - 1));
                int hi = lo + stride;
                bool up = ((lo & size) == 0);
                unsigned long long a = keys[lo], b = keys[hi];
                if ((a > b) == up) {
                    keys[lo] = b;
                    keys[hi] = a;
                }
            }
            __syncthreads();
        }
    }
    __syncthreads();
    if (tid >= 64) return;
    // From here one wave. Lane l holds the "placed" bits of sorted positions
    // 64 l .. 64 l + 63 (positions past n count as placed); searches over the
    // sorted keys are 64-way with a ballot per level.
    const int lane = tid;
    uint64_t placed = 0;
    if (64 * lane >= n) placed = ~0ull;
    else if (n - 64 * lane < 64) placed = ~0ull << (n - 64 * lane);

    auto kh = [&](int i) { return (int)(keys[i] >> 42); };
    auto kw = [&](int i) { return (int)((1 << 21) - 1 - (int)((keys[i] >> 21) & ((1ull << 21) - 1))); };
    auto ki = [&](int i) { return (int)(keys[i] & ((1ull << 21) - 1)); };
    // first position >= from not yet placed (n when none)
    auto first_free = [&](int from) {
        uint64_t fr = ~placed;
        const int wd = from >> 6;
        if (lane < wd) fr = 0;
        else if (lane == wd) fr &= ~0ull << (from & 63);
        const uint64_t has = __ballot(fr != 0);
        if (has == 0) return n;
        const int f = __builtin_ctzll(has);
        const uint32_t lo = __shfl((uint32_t)fr, f), hi = __shfl((uint32_t)(fr >> 32), f);
        const uint64_t w = ((uint64_t)hi << 32) | lo;
        return 64 * f + __builtin_ctzll(w);
    };
    // first position in [a, b) where pred holds (b when none), pred being
    // false then true along [a, b): blocks of `stride`, then within one block
    auto first_true = [&](int a, int b, auto pred) {
        if (a >= b) return b;
        const int stride = (b - a + 63) / 64;
        const int pos = a + lane * stride;
        const bool tp = pred(min(pos, b - 1));  // every lane reads a position inside [a, b)
        const uint64_t t = __ballot(pos < b && tp);
        int lo, hi;
        if (t & 1ull) return a;
        if (t) {
            const int f = __builtin_ctzll(t);
            lo = a + (f - 1) * stride + 1;
            hi = a + f * stride;  // pred(hi) holds
        } else {
            const int last = (b - 1 - a) / stride;  // last block with a valid start
            lo = a + last * stride + 1;
            hi = b;
        }
        const int p2 = lo + lane;
        const bool tp2 = pred(min(p2, b - 1));
        const uint64_t t2 = __ballot(p2 < hi && tp2);
        return t2 ? lo + __builtin_ctzll(t2) : hi;
    };
    auto mark = [&](int p) {
        if (lane == (p >> 6)) placed |= 1ull << (p & 63);
    };

    int y = 0;
    bool first_row = true;
    int b0 = 0;
    while (b0 < n) {
        const int hb = kh(b0);
        // the bucket [b0, b1) of height hb (heights ascend)
        const int b1 = first_true(b0 + 1, n, [&](int i) { return kh(i) > hb; });
        // the bucket is filled row by row
        while (true) {
            const int p = first_free(b0);
            if (p >= b1) break;
            if (!first_row) y += 1;  // separator row
            first_row = false;
            int used = kw(p);
            if (lane == 0) {
                const int k = ki(p);
                out[4 * k + 0] = y;
                out[4 * k + 1] = 0;
                out[4 * k + 2] = hb;
                out[4 * k + 3] = used;
            }
            mark(p);
            while (true) {
                const int cap = canvas_w - used - 1;
                if (cap < 1) break;
                // first candidate no wider than the space left (widths descend
                // within the bucket), then the first one not yet placed from there
                const int lo = first_true(b0, b1, [&](int i) { return kw(i) <= cap; });
                const int q = first_free(lo);
                if (q >= b1) break;
                const int wq = kw(q);
                if (lane == 0) {
                    const int kq = ki(q);
                    out[4 * kq + 0] = y;
                    out[4 * kq + 1] = used + 1;
                    out[4 * kq + 2] = hb;
                    out[4 * kq + 3] = wq;
                }
                used += 1 + wq;
                mark(q);
            }
            y += hb;
        }
        b0 = b1;
    }
    if (lane == 0) out[4 * n] = y;
}

hipError_t launch_pack_place(int n, int canvas_w, const int32_t* d_hw, int32_t* d_out, int32_t*,
                             hipStream_t s) {
    int npow2 = 1;
    while (npow2 < n) npow2 <<= 1;
    size_t lds = (size_t)npow2 * 8;
    hipLaunchKernelGGL(k_pack_place, dim3(1), dim3(PLACE_THREADS), lds, s, n, npow2, canvas_w, d_hw, d_out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Mask and rectangle ids: fill the canvas with the background value, then
// each workgroup paints one rectangle.
// ---------------------------------------------------------------------------
template <typename V>
__global__ void k_fill(V* __restrict__ p, int64_t count, V v) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < count; i += stride) p[i] = v;
}

template <typename V, bool USE_INDEX>
__global__ void k_paint_rects(const int32_t* __restrict__ rects, int canvas_w, V* __restrict__ out, V v,
                              unsigned* __restrict__ zero2) {
    const int k = blockIdx.x;
    if (zero2 && k == 0 && threadIdx.x < 2) zero2[threadIdx.x] = 0u;
    const int y0 = rects[4 * k], x0 = rects[4 * k + 1], h = rects[4 * k + 2], w = rects[4 * k + 3];
    const V val = USE_INDEX ? (V)k : v;
    for (int i = threadIdx.x; i < h * w; i += blockDim.x) {
        int yy = i / w, xx = i - yy * w;
        out[(int64_t)(y0 + yy) * canvas_w + (x0 + xx)] = val;
    }
}

static int fill_blocks(int64_t count) {
    int64_t b = (count + 255) / 256;
    return (int)(b < 4096 ? (b > 0 ? b : 1) : 4096);
}

hipError_t launch_mask(int n, const int32_t* d_rects, int canvas_h, int canvas_w, uint8_t* d_mask,
                       hipStream_t s) {
    int64_t cells = (int64_t)canvas_h * canvas_w;
    if (cells > 0)
        hipLaunchKernelGGL(k_fill<uint8_t>, dim3(fill_blocks(cells)), dim3(256), 0, s, d_mask, cells, (uint8_t)0);
    if (n > 0)
        hipLaunchKernelGGL((k_paint_rects<uint8_t, false>), dim3(n), dim3(256), 0, s, d_rects, canvas_w, d_mask,
                           (uint8_t)1, nullptr);
    return hipGetLastError();
}

hipError_t launch_rect_ids(int n, const int32_t* d_rects, int canvas_h, int canvas_w, int32_t* d_rid,
                           unsigned* d_zero2, hipStream_t s) {
    int64_t cells = (int64_t)canvas_h * canvas_w;
    if (cells > 0)
        hipLaunchKernelGGL(k_fill<int32_t>, dim3(fill_blocks(cells)), dim3(256), 0, s, d_rid, cells, (int32_t)-1);
    if (n > 0)
        hipLaunchKernelGGL((k_paint_rects<int32_t, true>), dim3(n), dim3(256), 0, s, d_rects, canvas_w, d_rid,
                           (int32_t)0, d_zero2);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Scatter / gather: block (k, row) copies one example row of w*c elements.
// Element size 2 or 4 bytes; copies run in 2-byte or 4-byte units.
// ---------------------------------------------------------------------------
template <typename E>
__global__ void k_scatter(const void* const* __restrict__ ptrs, const int32_t* __restrict__ rects, int canvas_w,
                          int c, E* __restrict__ canvas) {
    const int k = blockIdx.x, yy = blockIdx.y;
    const int y0 = rects[4 * k], x0 = rects[4 * k + 1], h = rects[4 * k + 2], w = rects[4 * k + 3];
    if (yy >= h) return;
    const E* src = reinterpret_cast<const E*>(ptrs[k]) + (int64_t)yy * w * c;
    E* dst = canvas + ((int64_t)(y0 + yy) * canvas_w + x0) * c;
    for (int i = threadIdx.x; i < w * c; i += blockDim.x) dst[i] = src[i];
}

template <typename E>
__global__ void k_gather(void* const* __restrict__ ptrs, const int32_t* __restrict__ rects, int canvas_w, int c,
                         const E* __restrict__ canvas) {
    const int k = blockIdx.x, yy = blockIdx.y;
    const int y0 = rects[4 * k], x0 = rects[4 * k + 1], h = rects[4 * k + 2], w = rects[4 * k + 3];
    if (yy >= h) return;
    E* dst = reinterpret_cast<E*>(ptrs[k]) + (int64_t)yy * w * c;
    const E* src = canvas + ((int64_t)(y0 + yy) * canvas_w + x0) * c;
    for (int i = threadIdx.x; i < w * c; i += blockDim.x) dst[i] = src[i];
}

hipError_t launch_scatter(int n, const void* const* d_ptrs, const int32_t* d_rects, int canvas_h, int canvas_w,
                          int c, int esize, void* d_canvas, int max_h, hipStream_t s) {
    int64_t bytes = (int64_t)canvas_h * canvas_w * c * esize;
    if (bytes > 0) {
        if (bytes % 8 == 0)
            hipLaunchKernelGGL(k_fill<uint2>, dim3(fill_blocks(bytes / 8)), dim3(256), 0, s,
                               reinterpret_cast<uint2*>(d_canvas), bytes / 8, make_uint2(0, 0));
        else
            hipLaunchKernelGGL(k_fill<uint16_t>, dim3(fill_blocks(bytes / 2)), dim3(256), 0, s,
                               reinterpret_cast<uint16_t*>(d_canvas), bytes / 2, (uint16_t)0);
    }
    if (n > 0 && max_h > 0) {
        dim3 grid(n, max_h);
        if (esize == 4)
            hipLaunchKernelGGL(k_scatter<float>, grid, dim3(256), 0, s, d_ptrs, d_rects, canvas_w, c,
                               reinterpret_cast<float*>(d_canvas));
        else
            hipLaunchKernelGGL(k_scatter<uint16_t>, grid, dim3(256), 0, s, d_ptrs, d_rects, canvas_w, c,
                               reinterpret_cast<uint16_t*>(d_canvas));
    }
    return hipGetLastError();
}

hipError_t launch_gather(int n, void* const* d_ptrs, const int32_t* d_rects, int canvas_w, int c, int esize,
                         const void* d_canvas, int max_h, hipStream_t s) {
    if (n > 0) {
        dim3 grid(n, max_h > 0 ? max_h : 1);
        if (esize == 4)
            hipLaunchKernelGGL(k_gather<float>, grid, dim3(256), 0, s, d_ptrs, d_rects, canvas_w, c,
                               reinterpret_cast<const float*>(d_canvas));
        else
            hipLaunchKernelGGL(k_gather<uint16_t>, grid, dim3(256), 0, s, d_ptrs, d_rects, canvas_w, c,
                               reinterpret_cast<const uint16_t*>(d_canvas));
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Zero the rows of invalid cells (mask 0 or outside every rectangle) of a
// [n_cells][width] tensor; width*esize is a multiple of 8 bytes.
// ---------------------------------------------------------------------------
// A wave takes 64 cells: each lane reads one cell's mask byte and rect id,
// then the wave writes the rows of the invalid ones, one row at a time with
// the lanes along the row.
__global__ void k_zero_invalid(int64_t n_cells, int row_words, const uint8_t* __restrict__ mask,
                               const int32_t* __restrict__ rid, uint2* __restrict__ t) {
    const int lane = threadIdx.x & 63;
    const int64_t wstride = (int64_t)gridDim.x * (blockDim.x >> 6) * 64;
    for (int64_t c0 = ((int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * 64; c0 < n_cells;
         c0 += wstride) {
        const int64_t p = c0 + lane;
        const bool bad = p < n_cells && (mask[p] == 0 || rid[p] < 0);
        for (uint64_t bm = __ballot(bad); bm; bm &= bm - 1) {
            uint2* row = t + (c0 + __builtin_ctzll(bm)) * row_words;
            for (int k = lane; k < row_words; k += 64) row[k] = make_uint2(0, 0);
        }
    }
}

hipError_t launch_zero_invalid(const LayerGeom& g, int width, const uint8_t* d_mask, const int32_t* d_rid,
                               void* d_t, hipStream_t s) {
    int esize = g.dtype == 1 ? 2 : 4;
    int row_words = width * esize / 8;
    if (g.n_cells > 0 && row_words > 0)
        hipLaunchKernelGGL(k_zero_invalid, dim3(fill_blocks(g.n_cells)), dim3(256), 0, s, g.n_cells, row_words,
                           d_mask, d_rid, reinterpret_cast<uint2*>(d_t));
    return hipGetLastError();
}

}  // namespace mdl
