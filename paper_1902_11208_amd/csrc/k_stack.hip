// Glue between the layers of a packed MDLSTM stack (Section V-B): block
// reshape of the input images, and the grouped block-strided convolution with
// tanh that maps one layer's packed output onto the next layer's packed input.
//
// A block-strided convolution has stride equal to its kernel, so every output
// pixel reads one disjoint bh x bw block of input pixels: per example it is a
// per-block linear map (tensor-list chunking, Fig. 1), which here runs
// directly between the two packed canvases. Group d (one per scan direction)
// reads the H channels d*H.. of the block's pixels, block index
// (dy*bw + dx)*H + j, and writes og output channels d*og + o.
//
// Blocks of all examples are numbered consecutively; blk_off[k] is the first
// block of example k (blk_off[n] = total), so a thread finds its example by
// binary search.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

namespace {

// Block of the convolutions between layers: 2 rows x 4 columns.
constexpr int CBH = 2, CBW = 4;

__device__ __forceinline__ int find_example(const int32_t* __restrict__ blk_off, int n, int b) {
    int lo = 0, hi = n - 1;  // largest k with blk_off[k] <= b
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (blk_off[mid] <= b) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

struct BlockPos {
    int64_t in0;   // canvas index of the block's top-left input pixel
    int64_t out;   // canvas index of the output pixel
};

// Position of block b: example k, block (by, bx) of its output rectangle.
__device__ __forceinline__ BlockPos block_pos(const int32_t* __restrict__ blk_off, int n, int b,
                                              const int32_t* __restrict__ in_rects, int in_w,
                                              const int32_t* __restrict__ out_rects, int out_w, int bh, int bw) {
    const int k = find_example(blk_off, n, b);
    const int local = b - blk_off[k];
    const int ow = out_rects[4 * k + 3];
    const int by = local / ow, bx = local - by * ow;
    BlockPos r;
    r.out = (int64_t)(out_rects[4 * k] + by) * out_w + out_rects[4 * k + 1] + bx;
    r.in0 = (int64_t)(in_rects[4 * k] + by * bh) * in_w + in_rects[4 * k + 1] + bx * bw;
    return r;
}

}  // namespace

// ---------------------------------------------------------------------------
// Block reshape of single images into a packed canvas: image k [h][w][c] ->
// rectangle k [h/bh][w/bw][bh*bw*c], channel (dy*bw + dx)*c + ch. One thread
// per output element.
// ---------------------------------------------------------------------------
__global__ void k_pack_blocks(const float* const* __restrict__ imgs, const int32_t* __restrict__ blk_off, int n,
                              const int32_t* __restrict__ rects, int canvas_w, int c, int bh, int bw,
                              float* __restrict__ canvas) {
    const int cb = bh * bw * c;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (int64_t)blk_off[n] * cb) return;
    const int b = (int)(gid / cb), e = (int)(gid - (int64_t)b * cb);
    const int k = find_example(blk_off, n, b);
    const int local = b - blk_off[k];
    const int ow = rects[4 * k + 3];
    const int by = local / ow, bx = local - by * ow;
    const int dyx = e / c, ch = e - dyx * c;
    const int dy = dyx / bw, dx = dyx - dy * bw;
    const int w = ow * bw;
    const float v = imgs[k][((int64_t)(by * bh + dy) * w + bx * bw + dx) * c + ch];
    canvas[((int64_t)(rects[4 * k] + by) * canvas_w + rects[4 * k + 1] + bx) * cb + e] = v;
}

// ---------------------------------------------------------------------------
// Forward: one thread per (block, group d); og outputs, K = bh*bw*H inputs.
// W of all groups sits in LDS.
// ---------------------------------------------------------------------------
template <int H, int OG>
__global__ void __launch_bounds__(256)
k_conv_fwd(const float* __restrict__ y, const float* __restrict__ W, const float* __restrict__ bias,
           const int32_t* __restrict__ blk_off, int n, const int32_t* __restrict__ in_rects, int in_w,
           const int32_t* __restrict__ out_rects, int out_w, float* __restrict__ out) {
    constexpr int bh = CBH, bw = CBW, K = bh * bw * H;
    __shared__ float sw[4 * OG * K];
    for (int i = threadIdx.x; i < 4 * OG * K; i += blockDim.x) sw[i] = W[i];
    __syncthreads();
    const int nb = blk_off[n];
    const int gid = blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= 4 * nb) return;
    const int b = gid >> 2, d = gid & 3;
    const BlockPos P = block_pos(blk_off, n, b, in_rects, in_w, out_rects, out_w, CBH, CBW);
    float acc[OG];
#pragma unroll
    for (int o = 0; o < OG; ++o) acc[o] = bias[d * OG + o];
    const float* wd = sw + d * OG * K;
    for (int dy = 0; dy < bh; ++dy)
        for (int dx = 0; dx < bw; ++dx) {
            const float* yp = y + (P.in0 + (int64_t)dy * in_w + dx) * (4 * H) + d * H;
            const int k0 = (dy * bw + dx) * H;
#pragma unroll
            for (int j = 0; j < H; j += 4) {
                const float4 v = *reinterpret_cast<const float4*>(yp + j);
#pragma unroll
                for (int o = 0; o < OG; ++o) {
                    const float* wr = wd + o * K + k0 + j;
                    acc[o] += wr[0] * v.x + wr[1] * v.y + wr[2] * v.z + wr[3] * v.w;
                }
            }
        }
    float* op = out + P.out * (4 * OG) + d * OG;
#pragma unroll
    for (int o = 0; o < OG; o += 4)
        *reinterpret_cast<float4*>(op + o) = make_float4(tanhf(acc[o]), tanhf(acc[o + 1]), tanhf(acc[o + 2]),
                                                         tanhf(acc[o + 3]));
}

// ---------------------------------------------------------------------------
// Backward, input gradient: one thread per (block, group d):
//   g[o] = dout[o] (1 - out[o]^2),  dy[pixel][d*H + j] = sum_o g[o] W[d][o][(dy*bw+dx)*H + j].
// ---------------------------------------------------------------------------
template <int H, int OG>
__global__ void __launch_bounds__(256)
k_conv_bwd_dy(const float* __restrict__ out, const float* __restrict__ dout, const float* __restrict__ W,
              const int32_t* __restrict__ blk_off, int n, const int32_t* __restrict__ in_rects, int in_w,
              const int32_t* __restrict__ out_rects, int out_w, float* __restrict__ dy) {
    constexpr int bh = CBH, bw = CBW, K = bh * bw * H;
    __shared__ float sw[4 * OG * K];
    for (int i = threadIdx.x; i < 4 * OG * K; i += blockDim.x) sw[i] = W[i];
    __syncthreads();
    const int nb = blk_off[n];
    const int gid = blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= 4 * nb) return;
    const int b = gid >> 2, d = gid & 3;
    const BlockPos P = block_pos(blk_off, n, b, in_rects, in_w, out_rects, out_w, CBH, CBW);
    float g[OG];
#pragma unroll
    for (int o = 0; o < OG; o += 4) {
        const float4 ov = *reinterpret_cast<const float4*>(out + P.out * (4 * OG) + d * OG + o);
        const float4 gv = *reinterpret_cast<const float4*>(dout + P.out * (4 * OG) + d * OG + o);
        g[o] = gv.x * (1.0f - ov.x * ov.x);
        g[o + 1] = gv.y * (1.0f - ov.y * ov.y);
        g[o + 2] = gv.z * (1.0f - ov.z * ov.z);
        g[o + 3] = gv.w * (1.0f - ov.w * ov.w);
    }
    const float* wd = sw + d * OG * K;
    for (int dyy = 0; dyy < bh; ++dyy)
        for (int dx = 0; dx < bw; ++dx) {
            float* dp = dy + (P.in0 + (int64_t)dyy * in_w + dx) * (4 * H) + d * H;
            const int k0 = (dyy * bw + dx) * H;
#pragma unroll
            for (int j = 0; j < H; j += 4) {
                float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int o = 0; o < OG; ++o) {
                    const float* wr = wd + o * K + k0 + j;
                    a.x += g[o] * wr[0];
                    a.y += g[o] * wr[1];
                    a.z += g[o] * wr[2];
                    a.w += g[o] * wr[3];
                }
                *reinterpret_cast<float4*>(dp + j) = a;
            }
        }
}

// ---------------------------------------------------------------------------
// Backward, weight and bias gradients. Workgroup c sums blocks
// [c*per, (c+1)*per) in order into partial[c][4*OG*K + 4*OG]; BPP blocks per
// pass are staged in LDS (their g values and input pixels), each thread owns
// fixed (d, o, k) entries. A second kernel adds the partials in chunk order,
// so the result does not depend on scheduling.
// ---------------------------------------------------------------------------
template <int H, int OG>
__global__ void __launch_bounds__(256)
k_conv_bwd_dw(const float* __restrict__ y, const float* __restrict__ out, const float* __restrict__ dout,
              const int32_t* __restrict__ blk_off, int n, const int32_t* __restrict__ in_rects, int in_w,
              const int32_t* __restrict__ out_rects, int out_w, int per, float* __restrict__ partial) {
    constexpr int bh = CBH, bw = CBW, BPP = 8;
    constexpr int K = bh * bw * H, CB = bh * bw;  // inputs per group, pixels per block
    constexpr int M = 4 * OG * K;
    constexpr int MAXE = (M + 255) / 256;          // (d, o, k) entries per thread
    __shared__ __attribute__((aligned(16))) float sg[BPP * 4 * OG];     // g of the staged blocks
    __shared__ __attribute__((aligned(16))) float sy[BPP * CB * 4 * H];  // their input pixels
    const int nb = blk_off[n];
    const int b0 = blockIdx.x * per, b1 = min(nb, b0 + per);
    float acc[MAXE];
    float accb = 0.0f;
#pragma unroll
    for (int e = 0; e < MAXE; ++e) acc[e] = 0.0f;
    for (int bb = b0; bb < b1; bb += BPP) {
        const int nblk = min(BPP, b1 - bb);
        // stage g = dout (1 - out^2) and the input pixels of nblk blocks
        for (int i = threadIdx.x; i < nblk * 4 * OG; i += blockDim.x) {
            const int lb = i / (4 * OG), ch = i - lb * (4 * OG);
            const BlockPos P = block_pos(blk_off, n, bb + lb, in_rects, in_w, out_rects, out_w, CBH, CBW);
            const float ov = out[P.out * (4 * OG) + ch];
            sg[i] = dout[P.out * (4 * OG) + ch] * (1.0f - ov * ov);
        }
        for (int i = threadIdx.x; i < nblk * CB * H; i += blockDim.x) {  // float4 units of [lb][pix][4H]
            const int lb = i / (CB * H), rem = i - lb * (CB * H);
            const int pix = rem / H, c4 = rem - pix * H;
            const int dyy = pix / bw, dx = pix - dyy * bw;
            const BlockPos P = block_pos(blk_off, n, bb + lb, in_rects, in_w, out_rects, out_w, CBH, CBW);
            reinterpret_cast<float4*>(sy)[i] =
                *reinterpret_cast<const float4*>(y + (P.in0 + (int64_t)dyy * in_w + dx) * (4 * H) + 4 * c4);
        }
        __syncthreads();
        for (int lb = 0; lb < nblk; ++lb) {
            const float* gb = sg + lb * 4 * OG;
            const float* yb = sy + lb * CB * 4 * H;
#pragma unroll
            for (int e = 0; e < MAXE; ++e) {
                const int idx = e * 256 + (int)threadIdx.x;  // entry (d, o, k) = ((d*OG + o)*K + k)
                if (idx < M) {
                    const int dk = idx / K, kk = idx - dk * K;  // dk = d*OG + o
                    const int d = dk / OG;
                    const int pix = kk / H, j = kk - pix * H;
                    acc[e] += gb[dk] * yb[pix * 4 * H + d * H + j];
                }
            }
            if ((int)threadIdx.x < 4 * OG) accb += gb[threadIdx.x];
        }
        __syncthreads();
    }
    float* pc = partial + (size_t)blockIdx.x * (M + 4 * OG);
#pragma unroll
    for (int e = 0; e < MAXE; ++e) {
        const int idx = e * 256 + (int)threadIdx.x;
        if (idx < M) pc[idx] = acc[e];
    }
    if ((int)threadIdx.x < 4 * OG) pc[M + threadIdx.x] = accb;
}

// Fixed-order sum of the chunk partials: a block takes 64 consecutive
// outputs; its four thread groups sum every fourth chunk each (loads batched
// eight at a time), and the four sums are added in a fixed order.
__global__ void __launch_bounds__(256)
k_sum_partials(const float* __restrict__ partial, int chunks, int m, float* __restrict__ dw,
               float* __restrict__ db, int mw) {
    __shared__ float ps[4][64];
    const int t = threadIdx.x & 63, grp = threadIdx.x >> 6;
    const int i = blockIdx.x * 64 + t;
    float s = 0.0f;
    if (i < m) {
        int c = grp;
        for (; c + 28 < chunks; c += 32) {
            float v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = partial[(size_t)(c + 4 * k) * m + i];
#pragma unroll
            for (int k = 0; k < 8; ++k) s += v[k];
        }
        for (; c < chunks; c += 4) s += partial[(size_t)c * m + i];
    }
    ps[grp][t] = s;
    __syncthreads();
    if (grp == 0 && i < m) {
        const float v = ((ps[0][t] + ps[1][t]) + ps[2][t]) + ps[3][t];
        if (i < mw) dw[i] = v;
        else db[i - mw] = v;
    }
}

__global__ void k_zero_f32(float* __restrict__ d, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        d[i] = 0.0f;
}

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------
hipError_t launch_zero_f32(float* d, int64_t n, hipStream_t s) {
    if (n > 0) {
        const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
        hipLaunchKernelGGL(k_zero_f32, dim3((unsigned)blocks), dim3(256), 0, s, d, n);
    }
    return hipGetLastError();
}

hipError_t launch_pack_blocks(int n, const float* const* d_imgs, const int32_t* d_blk_off, int total_blocks,
                              const int32_t* d_rects, int canvas_w, int c, int bh, int bw, float* d_canvas,
                              hipStream_t s) {
    const int64_t total = (int64_t)total_blocks * bh * bw * c;
    if (total > 0)
        hipLaunchKernelGGL(k_pack_blocks, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, d_imgs, d_blk_off,
                           n, d_rects, canvas_w, c, bh, bw, d_canvas);
    return hipGetLastError();
}

bool conv_supported(int hidden, int og, int bh, int bw) {
    const bool h_ok = hidden == 4 || hidden == 8 || hidden == 16 || hidden == 32 || hidden == 64;
    const bool o_ok = og == 4 || og == 8 || og == 16 || og == 32;
    return h_ok && o_ok && bh == CBH && bw == CBW && 4 * og * CBH * CBW * hidden * 4 <= 64 * 1024;
}

int conv_chunks(int total_blocks) { return total_blocks <= 0 ? 1 : (total_blocks < 512 ? total_blocks : 512); }

size_t conv_partial_bytes(int hidden, int og, int bh, int bw, int total_blocks) {
    return (size_t)conv_chunks(total_blocks) * (4 * og * bh * bw * hidden + 4 * og) * 4;
}

template <int H, int OG>
static hipError_t conv_launch(bool fwd, const ConvArgs& a, hipStream_t s) {
    if constexpr (4 * OG * CBH * CBW * H * 4 > 64 * 1024) {
        return hipErrorInvalidValue;  // rejected by conv_supported
    } else {
        constexpr int K = CBH * CBW * H;
        const unsigned grid = (unsigned)((4 * a.total_blocks + 255) / 256);
        if (fwd) {
            hipLaunchKernelGGL((k_conv_fwd<H, OG>), dim3(grid), dim3(256), 0, s, a.y, a.w, a.b, a.blk_off, a.n,
                               a.in_rects, a.in_w, a.out_rects, a.out_w, a.out);
            return hipGetLastError();
        }
        hipLaunchKernelGGL((k_conv_bwd_dy<H, OG>), dim3(grid), dim3(256), 0, s, a.out, a.dout, a.w, a.blk_off, a.n,
                           a.in_rects, a.in_w, a.out_rects, a.out_w, a.dy);
        const int chunks = conv_chunks(a.total_blocks);
        const int per = (a.total_blocks + chunks - 1) / chunks;
        hipLaunchKernelGGL((k_conv_bwd_dw<H, OG>), dim3(chunks), dim3(256), 0, s, a.y, a.out, a.dout, a.blk_off,
                           a.n, a.in_rects, a.in_w, a.out_rects, a.out_w, per, a.partial);
        const int m = 4 * OG * K + 4 * OG;
        hipLaunchKernelGGL(k_sum_partials, dim3((m + 63) / 64), dim3(256), 0, s, a.partial, chunks, m, a.dw,
                           a.db, 4 * OG * K);
        return hipGetLastError();
    }
}

template <int H>
static hipError_t conv_og(bool fwd, const ConvArgs& a, hipStream_t s) {
    switch (a.og) {
        case 4: return conv_launch<H, 4>(fwd, a, s);
        case 8: return conv_launch<H, 8>(fwd, a, s);
        case 16: return conv_launch<H, 16>(fwd, a, s);
        case 32: return conv_launch<H, 32>(fwd, a, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_block_conv(bool fwd, const ConvArgs& a, hipStream_t s) {
    if (a.total_blocks <= 0) return hipSuccess;
    switch (a.hidden) {
        case 4: return conv_og<4>(fwd, a, s);
        case 8: return conv_og<8>(fwd, a, s);
        case 16: return conv_og<16>(fwd, a, s);
        case 32: return conv_og<32>(fwd, a, s);
        case 64: return conv_og<64>(fwd, a, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mdl
