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
// The convolution kernels take the blocks in steps of consecutive blocks
// (grid-stride over steps). A step mostly lies in one block row of one
// rectangle, where block t's pixels sit t * bw columns right of the first
// block's and its output pixel t to the right: only the first block's
// position needs the search over the examples.
// ---------------------------------------------------------------------------
struct ConvGeo {
    const int32_t* blk_off;
    int n;
    const int32_t* in_rects;
    int in_w;
    const int32_t* out_rects;
    int out_w;
};

struct RowPos {
    int64_t in0, out;
    int rem;  // blocks from this one to the end of its block row
};

__device__ __forceinline__ RowPos row_pos(const ConvGeo& g, int b) {
    const int k = find_example(g.blk_off, g.n, b);
    const int local = b - g.blk_off[k];
    const int ow = g.out_rects[4 * k + 3];
    const int by = local / ow, bx = local - by * ow;
    RowPos r;
    r.out = (int64_t)(g.out_rects[4 * k] + by) * g.out_w + g.out_rects[4 * k + 1] + bx;
    r.in0 = (int64_t)(g.in_rects[4 * k] + by * CBH) * g.in_w + g.in_rects[4 * k + 1] + bx * CBW;
    r.rem = ow - bx;
    return r;
}

// Block s0 + t, given block s0's position r0.
__device__ __forceinline__ BlockPos step_pos(const ConvGeo& g, const RowPos& r0, int s0, int t) {
    if (t < r0.rem) return BlockPos{r0.in0 + (int64_t)t * CBW, r0.out + t};
    const RowPos r = row_pos(g, s0 + t);
    return BlockPos{r.in0, r.out};
}

// Every kernel runs a wave per (group d, step of NG = 64 / OG consecutive
// blocks), with no LDS buffer and no barrier. Lane l holds inputs k = l,
// l + 64, ... of the K = bh * bw * H inputs of each block of the step (pixel
// k / H, channel d*H + k % H) with their OG weights, or weight-gradient sums,
// in registers; the step's data loads one step ahead.
template <int H, int OG>
struct ConvCfg {
    static constexpr int K = CBH * CBW * H, KL = (K + 63) / 64, NG = 64 / OG;
    static_assert(64 % OG == 0, "outputs per group");
};

// Canvas float index of input k of group d of the block at in0.
template <int H>
__device__ __forceinline__ int64_t in_index(int64_t in0, int in_w, int d, int k) {
    const int pix = k / H, j = k - pix * H, dyy = pix / CBW, dx = pix - dyy * CBW;
    return (in0 + (int64_t)dyy * in_w + dx) * (4 * H) + d * H + j;
}

// The step's inputs of group d: x[t][i] = input lane + 64 i of block s0 + t
// (zero past the last block or past K).
template <int H, int OG>
__device__ __forceinline__ void load_step(const ConvGeo& g, const float* __restrict__ y, int d, int lane, int s0,
                                          int lim, RowPos& r0,
                                          float (&x)[ConvCfg<H, OG>::NG][ConvCfg<H, OG>::KL]) {
    using Cg = ConvCfg<H, OG>;
    r0 = row_pos(g, s0);
#pragma unroll
    for (int t = 0; t < Cg::NG; ++t) {
        const bool live = s0 + t < lim;
        const BlockPos P = live ? step_pos(g, r0, s0, t) : BlockPos{0, 0};
#pragma unroll
        for (int i = 0; i < Cg::KL; ++i) {
            const int k = lane + 64 * i;
            x[t][i] = live && k < Cg::K ? y[in_index<H>(P.in0, g.in_w, d, k)] : 0.0f;
        }
    }
}

// Sums a[v] over the 64 lanes of the wave and leaves the sum for v = lane in
// a[0]: each halving step keeps the half of the values selected by one lane
// bit and adds the partner lane's copy of that half (fixed order).
template <int C>
__device__ __forceinline__ void reduce_scatter_step(float (&a)[64], int lane) {
    constexpr int HALF = C / 2;
    const bool up = (lane & HALF) != 0;
#pragma unroll
    for (int j = 0; j < HALF; ++j) {
        const float mine = up ? a[HALF + j] : a[j], other = up ? a[j] : a[HALF + j];
        a[j] = mine + __shfl_xor(other, HALF);
    }
}

__device__ __forceinline__ float reduce_scatter64(float (&a)[64], int lane) {
    reduce_scatter_step<64>(a, lane);
    reduce_scatter_step<32>(a, lane);
    reduce_scatter_step<16>(a, lane);
    reduce_scatter_step<8>(a, lane);
    reduce_scatter_step<4>(a, lane);
    reduce_scatter_step<2>(a, lane);
    return a[0];
}

// Forward: out[d*OG + o] = tanh(b[d][o] + sum_k W[d][o][k] in_d[k]). A lane's
// partial sums for the step's NG x OG outputs are summed over the wave by a
// reduce-scatter that leaves output (t, o) = (lane / OG, lane % OG) in lane l.
template <int H, int OG>
__global__ void __launch_bounds__(256)
k_conv_fwd(const float* __restrict__ y, const float* __restrict__ W, const float* __restrict__ bias, ConvGeo geo,
           float* __restrict__ out) {
    using Cg = ConvCfg<H, OG>;
    constexpr int K = Cg::K, KL = Cg::KL, NG = Cg::NG;
    const int d = threadIdx.x >> 6, lane = threadIdx.x & 63, to = lane / OG, oo = lane % OG;
    float w[KL][OG];
#pragma unroll
    for (int i = 0; i < KL; ++i) {
        const int k = lane + 64 * i;
#pragma unroll
        for (int o = 0; o < OG; ++o) w[i][o] = k < K ? W[((int64_t)d * OG + o) * K + k] : 0.0f;
    }
    const float bo = bias[d * OG + oo];
    const int nb = geo.blk_off[geo.n], nst = (nb + NG - 1) / NG;
    float x[NG][KL];
    RowPos r0;
    int st = blockIdx.x;
    if (st < nst) load_step<H, OG>(geo, y, d, lane, st * NG, nb, r0, x);
    for (; st < nst; st += gridDim.x) {
        float a[64];
#pragma unroll
        for (int t = 0; t < NG; ++t)
#pragma unroll
            for (int o = 0; o < OG; ++o) {
                float acc = 0.0f;
#pragma unroll
                for (int i = 0; i < KL; ++i) acc += w[i][o] * x[t][i];
                a[t * OG + o] = acc;
            }
        const RowPos rc = r0;
        const int s0 = st * NG;
        if (st + (int)gridDim.x < nst) load_step<H, OG>(geo, y, d, lane, (st + gridDim.x) * NG, nb, r0, x);
        const float v = reduce_scatter64(a, lane);
        if (s0 + to < nb) {
            const BlockPos P = step_pos(geo, rc, s0, to);
            out[P.out * (4 * OG) + d * OG + oo] = tanhf(v + bo);
        }
    }
}

// Backward, input gradient: g[o] = dout[o] (1 - out[o]^2),
// dy[pixel][d*H + j] = sum_o g[o] W[d][o][(dy*bw+dx)*H + j]. Lane (t, o)
// loads block t's g[o] (one step ahead); the g values reach every lane as
// scalars.
template <int H, int OG>
__global__ void __launch_bounds__(256)
k_conv_bwd_dy(const float* __restrict__ out, const float* __restrict__ dout, const float* __restrict__ W,
              ConvGeo geo, float* __restrict__ dy) {
    using Cg = ConvCfg<H, OG>;
    constexpr int K = Cg::K, KL = Cg::KL, NG = Cg::NG;
    const int d = threadIdx.x >> 6, lane = threadIdx.x & 63, tb = lane / OG, ob = lane % OG;
    float w[KL][OG];
#pragma unroll
    for (int i = 0; i < KL; ++i) {
        const int k = min(lane + 64 * i, K - 1);
#pragma unroll
        for (int o = 0; o < OG; ++o) w[i][o] = W[((int64_t)d * OG + o) * K + k];
    }
    const int nb = geo.blk_off[geo.n], nst = (nb + NG - 1) / NG;
    RowPos r0;
    float ov = 0.0f, gv = 0.0f;
    auto fetch = [&](int st) {
        const int s0 = st * NG;
        r0 = row_pos(geo, s0);
        ov = gv = 0.0f;
        if (s0 + tb < nb) {
            const BlockPos P = step_pos(geo, r0, s0, tb);
            ov = out[P.out * (4 * OG) + d * OG + ob];
            gv = dout[P.out * (4 * OG) + d * OG + ob];
        }
    };
    int st = blockIdx.x;
    if (st < nst) fetch(st);
    for (; st < nst; st += gridDim.x) {
        const float gl = gv * (1.0f - ov * ov);
        const RowPos rc = r0;
        const int s0 = st * NG, cnt = min(NG, nb - s0);
        if (st + (int)gridDim.x < nst) fetch(st + gridDim.x);
#pragma unroll
        for (int t = 0; t < NG; ++t) {
            if (t < cnt) {
                float g[OG];
#pragma unroll
                for (int o = 0; o < OG; ++o)
                    g[o] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gl), t * OG + o));
                const BlockPos P = step_pos(geo, rc, s0, t);
#pragma unroll
                for (int i = 0; i < KL; ++i) {
                    const int k = lane + 64 * i;
                    if (k < K) {
                        float a = 0.0f;
#pragma unroll
                        for (int o = 0; o < OG; ++o) a += g[o] * w[i][o];
                        dy[in_index<H>(P.in0, geo.in_w, d, k)] = a;
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Backward, weight and bias gradients. Workgroup c sums blocks
// [c*per, (c+1)*per) in order into partial[c][4*OG*K + 4*OG] (entry
// (d, o, k) at (d*OG + o)*K + k, then the biases): lane l of wave d
// accumulates g[o] in_d[k] for its inputs k and every o, and lane (t, o) the
// g[o] of the step's block t, added over t at the end. A second kernel adds
// the partials in chunk order, so the result does not depend on scheduling.
// ---------------------------------------------------------------------------
template <int H, int OG>
__global__ void __launch_bounds__(256)
k_conv_bwd_dw(const float* __restrict__ y, const float* __restrict__ out, const float* __restrict__ dout,
              ConvGeo geo, int per, float* __restrict__ partial) {
    using Cg = ConvCfg<H, OG>;
    constexpr int K = Cg::K, KL = Cg::KL, NG = Cg::NG, M = 4 * OG * K;
    const int d = threadIdx.x >> 6, lane = threadIdx.x & 63, tb = lane / OG, ob = lane % OG;
    const int nb = geo.blk_off[geo.n];
    const int b0 = blockIdx.x * per, b1 = min(nb, b0 + per);
    float acc[KL][OG];
#pragma unroll
    for (int i = 0; i < KL; ++i)
#pragma unroll
        for (int o = 0; o < OG; ++o) acc[i][o] = 0.0f;
    float accb = 0.0f;
    float x[NG][KL];
    float ov = 0.0f, gv = 0.0f;
    auto fetch = [&](int s0) {
        RowPos r0;
        load_step<H, OG>(geo, y, d, lane, s0, b1, r0, x);
        ov = gv = 0.0f;
        if (s0 + tb < b1) {
            const BlockPos P = step_pos(geo, r0, s0, tb);
            ov = out[P.out * (4 * OG) + d * OG + ob];
            gv = dout[P.out * (4 * OG) + d * OG + ob];
        }
    };
    if (b0 < b1) fetch(b0);
    for (int s0 = b0; s0 < b1; s0 += NG) {
        const float gl = gv * (1.0f - ov * ov);  // zero past b1, as are the inputs
        float xc[NG][KL];
#pragma unroll
        for (int t = 0; t < NG; ++t)
#pragma unroll
            for (int i = 0; i < KL; ++i) xc[t][i] = x[t][i];
        if (s0 + NG < b1) fetch(s0 + NG);
        accb += gl;
#pragma unroll
        for (int t = 0; t < NG; ++t)
#pragma unroll
            for (int o = 0; o < OG; ++o) {
                const float g = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gl), t * OG + o));
#pragma unroll
                for (int i = 0; i < KL; ++i) acc[i][o] += g * xc[t][i];
            }
    }
#pragma unroll
    for (int m = OG; m < 64; m <<= 1) accb += __shfl_xor(accb, m);
    float* pc = partial + (size_t)blockIdx.x * (M + 4 * OG);
#pragma unroll
    for (int i = 0; i < KL; ++i) {
        const int k = lane + 64 * i;
        if (k < K) {
#pragma unroll
            for (int o = 0; o < OG; ++o) pc[((int64_t)d * OG + o) * K + k] = acc[i][o];
        }
    }
    if (tb == 0) pc[M + d * OG + ob] = accb;
}

// Fixed-order sum of the chunk partials: a block takes 64 consecutive
// outputs; its four thread groups sum every fourth chunk each (loads batched
// 32 at a time), and the four sums are added in a fixed order.
__global__ void __launch_bounds__(256)
k_sum_partials(const float* __restrict__ partial, int chunks, int m, float* __restrict__ dw,
               float* __restrict__ db, int mw) {
    __shared__ float ps[4][64];
    const int t = threadIdx.x & 63, grp = threadIdx.x >> 6;
    const int i = blockIdx.x * 64 + t;
    float s = 0.0f;
    if (i < m) {
        int c = grp;
        for (; c + 124 < chunks; c += 128) {
            float v[32];
#pragma unroll
            for (int k = 0; k < 32; ++k) v[k] = partial[(size_t)(c + 4 * k) * m + i];
#pragma unroll
            for (int k = 0; k < 32; ++k) s += v[k];
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

// Workgroups of 256 threads of `kernel` that the device holds at once (2048
// if the runtime cannot say; its error is then cleared, so that it is not
// reported for the launch that follows).
template <typename K>
static int resident_workgroups(K kernel) {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, 256, 0) != hipSuccess || per_cu < 1 ||
        hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) {
        (void)hipGetLastError();
        return 2048;
    }
    return per_cu * cus;
}

template <int H, int OG>
static hipError_t conv_launch(bool fwd, const ConvArgs& a, hipStream_t s) {
    if constexpr (4 * OG * CBH * CBW * H * 4 > 64 * 1024) {
        return hipErrorInvalidValue;  // rejected by conv_supported
    } else {
        constexpr int K = CBH * CBW * H;
        const ConvGeo geo{a.blk_off, a.n, a.in_rects, a.in_w, a.out_rects, a.out_w};
        // one round of resident workgroups (each loads its weights once and
        // then strides over the steps), or one per step if there are fewer
        constexpr int NG = ConvCfg<H, OG>::NG;
        const int steps = (a.total_blocks + NG - 1) / NG;
        if (fwd) {
            static const int resident = resident_workgroups(k_conv_fwd<H, OG>);
            const unsigned grid = (unsigned)std::min(steps, resident);
            hipLaunchKernelGGL((k_conv_fwd<H, OG>), dim3(grid), dim3(256), 0, s, a.y, a.w, a.b, geo, a.out);
            return hipGetLastError();
        }
        static const int resident = resident_workgroups(k_conv_bwd_dy<H, OG>);
        const unsigned grid = (unsigned)std::min(steps, resident);
        hipLaunchKernelGGL((k_conv_bwd_dy<H, OG>), dim3(grid), dim3(256), 0, s, a.out, a.dout, a.w, geo, a.dy);
        const int chunks = conv_chunks(a.total_blocks);
        const int per = (a.total_blocks + chunks - 1) / chunks;
        hipLaunchKernelGGL((k_conv_bwd_dw<H, OG>), dim3(chunks), dim3(256), 0, s, a.y, a.out, a.dout, geo, per,
                           a.partial);
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
