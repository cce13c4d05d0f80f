// Output layer shared by the four scan directions, the collapse of the rows,
// and the CTC loss (Section II: the last fully-connected layer is shared
// across directions, the model is trained with connectionist temporal
// classification; Section V-B treats that layer as a block-strided layer with
// 1 x 1 blocks, so it runs straight on the packed canvas).
//
// For example i at rectangle (y0, x0, h, w) of the last layer's output canvas
// Y [canvas][4H] (channel d*H + j), frame t = 0 .. w - 1 is column x0 + t:
//   S[t]      = sum_y sum_d h_d(y0 + y, x0 + t)              (H values)
//   logits[t] = W S[t] + 4 h b                                (K values)
// which is sum_y sum_d (W h_d + b): the shared layer applied to every cell of
// every direction, summed over the directions and the rows. Class 0 is the
// CTC blank.
//
// CTC (Graves et al. 2006), one workgroup per example, in double precision:
// log-softmax per frame; the forward variables alpha_t(s) over the extended
// label l' (blanks around and between the labels, S = 2L + 1 states) frame by
// frame; log p = logsumexp(alpha_{T-1}(S-1), alpha_{T-1}(S-2)); then the
// backward variables beta_t(s) frame by frame from the last, and at each frame
// the gradient of -ln p with respect to the scores,
//   dlogits[t][k] = softmax_t(k) - sum_{s: l'_s = k} exp(alpha_t(s) + beta_t(s) - lp_t(k) - log p),
// summed in ascending s (blanks by a fixed-order wave reduction).
#include <math.h>

#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

namespace {

constexpr int HT = 256;  // threads per workgroup
constexpr int HC = 64;   // frames (columns) per tile
constexpr int DWF = 64;   // frames per weight-gradient chunk

__device__ __forceinline__ double lse2(double a, double b) {
    const double m = fmax(a, b);
    if (m == -INFINITY) return -INFINITY;
    return m + log(exp(a - m) + exp(b - m));
}

__device__ __forceinline__ double lse3(double a, double b, double c) {
    const double m = fmax(fmax(a, b), c);
    if (m == -INFINITY) return -INFINITY;
    return m + log(exp(a - m) + exp(b - m) + exp(c - m));
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ __forceinline__ double wave_max(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
    return v;
}

}  // namespace

// Forward: tile j covers frames [t0, t0 + HC) of example tiles[2j] (t0 =
// tiles[2j + 1]). Writes logits [frames][K] and S [frames][H + 4] (S[.][H] =
// 4h, the bias's multiplier; the last three columns zero).
__global__ void __launch_bounds__(HT)
k_head_fwd(int H, int K, int canvas_w, const float* __restrict__ Y, const int32_t* __restrict__ rects,
           const int32_t* __restrict__ frame_off, const int32_t* __restrict__ tiles, const float* __restrict__ W,
           const float* __restrict__ b, float* __restrict__ logits, float* __restrict__ S) {
    extern __shared__ __attribute__((aligned(16))) float hsm[];
    float* sW = hsm;         // [K][H]
    float* sS = sW + K * H;  // [HC][H]
    const int tid = threadIdx.x;
    const int ex = tiles[2 * blockIdx.x], t0 = tiles[2 * blockIdx.x + 1];
    const int y0 = rects[4 * ex], x0 = rects[4 * ex + 1], h = rects[4 * ex + 2], w = rects[4 * ex + 3];
    const int nc = min(HC, w - t0);
    for (int e = tid; e < K * H; e += HT) sW[e] = W[e];
    // column sums: slot e = (cell c, hidden units 4 j4 .. 4 j4 + 3); each slot
    // sums its four directions' channels d*H + 4 j4 over the rows, then the
    // directions in a fixed order
    const int H4 = H / 4, slots = HC * H4;
    for (int e = tid; e < slots; e += HT) {
        const int c = e / H4, j4 = e - c * H4;
        float4 a[4];
#pragma unroll
        for (int d = 0; d < 4; ++d) a[d] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (c < nc) {
            const float* p = Y + ((int64_t)y0 * canvas_w + x0 + t0 + c) * (4 * H) + 4 * j4;
            for (int y = 0; y < h; ++y) {
                const float* q = p + (int64_t)y * canvas_w * (4 * H);
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    const float4 v = *reinterpret_cast<const float4*>(q + d * H);
                    a[d].x += v.x;
                    a[d].y += v.y;
                    a[d].z += v.z;
                    a[d].w += v.w;
                }
            }
        }
        float4 t;
        t.x = ((a[0].x + a[1].x) + a[2].x) + a[3].x;
        t.y = ((a[0].y + a[1].y) + a[2].y) + a[3].y;
        t.z = ((a[0].z + a[1].z) + a[2].z) + a[3].z;
        t.w = ((a[0].w + a[1].w) + a[2].w) + a[3].w;
        *reinterpret_cast<float4*>(&sS[c * H + 4 * j4]) = t;
    }
    __syncthreads();
    const int f0 = frame_off[ex] + t0;
    const int SP = H + 4;
    for (int e = tid; e < nc * SP; e += HT) {
        const int c = e / SP, j = e - c * SP;
        S[(int64_t)(f0 + c) * SP + j] = j < H ? sS[c * H + j] : (j == H ? 4.0f * h : 0.0f);
    }
    for (int e = tid; e < nc * K; e += HT) {
        const int c = e / K, k = e - c * K;
        const float* wk = &sW[k * H];
        const float* sv = &sS[c * H];
        float acc = 0.0f;
        for (int j = 0; j < H; ++j) acc = fmaf(wk[j], sv[j], acc);
        logits[(int64_t)(f0 + c) * K + k] = acc + 4.0f * h * b[k];
    }
}

// CTC loss and gradient of one example per workgroup (see the file comment).
// lab_off[i] / frame_off[i]: first label / frame of example i; a_off[i]: first
// double of its alpha table [T][S]; lp: log-softmax workspace [frames][K].
__global__ void __launch_bounds__(HT)
k_ctc(int K, const int32_t* __restrict__ frame_off, const int32_t* __restrict__ lab_off,
      const int32_t* __restrict__ labels, const int64_t* __restrict__ a_off, const float* __restrict__ logits,
      double* __restrict__ lp_ws, double* __restrict__ alpha_ws, float* __restrict__ losses,
      float* __restrict__ dlogits) {
    extern __shared__ __attribute__((aligned(16))) double csm[];
    const int ex = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int f0 = frame_off[ex], T = frame_off[ex + 1] - f0;
    const int L = lab_off[ex + 1] - lab_off[ex], S = 2 * L + 1;
    double* A0 = csm;        // [S]
    double* A1 = A0 + S;     // [S]
    double* G = A1 + S;      // [S]
    __shared__ double s_logp;
    int32_t* lab = reinterpret_cast<int32_t*>(G + S);  // [S]
    int32_t* nxt = lab + S;                              // [S]
    int32_t* first = nxt + S;                            // [K]
    const int32_t* lb = labels + lab_off[ex];
    for (int s = tid; s < S; s += HT) lab[s] = (s & 1) ? lb[s >> 1] : 0;
    for (int k = tid; k < K; k += HT) first[k] = -1;
    __syncthreads();
    if (tid == 0) {  // occurrence lists of the labels (the odd states), ascending s
        for (int s = S - 2; s >= 1; s -= 2) {
            nxt[s] = first[lab[s]];
            first[lab[s]] = s;
        }
    }
    // log-softmax of every frame, one wave per frame
    double* lp = lp_ws + (int64_t)f0 * K;
    for (int t = wave; t < T; t += HT / 64) {
        const float* z = logits + (int64_t)(f0 + t) * K;
        double m = -INFINITY;
        for (int k = lane; k < K; k += 64) m = fmax(m, (double)z[k]);
        m = wave_max(m);
        double se = 0.0;
        for (int k = lane; k < K; k += 64) se += exp((double)z[k] - m);
        se = wave_sum(se);
        const double ls = m + log(se);
        for (int k = lane; k < K; k += 64) lp[(int64_t)t * K + k] = (double)z[k] - ls;
    }
    __syncthreads();  // lp (global, this workgroup's) and the lists are complete
    double* al = alpha_ws + a_off[ex];
    auto skip_ok = [&](int s) { return s >= 2 && (s & 1) && lab[s] != lab[s - 2]; };
    // alpha
    for (int s = tid; s < S; s += HT) {
        const double v = s < 2 ? lp[lab[s]] : -INFINITY;
        A0[s] = v;
        al[s] = v;
    }
    __syncthreads();
    double* ap = A0;
    double* ac = A1;
    for (int t = 1; t < T; ++t) {
        const double* lpt = lp + (int64_t)t * K;
        for (int s = tid; s < S; s += HT) {
            const double a = ap[s], b1 = s >= 1 ? ap[s - 1] : -INFINITY;
            const double v = (skip_ok(s) ? lse3(a, b1, ap[s - 2]) : lse2(a, b1)) + lpt[lab[s]];
            ac[s] = v;
            al[(int64_t)t * S + s] = v;
        }
        __syncthreads();
        double* tmp = ap;
        ap = ac;
        ac = tmp;
    }
    if (tid == 0) {
        s_logp = S > 1 ? lse2(ap[S - 1], ap[S - 2]) : ap[0];
        losses[ex] = (float)(-s_logp);
    }
    __syncthreads();
    const double logp = s_logp;
    // beta and the gradient, from the last frame back
    double* bc = ac;  // beta of frame t
    double* bp = ap;  // beta of frame t - 1 (free: alpha is in global memory)
    {
        const double* lpt = lp + (int64_t)(T - 1) * K;
        for (int s = tid; s < S; s += HT) bc[s] = s >= S - 2 ? lpt[lab[s]] : -INFINITY;
    }
    __syncthreads();
    for (int t = T - 1; t >= 0; --t) {
        const double* lpt = lp + (int64_t)t * K;
        for (int s = tid; s < S; s += HT) {
            const double v = al[(int64_t)t * S + s] + bc[s] - lpt[lab[s]] - logp;
            G[s] = v == -INFINITY ? 0.0 : exp(v);
        }
        __syncthreads();
        float* dz = dlogits + (int64_t)(f0 + t) * K;
        if (wave == 0) {  // the blank: the even states, a fixed-order reduction
            double o = 0.0;
            for (int s = 2 * lane; s < S; s += 128) o += G[s];
            o = wave_sum(o);
            if (lane == 0) dz[0] = (float)(exp(lpt[0]) - o);
        } else {
            for (int k = 1 + (tid - 64); k < K; k += HT - 64) {
                double o = 0.0;
                for (int s = first[k]; s >= 0; s = nxt[s]) o += G[s];
                dz[k] = (float)(exp(lpt[k]) - o);
            }
        }
        if (t > 0) {
            const double* lpp = lp + (int64_t)(t - 1) * K;
            for (int s = tid; s < S; s += HT) {
                const double a = bc[s], b1 = s + 1 < S ? bc[s + 1] : -INFINITY;
                const bool sk = s + 2 < S && (s & 1) && lab[s] != lab[s + 2];
                bp[s] = (sk ? lse3(a, b1, bc[s + 2]) : lse2(a, b1)) + lpp[lab[s]];
            }
        }
        __syncthreads();
        double* tmp = bc;
        bc = bp;
        bp = tmp;
    }
}

// Backward, input gradient: every row of frame t's column, in every
// direction, receives W^T dlogits[t] (the canvas is zeroed beforehand).
__global__ void __launch_bounds__(HT)
k_head_bwd_dy(int H, int K, int canvas_w, const int32_t* __restrict__ rects, const int32_t* __restrict__ frame_off,
              const int32_t* __restrict__ tiles, const float* __restrict__ W, const float* __restrict__ dlogits,
              float* __restrict__ dY) {
    extern __shared__ __attribute__((aligned(16))) float hsm[];
    float* sW = hsm;         // [K][H]
    float* sG = sW + K * H;  // [HC][H]
    const int tid = threadIdx.x;
    const int ex = tiles[2 * blockIdx.x], t0 = tiles[2 * blockIdx.x + 1];
    const int y0 = rects[4 * ex], x0 = rects[4 * ex + 1], h = rects[4 * ex + 2], w = rects[4 * ex + 3];
    const int nc = min(HC, w - t0);
    const int f0 = frame_off[ex] + t0;
    for (int e = tid; e < K * H; e += HT) sW[e] = W[e];
    __syncthreads();
    for (int e = tid; e < nc * H; e += HT) {
        const int c = e / H, j = e - c * H;
        const float* dz = dlogits + (int64_t)(f0 + c) * K;
        float acc = 0.0f;
        for (int k = 0; k < K; ++k) acc = fmaf(sW[k * H + j], dz[k], acc);
        sG[e] = acc;
    }
    __syncthreads();
    const int slots = nc * H;  // float4 slots of one row segment: nc cells x 4H channels
    for (int y = 0; y < h; ++y) {
        float* row = dY + ((int64_t)(y0 + y) * canvas_w + x0 + t0) * (4 * H);
        for (int e = tid; e < slots; e += HT) {
            const int c = e / H, q = e - c * H;
            const int j = (4 * q) % H;  // channels 4q .. 4q + 3 are units j .. j + 3 of direction 4q / H
            *reinterpret_cast<float4*>(row + (int64_t)c * 4 * H + 4 * q) = *reinterpret_cast<const float4*>(&sG[c * H + j]);
        }
    }
}

// Backward, weight gradients: chunk c of DWF frames adds
// part[c][k][j] = sum_t dlogits[t][k] S[t][j], j <= H (column H: the bias).
__global__ void __launch_bounds__(HT)
k_head_bwd_dw(int H, int K, int frames, const float* __restrict__ dlogits, const float* __restrict__ S,
              float* __restrict__ part) {
    extern __shared__ __attribute__((aligned(16))) float hsm[];
    const int SP = H + 4, NJ = H + 1;
    float* sD = hsm;            // [DWF][K]
    float* sS = sD + DWF * K;   // [DWF][SP]
    const int tid = threadIdx.x;
    const int fb = blockIdx.x * DWF, nf = min(DWF, frames - fb);
    for (int e = tid; e < nf * K; e += HT) sD[e] = dlogits[(int64_t)fb * K + e];
    for (int e = tid; e < nf * SP; e += HT) sS[e] = S[(int64_t)fb * SP + e];
    __syncthreads();
    float* out = part + (int64_t)blockIdx.x * K * NJ;
    for (int e = tid; e < K * NJ; e += HT) {
        const int k = e / NJ, j = e - k * NJ;
        float acc = 0.0f;
        for (int t = 0; t < nf; ++t) acc = fmaf(sD[t * K + k], sS[t * SP + j], acc);
        out[e] = acc;
    }
}

__global__ void k_head_dw_reduce(int H, int K, int chunks, const float* __restrict__ part, float* __restrict__ dW,
                                 float* __restrict__ db) {
    const int NJ = H + 1;
    for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < K * NJ; e += gridDim.x * blockDim.x) {
        float s = 0.0f;
        for (int c = 0; c < chunks; ++c) s += part[(int64_t)c * K * NJ + e];
        const int k = e / NJ, j = e - k * NJ;
        if (j < H) dW[k * H + j] = s;
        else db[k] = s;
    }
}

__global__ void k_zero_f4(float4* __restrict__ p, int64_t n4) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

__global__ void k_zero_f(float* __restrict__ p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0.0f;
}

// --- host ------------------------------------------------------------------------
int head_tile_frames() { return HC; }
int head_dw_chunk_frames() { return DWF; }

size_t head_fwd_lds(int H, int K) { return (size_t)(K * H + HC * H) * 4; }
size_t head_bwd_lds(int H, int K) { return (size_t)(K * H + HC * H) * 4; }
size_t head_dw_lds(int H, int K) { return (size_t)(DWF * K + DWF * (H + 4)) * 4; }
size_t ctc_lds(int max_labels, int K) {
    const int S = 2 * max_labels + 1;
    return (size_t)3 * S * 8 + (size_t)(2 * S + K) * 4;
}

hipError_t launch_head_fwd(const HeadArgs& a, hipStream_t s) {
    if (a.n_tiles == 0) return hipSuccess;
    hipLaunchKernelGGL(k_head_fwd, dim3(a.n_tiles), dim3(HT), head_fwd_lds(a.H, a.K), s, a.H, a.K, a.canvas_w, a.y,
                       a.rects, a.frame_off, a.tiles, a.w, a.b, a.logits, a.S);
    return hipGetLastError();
}

hipError_t launch_ctc(const CtcArgs& a, hipStream_t s) {
    if (a.n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_ctc, dim3(a.n), dim3(HT), ctc_lds(a.max_labels, a.K), s, a.K, a.frame_off, a.lab_off,
                       a.labels, a.a_off, a.logits, a.lp, a.alpha, a.losses, a.dlogits);
    return hipGetLastError();
}

hipError_t launch_head_bwd(const HeadArgs& a, int64_t canvas_floats, hipStream_t s) {
    if (canvas_floats > 0) {
        const int zb = (int)std::min<int64_t>((canvas_floats / 4 + 255) / 256, 8192);
        hipLaunchKernelGGL(k_zero_f4, dim3(zb), dim3(256), 0, s, reinterpret_cast<float4*>(a.dy), canvas_floats / 4);
    }
    if (a.n_tiles > 0)
        hipLaunchKernelGGL(k_head_bwd_dy, dim3(a.n_tiles), dim3(HT), head_bwd_lds(a.H, a.K), s, a.H, a.K,
                           a.canvas_w, a.rects, a.frame_off, a.tiles, a.w, a.dlogits, a.dy);
    const int chunks = (a.frames + DWF - 1) / DWF;
    if (chunks > 0)
        hipLaunchKernelGGL(k_head_bwd_dw, dim3(chunks), dim3(HT), head_dw_lds(a.H, a.K), s, a.H, a.K, a.frames,
                           a.dlogits, a.S, a.part);
    const int nj = a.K * (a.H + 1);
    if (chunks > 0) {
        hipLaunchKernelGGL(k_head_dw_reduce, dim3((nj + 255) / 256), dim3(256), 0, s, a.H, a.K, chunks, a.part, a.dw,
                           a.db);
    } else {  // no frames: zero gradients
        hipLaunchKernelGGL(k_zero_f, dim3((a.K * a.H + 255) / 256), dim3(256), 0, s, a.dw, a.K * a.H);
        hipLaunchKernelGGL(k_zero_f, dim3((a.K + 255) / 256), dim3(256), 0, s, a.db, a.K);
    }
    return hipGetLastError();
}

}  // namespace mdl
