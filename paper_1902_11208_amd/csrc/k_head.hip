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
// CTC (Graves et al. 2006) in double precision, with the rescaled forward
// and backward variables of that paper (each frame's variables divided by
// their sum, the logarithms of the sums accumulated), over the extended label
// l' (blanks around and between the labels, S = 2L + 1 states):
//   1. softmax y_t of every frame (one wave per frame, all frames at once);
//   2. per example, one wave runs the forward variables
//        a_t(s) = (a_{t-1}(s) + a_{t-1}(s-1) [+ a_{t-1}(s-2)]) y_t(l'_s),
//      the skip allowed where l'_s is a label different from l'_{s-2}, and
//      -ln p = -(sum_t ln C_t + ln(a_{T-1}(S-1) + a_{T-1}(S-2))), C_t the
//      sum of frame t's unscaled variables; a second wave runs the backward
//      variables without the current frame's output,
//        b_{t-1}(s) = b_t(s) y_t(l'_s) + b_t(s+1) y_t(l'_{s+1}) [+ b_t(s+2) y_t(l'_{s+2})];
//      both store every frame's rescaled variables;
//   3. per frame, the state posteriors g_t(s) = a_t(s) b_t(s) / sum_s a_t(s) b_t(s)
//      give the gradient of -ln p with respect to the logits,
//        dlogits[t][k] = y_t(k) - sum_{s: l'_s = k} g_t(s),
//      summed in ascending s (the blank's states by a fixed-order wave
//      reduction).
// The rescaling keeps every variable in range without a logarithm or an
// exponential on the sequential path.
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

// CTC step 1: softmax of frame f (one wave per frame), y [frames][K].
__global__ void __launch_bounds__(256)
k_ctc_softmax(int64_t frames, int K, const float* __restrict__ logits, double* __restrict__ y) {
    const int lane = threadIdx.x & 63;
    const int64_t f = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (f >= frames) return;
    const float* z = logits + f * K;
    double m = -INFINITY;
    for (int k = lane; k < K; k += 64) m = fmax(m, (double)z[k]);
    m = wave_max(m);
    double se = 0.0;
    for (int k = lane; k < K; k += 64) se += exp((double)z[k] - m);
    const double inv = 1.0 / wave_sum(se);
    for (int k = lane; k < K; k += 64) y[f * K + k] = exp((double)z[k] - m) * inv;
}

// A nonnegative number as a double mantissa (0, or in [0.5, 1)) and an int
// exponent: the CTC variables span far more than the double range (states
// behind and ahead of the bulk of the probability), so each keeps its own
// exponent and no frame needs rescaling.
constexpr int XNEG = -(1 << 30);  // exponent of zero
struct Xd {
    double m;
    int e;
};
__device__ __forceinline__ Xd xnorm(double v, int e) {
    int d;
    const double m = frexp(v, &d);
    return m == 0.0 ? Xd{0.0, XNEG} : Xd{m, e + d};
}
// a + b + c (c only with `with_c`), aligned to the largest exponent
__device__ __forceinline__ Xd xsum3(Xd a, Xd b, Xd c, bool with_c) {
    int E = max(a.e, b.e);
    if (with_c) E = max(E, c.e);
    double v = ldexp(a.m, a.e - E) + ldexp(b.m, b.e - E);
    if (with_c) v += ldexp(c.m, c.e - E);
    return xnorm(v, E);
}
__device__ __forceinline__ Xd xshfl_up(Xd v, int d) { return Xd{__shfl_up(v.m, d), __shfl_up(v.e, d)}; }
__device__ __forceinline__ Xd xshfl_down(Xd v, int d) { return Xd{__shfl_down(v.m, d), __shfl_down(v.e, d)}; }

// CTC step 2: wave 0 the forward variables, wave 1 the backward ones, of
// example blockIdx.x; lane l owns states l*NM .. l*NM + NM - 1 and stores
// them for every frame into rows of 64 NM entries (mantissas am / bm
// [frames][64 NM], exponents ae / be). Frame rows of y are loaded D frames
// ahead; every frame issues the same loads and stores, so the waits are for
// exactly those loads.
template <int NM, int D>
__global__ void __launch_bounds__(128)
k_ctc_scan(int K, const int32_t* __restrict__ frame_off, const int32_t* __restrict__ lab_off,
           const int32_t* __restrict__ labels, const double* __restrict__ y, double* __restrict__ am,
           int32_t* __restrict__ ae, double* __restrict__ bm, int32_t* __restrict__ be, float* __restrict__ losses) {
    constexpr int RS = 64 * NM;
    __shared__ double ys[2][2][2 * 64];  // per wave: y rows by frame parity (K <= 128)
    __shared__ double finm[RS];          // the forward variables of the last frame
    __shared__ int fine[RS];
    const int ex = blockIdx.x, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int f0 = frame_off[ex], T = frame_off[ex + 1] - f0;
    const int lo = lab_off[ex], L = lab_off[ex + 1] - lo, S = 2 * L + 1;
    // the lane's states: class, valid, skip into s (from s - 2), skip out of s (into s + 2)
    int cls[NM];
    uint32_t vm = 0, skin = 0, skout = 0;
#pragma unroll
    for (int i = 0; i < NM; ++i) {
        const int st = lane * NM + i;
        const bool v = st < S;
        const bool lab = v && (st & 1);
        cls[i] = lab ? labels[lo + (st >> 1)] : 0;
        vm |= (uint32_t)v << i;
        if (lab && st >= 3 && cls[i] != labels[lo + (st >> 1) - 1]) skin |= 1u << i;
        if (lab && st + 2 < S && labels[lo + (st >> 1) + 1] != cls[i]) skout |= 1u << i;
    }
    const double* yb = y + (int64_t)f0 * K;
    const int k0 = min(lane, K - 1), k1 = min(lane + 64, K - 1);  // the lane's y columns (clamped)
    double* yl0 = ys[wave][0];
    double* yl1 = ys[wave][1];
    const Xd zero{0.0, XNEG};
    Xd v[NM];
    double r0[D], r1[D];
    if (wave == 0) {
        double* ambase = am + (int64_t)f0 * RS + lane * NM;
        int32_t* aebase = ae + (int64_t)f0 * RS + lane * NM;
        auto store = [&](int t) {
#pragma unroll
            for (int i = 0; i < NM; ++i) {
                ambase[(int64_t)t * RS + i] = v[i].m;
                aebase[(int64_t)t * RS + i] = v[i].e;
            }
        };
        // frame 0: the first blank and the first label
        yl0[lane] = yb[k0];
        yl0[lane + 64] = yb[k1];
#pragma unroll
        for (int i = 0; i < NM; ++i) {
            const int st = lane * NM + i;
            v[i] = ((vm >> i) & 1) && st < 2 ? xnorm(yl0[cls[i]], 0) : zero;
        }
        store(0);
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int t = min(1 + j, T - 1);
            r0[j] = yb[(int64_t)t * K + k0];
            r1[j] = yb[(int64_t)t * K + k1];
        }
        auto step = [&](int t, int j) {
            double* yl = (t & 1) ? yl1 : yl0;
            yl[lane] = r0[j];
            yl[lane + 64] = r1[j];
            const int tn = min(t + D, T - 1);
            r0[j] = yb[(int64_t)tn * K + k0];
            r1[j] = yb[(int64_t)tn * K + k1];
            Xd p1 = xshfl_up(v[NM - 1], 1);
            Xd p2 = NM >= 2 ? xshfl_up(v[NM >= 2 ? NM - 2 : 0], 1) : xshfl_up(v[NM - 1], 2);
            if (lane < 1) p1 = zero;
            if (lane < (NM >= 2 ? 1 : 2)) p2 = zero;
            Xd n[NM];
#pragma unroll
            for (int i = 0; i < NM; ++i) {
                const Xd m1 = i >= 1 ? v[i - 1] : p1;
                const Xd m2 = i >= 2 ? v[i - 2] : (i == 1 ? p1 : p2);
                const Xd x = xsum3(v[i], m1, m2, (skin >> i) & 1);
                n[i] = ((vm >> i) & 1) ? xnorm(x.m * yl[cls[i]], x.e) : zero;
            }
#pragma unroll
            for (int i = 0; i < NM; ++i) v[i] = n[i];
            store(t);
        };
        // whole rounds of D frames (the same loads and stores in each, so the
        // waits stay exact), then the remaining frames
        int tb = 1;
        for (; tb + D <= T; tb += D) {
#pragma unroll
            for (int j = 0; j < D; ++j) step(tb + j, j);
        }
#pragma unroll
        for (int j = 0; j < D; ++j)
            if (tb + j < T) step(tb + j, j);
        // -ln p from the last frame's variables at S - 1 and S - 2
#pragma unroll
        for (int i = 0; i < NM; ++i) {
            finm[lane * NM + i] = v[i].m;
            fine[lane * NM + i] = v[i].e;
        }
        if (lane == 0) {
            const Xd a1{finm[S - 1], fine[S - 1]};
            const Xd a2 = S >= 2 ? Xd{finm[S - 2], fine[S - 2]} : zero;
            const Xd p = xsum3(a1, a2, zero, false);
            losses[ex] = (float)(-(log(p.m) + p.e * 0.69314718055994530942));
        }
    } else {
        double* bmbase = bm + (int64_t)f0 * RS + lane * NM;
        int32_t* bebase = be + (int64_t)f0 * RS + lane * NM;
        auto store = [&](int t) {
#pragma unroll
            for (int i = 0; i < NM; ++i) {
                bmbase[(int64_t)t * RS + i] = v[i].m;
                bebase[(int64_t)t * RS + i] = v[i].e;
            }
        };
        // frame T - 1: 1 at the final blank and the last label
#pragma unroll
        for (int i = 0; i < NM; ++i) {
            const int st = lane * NM + i;
            v[i] = ((vm >> i) & 1) && st >= S - 2 ? Xd{0.5, 1} : zero;
        }
        store(T - 1);
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int t = max(T - 1 - j, 0);
            r0[j] = yb[(int64_t)t * K + k0];
            r1[j] = yb[(int64_t)t * K + k1];
        }
        // step t -> t - 1 uses y_t
        auto step = [&](int t, int j) {
            double* yl = (t & 1) ? yl1 : yl0;
            yl[lane] = r0[j];
            yl[lane + 64] = r1[j];
            const int tn = max(t - D, 0);
            r0[j] = yb[(int64_t)tn * K + k0];
            r1[j] = yb[(int64_t)tn * K + k1];
            Xd e[NM];
#pragma unroll
            for (int i = 0; i < NM; ++i) e[i] = xnorm(v[i].m * yl[cls[i]], v[i].e);
            Xd q1 = xshfl_down(e[0], 1);
            Xd q2 = NM >= 2 ? xshfl_down(e[NM >= 2 ? 1 : 0], 1) : xshfl_down(e[0], 2);
            if (lane >= 63) q1 = zero;
            if (lane >= (NM >= 2 ? 63 : 62)) q2 = zero;
#pragma unroll
            for (int i = 0; i < NM; ++i) {
                const Xd u1 = i + 1 < NM ? e[i + 1] : q1;
                const Xd u2 = i + 2 < NM ? e[i + 2] : (i + 1 < NM ? q1 : q2);
                v[i] = ((vm >> i) & 1) ? xsum3(e[i], u1, u2, (skout >> i) & 1) : zero;
            }
            store(t - 1);
        };
        int tb = T - 1;
        for (; tb - D + 1 >= 1; tb -= D) {
#pragma unroll
            for (int j = 0; j < D; ++j) step(tb - j, j);
        }
#pragma unroll
        for (int j = 0; j < D; ++j)
            if (tb - j >= 1) step(tb - j, j);
    }
}

// CTC step 3: the gradient of frame f (one wave per frame): state posteriors
// from the stored variables (products aligned to the largest exponent of the
// frame), per-class sums in ascending state order (the labels through occ:
// bit 30 marks a class's first occurrence in the example, bits 0-29 the next
// occurrence or all ones), dlogits = y - sums.
__global__ void __launch_bounds__(256)
k_ctc_grad(int n, int64_t frames, int K, int RS, const int32_t* __restrict__ frame_off,
           const int32_t* __restrict__ lab_off, const int32_t* __restrict__ labels, const int32_t* __restrict__ occ,
           const double* __restrict__ y, const double* __restrict__ am, const int32_t* __restrict__ ae,
           const double* __restrict__ bm, const int32_t* __restrict__ be, float* __restrict__ dlogits) {
    extern __shared__ __attribute__((aligned(16))) double gsm[];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t f = (int64_t)blockIdx.x * 4 + wave;
    if (f >= frames) return;
    double* g = gsm + (int64_t)wave * (RS + 128);  // posteriors of the frame's states
    double* dl = g + RS;                           // the frame's gradient row
    // example of frame f: the last i with frame_off[i] <= f
    int lo_i = 0, hi_i = n - 1;
    while (lo_i < hi_i) {
        const int mid = (lo_i + hi_i + 1) >> 1;
        if (frame_off[mid] <= f) lo_i = mid;
        else hi_i = mid - 1;
    }
    const int ex = lo_i;
    const int lo = lab_off[ex], L = lab_off[ex + 1] - lo, S = 2 * L + 1;
    const int64_t r = f * RS;
    int emax = XNEG;
    for (int st = lane; st < S; st += 64)
        if (am[r + st] != 0.0 && bm[r + st] != 0.0) emax = max(emax, ae[r + st] + be[r + st]);
    for (int o = 32; o > 0; o >>= 1) emax = max(emax, __shfl_xor(emax, o));
    double z = 0.0, zb = 0.0;  // all states, blank states (fixed order: lane's states ascending, then the butterfly)
    for (int st = lane; st < S; st += 64) {
        const double pm = am[r + st] * bm[r + st];
        const double x = pm == 0.0 ? 0.0 : ldexp(pm, ae[r + st] + be[r + st] - emax);
        g[st] = x;
        z += x;
        if (!(st & 1)) zb += x;
    }
    z = wave_sum(z);
    zb = wave_sum(zb);
    const double inv = 1.0 / z;
    const double* yr = y + f * K;
    for (int k = lane; k < K; k += 64) dl[k] = yr[k];
    if (lane == 0) dl[0] = yr[0] - zb * inv;
    for (int j = lane; j < L; j += 64) {
        const int o = occ[lo + j];
        if (!(o & (1 << 30))) continue;  // not the first occurrence of its class
        double sum = 0.0;
        for (int q = j; q >= 0;) {
            sum += g[2 * q + 1];
            const int nx = occ[lo + q] & 0x3fffffff;
            q = nx == 0x3fffffff ? -1 : nx;
        }
        const int k = labels[lo + j];
        dl[k] = yr[k] - sum * inv;
    }
    for (int k = lane; k < K; k += 64) dlogits[f * K + k] = (float)dl[k];
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

// Fixed-order sum of the chunk partials: a workgroup owns 64 consecutive
// outputs (one per lane); its four waves sum four consecutive ranges of the
// chunks (loads of 64 outputs per chunk are contiguous), and the ranges are
// added in order.
__global__ void __launch_bounds__(256)
k_head_dw_reduce(int H, int K, int chunks, const float* __restrict__ part, float* __restrict__ dW,
                 float* __restrict__ db) {
    __shared__ float acc[4][64];
    const int NJ = H + 1, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int e = blockIdx.x * 64 + lane;
    const int q = (chunks + 3) / 4, c0 = wave * q, c1 = min(chunks, c0 + q);
    float s = 0.0f;
    if (e < K * NJ) {
#pragma unroll 8
        for (int c = c0; c < c1; ++c) s += part[(int64_t)c * K * NJ + e];
    }
    acc[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && e < K * NJ) {
        const float t = ((acc[0][lane] + acc[1][lane]) + acc[2][lane]) + acc[3][lane];
        const int k = e / NJ, j = e - k * NJ;
        if (j < H) dW[k * H + j] = t;
        else db[k] = t;
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
int ctc_states_per_lane(int max_labels) {
    const int S = 2 * max_labels + 1;
    int nm = 1;
    while (64 * nm < S) nm *= 2;
    return nm;
}

hipError_t launch_head_fwd(const HeadArgs& a, hipStream_t s) {
    if (a.n_tiles == 0) return hipSuccess;
    hipLaunchKernelGGL(k_head_fwd, dim3(a.n_tiles), dim3(HT), head_fwd_lds(a.H, a.K), s, a.H, a.K, a.canvas_w, a.y,
                       a.rects, a.frame_off, a.tiles, a.w, a.b, a.logits, a.S);
    return hipGetLastError();
}

template <int NM>
static void launch_scan(const CtcArgs& a, hipStream_t s) {
    constexpr int D = NM <= 4 ? 8 : (NM <= 8 ? 4 : 2);  // frames of y loaded ahead
    hipLaunchKernelGGL((k_ctc_scan<NM, D>), dim3(a.n), dim3(128), 0, s, a.K, a.frame_off, a.lab_off, a.labels, a.y,
                       a.am, a.ae, a.bm, a.be, a.losses);
}

hipError_t launch_ctc(const CtcArgs& a, hipStream_t s) {
    if (a.n == 0 || a.frames == 0) return hipSuccess;
    const unsigned fb = (unsigned)((a.frames + 3) / 4);
    hipLaunchKernelGGL(k_ctc_softmax, dim3(fb), dim3(256), 0, s, a.frames, a.K, a.logits, a.y);
    switch (a.nm) {
        case 1: launch_scan<1>(a, s); break;
        case 2: launch_scan<2>(a, s); break;
        case 4: launch_scan<4>(a, s); break;
        case 8: launch_scan<8>(a, s); break;
        case 16: launch_scan<16>(a, s); break;
        case 32: launch_scan<32>(a, s); break;
        default: return hipErrorInvalidValue;
    }
    const int rs = 64 * a.nm;
    hipLaunchKernelGGL(k_ctc_grad, dim3(fb), dim3(256), (size_t)4 * (rs + 128) * 8, s, a.n, a.frames, a.K, rs,
                       a.frame_off, a.lab_off, a.labels, a.occ, a.y, a.am, a.ae, a.bm, a.be, a.dlogits);
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
        hipLaunchKernelGGL(k_head_dw_reduce, dim3((nj + 63) / 64), dim3(256), 0, s, a.H, a.K, chunks, a.part, a.dw,
                           a.db);
    } else {  // no frames: zero gradients
        hipLaunchKernelGGL(k_zero_f, dim3((a.K * a.H + 255) / 256), dim3(256), 0, s, a.dw, a.K * a.H);
        hipLaunchKernelGGL(k_zero_f, dim3((a.K + 255) / 256), dim3(256), 0, s, a.db, a.K);
    }
    return hipGetLastError();
}

}  // namespace mdl
