// Input and weight gradients from dZ in one pass over the canvas, staged
// through LDS strip by strip.
//
// A strip is TC consecutive cells of one canvas row. For each strip the
// workgroup loads, with independent coalesced loads, dZ [TC][20H], X
// [TC][C_in], the layer output Y of the strip's row (one cell of halo on each
// side) and of the rows above and below, and per cell a validity byte (cell
// valid; left/right/up/down neighbour in the same rectangle and unmasked).
// Then, from LDS:
//   dW_d[r][col] += sum_cells dZ[cell][d*5H + r] * B_d[cell][col],
//     B_d = [X | h_L,d | h_T,d | 1]  (the layer output shifted one cell in
//     direction d's frame: the shifted recurrent operand of Appendix A)
//   dX[cell] = sum_d dZ_d[cell] Wx_d
// Wave w of the workgroup owns direction d = w / WPD and a slice of the gate
// rows; the dW tiles stay in its registers across all strips of the
// workgroup, and are written once as the workgroup's partial. A fixed-order
// reduction over workgroups gives deterministic weight gradients.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

namespace {

constexpr int STRIP_WGS = 512;  // workgroups (two per CU)

template <int H, int C>
struct StripCfg {
    static constexpr int G = 5 * H, N = 20 * H;
    static constexpr int RT = (G + 15) / 16;          // gate-row tiles per direction
    static constexpr int CT = (C + 2 * H + 1 + 15) / 16;  // dW column tiles
    static constexpr int CXT = (C + 15) / 16;         // dX channel tiles
    static constexpr int WPD = H >= 32 ? 2 : 1;       // waves per direction
    static constexpr int RTW = (RT + WPD - 1) / WPD;  // gate-row tiles per wave
    static constexpr int TC = H >= 32 ? 16 : 32;      // cells per strip
    static constexpr int THREADS = 256 * WPD;
    static constexpr int ZP = N + 16;                 // LDS pitch of dZ rows: 4 cell slots hit distinct banks
    static constexpr int YP = 4 * H + 4;              // LDS pitch of Y rows
    static constexpr int XP = CXT * 16 + 4;           // LDS pitch of X rows and dX partials
    static constexpr int SY = 3 * (TC + 2) * YP, SDX = 4 * TC * XP;
};

// 4 consecutive elements of storage type T as fp32.
template <typename T>
struct V4;
template <>
struct V4<float> {
    using R = float4;
    static __device__ __forceinline__ R load(const float* p) { return *reinterpret_cast<const float4*>(p); }
    static __device__ __forceinline__ float4 f(R v) { return v; }
    static __device__ __forceinline__ R zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
};
template <>
struct V4<bf16_t> {
    using R = uint2;
    static __device__ __forceinline__ R load(const bf16_t* p) { return *reinterpret_cast<const uint2*>(p); }
    static __device__ __forceinline__ float4 f(R v) {
        return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u), __uint_as_float(v.y << 16),
                           __uint_as_float(v.y & 0xffff0000u));
    }
    static __device__ __forceinline__ R zero() { return make_uint2(0, 0); }
};

template <typename T>
__device__ __forceinline__ float to_f(T v);
template <>
__device__ __forceinline__ float to_f<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f<bf16_t>(bf16_t v) { return bf2f(v); }

__device__ __forceinline__ void st_f4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }

}  // namespace

template <typename T, int H, int C>
__global__ void __launch_bounds__((StripCfg<H, C>::THREADS))
k_bwd_strip(int canvas_h, int canvas_w, int n_strips, int segs, const T* __restrict__ dZ, const T* __restrict__ X,
            const T* __restrict__ Y, const T* __restrict__ Wx, const uint8_t* __restrict__ mask,
            const int32_t* __restrict__ rid, T* __restrict__ dX, float* __restrict__ part) {
    using Cf = StripCfg<H, C>;
    using L4 = V4<T>;
    constexpr int TC = Cf::TC, RTW = Cf::RTW, WPD = Cf::WPD, CT = Cf::CT, CXT = Cf::CXT;
    constexpr int N = Cf::N, G = Cf::G, ZP = Cf::ZP, YP = Cf::YP, XP = Cf::XP, NTH = Cf::THREADS;
    __shared__ __attribute__((aligned(16))) float sz[TC][ZP];
    __shared__ __attribute__((aligned(16))) float sx[TC][XP];
    // Y rows above, same (with one cell of halo each side), below; later the
    // per-direction dX partials
    __shared__ __attribute__((aligned(16))) float sy_raw[Cf::SY > Cf::SDX ? Cf::SY : Cf::SDX];
    __shared__ uint8_t sflag[TC];
    auto sy = reinterpret_cast<float(*)[TC + 2][YP]>(sy_raw);
    auto sdx = reinterpret_cast<float(*)[TC][XP]>(sy_raw);

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int d = wave / WPD, rslice = wave % WPD;
    const int rt0 = rslice * RTW;

    floatx4 acc[RTW][CT];
#pragma unroll
    for (int a = 0; a < RTW; ++a)
#pragma unroll
        for (int b = 0; b < CT; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    // dX: wave (d, rslice) owns channel tiles ct = rslice, rslice + WPD, ...;
    // its A operand Wx_d^T (row = channel, K = gate rows 4 ks + g) stays in registers.
    constexpr int CXW = (CXT + WPD - 1) / WPD;
    float wa[CXW][G / 4];
#pragma unroll
    for (int cc = 0; cc < CXW; ++cc) {
        const int ch = (rslice + cc * WPD) * 16 + i16;
#pragma unroll
        for (int ks = 0; ks < G / 4; ++ks)
            wa[cc][ks] = ch < C ? to_f<T>(Wx[((int64_t)d * G + 4 * ks + g) * C + ch]) : 0.0f;
    }

    for (int strip = blockIdx.x; strip < n_strips; strip += gridDim.x) {
        const int cy = strip / segs;
        const int cx0 = (strip - cy * segs) * TC;
        const int len = min(TC, canvas_w - cx0);
        const int64_t p0 = (int64_t)cy * canvas_w + cx0;

        // --- stage (all loads independent; issued in batches before the LDS stores)
        {
            constexpr int NZ = TC * N / 4, PZ = (NZ + NTH - 1) / NTH;
            typename L4::R v[PZ];
#pragma unroll
            for (int k = 0; k < PZ; ++k) {
                const int e = tid + k * NTH;
                const int c = (4 * e) / N;
                v[k] = (e < NZ && c < len) ? L4::load(dZ + p0 * N + 4 * e) : L4::zero();
            }
#pragma unroll
            for (int k = 0; k < PZ; ++k) {
                const int e = tid + k * NTH;
                if (e < NZ) {
                    const int c = (4 * e) / N, n = 4 * e - c * N;
                    st_f4(&sz[c][n], L4::f(v[k]));
                }
            }
        }
        {
            constexpr int NYR = (TC + 2) * H, NY = 3 * NYR, PY = (NY + NTH - 1) / NTH;  // float4 units
            typename L4::R v[PY];
#pragma unroll
            for (int k = 0; k < PY; ++k) {
                const int e = tid + k * NTH;
                const int row = e / NYR, rem = e - row * NYR;
                const int c = rem / H, k4 = rem - c * H;
                const int yy = cy + row - 1, xx = cx0 + c - 1;
                v[k] = (e < NY && yy >= 0 && yy < canvas_h && xx >= 0 && xx < canvas_w && c <= len + 1)
                           ? L4::load(Y + ((int64_t)yy * canvas_w + xx) * (4 * H) + 4 * k4)
                           : L4::zero();
            }
#pragma unroll
            for (int k = 0; k < PY; ++k) {
                const int e = tid + k * NTH;
                if (e < NY) {
                    const int row = e / NYR, rem = e - row * NYR;
                    const int c = rem / H, k4 = rem - c * H;
                    st_f4(&sy[row][c][4 * k4], L4::f(v[k]));
                }
            }
        }
        for (int e = tid; e < TC * CXT * 4; e += NTH) {
            const int c = e / (CXT * 4), k4 = e - c * (CXT * 4);
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (c < len && 4 * k4 < C) v = L4::f(L4::load(X + (p0 + c) * C + 4 * k4));
            st_f4(&sx[c][4 * k4], v);
        }
        // validity byte per cell: bit0 valid, bit1 left, bit2 right, bit3 up, bit4 down.
        // All ten loads are issued at once (neighbours outside the canvas
        // re-read the cell itself and are discarded).
        for (int c = tid; c < TC; c += NTH) {
            const int cc = min(c, len - 1), cx = cx0 + cc;
            const int64_t p = p0 + cc;
            const bool hl = cx > 0, hr = cx + 1 < canvas_w, hu = cy > 0, hd = cy + 1 < canvas_h;
            const int64_t pl = hl ? p - 1 : p, pr = hr ? p + 1 : p;
            const int64_t pu = hu ? p - canvas_w : p, pd = hd ? p + canvas_w : p;
            const int r = rid[p], rl = rid[pl], rr = rid[pr], ru = rid[pu], rd = rid[pd];
            const uint8_t m = mask[p], ml = mask[pl], mr = mask[pr], mu = mask[pu], md = mask[pd];
            uint8_t f = 0;
            if (c < len && m && r >= 0) {
                f = 1;
                if (hl && rl == r && ml) f |= 2;
                if (hr && rr == r && mr) f |= 4;
                if (hu && ru == r && mu) f |= 8;
                if (hd && rd == r && md) f |= 16;
            }
            sflag[c] = f;
        }
        __syncthreads();

        // --- dW: K = cells of the strip, 4 per MFMA step (slot g = cell offset)
#pragma unroll 2
        for (int ks = 0; ks < TC / 4; ++ks) {
            const int c = 4 * ks + g;
            const uint8_t f = sflag[c];
            const bool v = f & 1;
            const bool vl = (d & 1) ? (f & 4) : (f & 2);
            const bool vt = (d & 2) ? (f & 16) : (f & 8);
            const int lc = (d & 1) ? c + 2 : c;  // left predecessor in the halo-shifted same row
            const int trow = (d & 2) ? 2 : 0;    // row of the top predecessor
            float av[RTW], bv[CT];
#pragma unroll
            for (int a = 0; a < RTW; ++a) {
                const int r = (rt0 + a) * 16 + i16;
                av[a] = (v && r < G) ? sz[c][d * G + r] : 0.0f;
            }
#pragma unroll
            for (int b = 0; b < CT; ++b) {
                const int col = b * 16 + i16;
                float x = 0.0f;
                if (col < C) x = sx[c][col];
                else if (col < C + H) x = vl ? sy[1][lc][d * H + col - C] : 0.0f;
                else if (col < C + 2 * H) x = vt ? sy[trow][c + 1][d * H + col - C - H] : 0.0f;
                else if (col == C + 2 * H) x = 1.0f;
                bv[b] = v ? x : 0.0f;
            }
#pragma unroll
            for (int a = 0; a < RTW; ++a)
#pragma unroll
                for (int b = 0; b < CT; ++b) acc[a][b] = mfma_f32(av[a], bv[b], acc[a][b]);
        }

        // --- dX partial of direction d: M = channels, N = cells, K = 5H gate rows
        floatx4 axs[CXW][TC / 16];
#pragma unroll
        for (int cc = 0; cc < CXW; ++cc) {
#pragma unroll
            for (int nt = 0; nt < TC / 16; ++nt) {
                floatx4 ax = floatx4{0.f, 0.f, 0.f, 0.f};
                const int cell = nt * 16 + i16;
                const bool v = sflag[cell] & 1;
                if ((rslice + cc * WPD) < CXT) {
                    // B operands in groups of ten: one LDS round trip per group
                    constexpr int KB = 10, NKS = G / 4;
#pragma unroll
                    for (int k0 = 0; k0 < NKS; k0 += KB) {
                        float bz[KB];
#pragma unroll
                        for (int kk = 0; kk < KB; ++kk)
                            bz[kk] = (v && k0 + kk < NKS) ? sz[cell][d * G + 4 * (k0 + kk) + g] : 0.0f;
#pragma unroll
                        for (int kk = 0; kk < KB; ++kk)
                            if (k0 + kk < NKS) ax = mfma_f32(wa[cc][k0 + kk], bz[kk], ax);
                    }
                }
                axs[cc][nt] = ax;
            }
        }
        __syncthreads();  // every wave is done reading the staged Y rows
#pragma unroll
        for (int cc = 0; cc < CXW; ++cc) {
            const int ct = rslice + cc * WPD;
            if (ct < CXT) {
#pragma unroll
                for (int nt = 0; nt < TC / 16; ++nt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) sdx[d][nt * 16 + i16][ct * 16 + 4 * g + r] = axs[cc][nt][r];
            }
        }
        __syncthreads();
        // sum the four directions in a fixed order; dX is 0 at invalid cells
        for (int e = tid; e < TC * C; e += NTH) {
            const int c = e / C, k = e - c * C;
            if (c < len) {
                const float s4 = ((sdx[0][c][k] + sdx[1][c][k]) + sdx[2][c][k]) + sdx[3][c][k];
                St<T>::st1(dX + (p0 + c) * C + k, (sflag[c] & 1) ? s4 : 0.0f);
            }
        }
        __syncthreads();
    }

    // partial of this workgroup: [wg][4][RT*16][CT*16]
    float* out = part + (int64_t)blockIdx.x * 4 * (Cf::RT * 16) * (CT * 16) + (int64_t)d * (Cf::RT * 16) * (CT * 16);
#pragma unroll
    for (int a = 0; a < RTW; ++a) {
        if (rt0 + a >= Cf::RT) continue;
#pragma unroll
        for (int b = 0; b < CT; ++b)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                out[(int64_t)((rt0 + a) * 16 + 4 * g + r) * (CT * 16) + b * 16 + i16] = acc[a][b][r];
    }
}

// Fixed-order sum over workgroup partials; one thread per output element,
// loads batched so the sum is bandwidth- rather than latency-bound.
__global__ void k_strip_reduce(int C, int H, int RT, int CT, int nwg, const float* __restrict__ part,
                               float* __restrict__ dwx, float* __restrict__ du, float* __restrict__ db) {
    const int G = 5 * H, NB = C + 2 * H + 1;
    const int64_t total = (int64_t)4 * G * NB;
    const int64_t stride = (int64_t)4 * (RT * 16) * (CT * 16);
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int d = (int)(idx / ((int64_t)G * NB));
        const int rem = (int)(idx - (int64_t)d * G * NB);
        const int r = rem / NB, col = rem - r * NB;
        const float* src = part + (int64_t)d * (RT * 16) * (CT * 16) + (int64_t)r * (CT * 16) + col;
        float s = 0.0f;
        int w = 0;
        for (; w + 8 <= nwg; w += 8) {
            float v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = src[(int64_t)(w + k) * stride];
#pragma unroll
            for (int k = 0; k < 8; ++k) s += v[k];
        }
        for (; w < nwg; ++w) s += src[(int64_t)w * stride];
        if (col < C) dwx[((int64_t)d * G + r) * C + col] = s;
        else if (col < C + 2 * H) du[((int64_t)d * G + r) * (2 * H) + (col - C)] = s;
        else db[(int64_t)d * G + r] = s;
    }
}

// Instantiated (storage, H, c_in) shapes; other shapes use the two-kernel path.
#define MDL_STRIP_SHAPES(X) \
    X(float, 4, 4) X(float, 4, 8) X(float, 8, 8) X(float, 16, 8) X(float, 16, 16) X(float, 32, 16) \
    X(float, 32, 32) X(bf16_t, 32, 16) X(bf16_t, 32, 32)

static int strip_tc(int hidden) { return hidden >= 32 ? 16 : 32; }

bool strip_supported(const LayerGeom& g) {
#define MDL_STRIP_MATCH(T, H, C) \
    if ((g.dtype == 1) == std::is_same<T, bf16_t>::value && g.hidden == H && g.c_in == C) return true;
    MDL_STRIP_SHAPES(MDL_STRIP_MATCH)
#undef MDL_STRIP_MATCH
    return false;
}

static int strip_wgs(const LayerGeom& g) {
    const int tc = strip_tc(g.hidden);
    const int64_t strips = (int64_t)g.canvas_h * ((g.canvas_w + tc - 1) / tc);
    return (int)std::max<int64_t>(1, std::min<int64_t>(STRIP_WGS, strips));
}

size_t strip_partial_bytes(const LayerGeom& g) {
    const int RT = (5 * g.hidden + 15) / 16, CT = (g.c_in + 2 * g.hidden + 1 + 15) / 16;
    return (size_t)strip_wgs(g) * 4 * RT * 16 * CT * 16 * sizeof(float);
}

hipError_t launch_bwd_strip(const LayerGeom& g, const void* d_dz, const void* d_x, const void* d_y, const void* d_wx,
                            const uint8_t* d_mask, const int32_t* d_rid, void* d_dx, float* d_part, float* d_dwx,
                            float* d_du, float* d_db, hipStream_t s) {
    const int tc = strip_tc(g.hidden);
    const int segs = (g.canvas_w + tc - 1) / tc;
    const int n_strips = g.canvas_h * segs;
    const int nwg = strip_wgs(g);
    const int RT = (5 * g.hidden + 15) / 16, CT = (g.c_in + 2 * g.hidden + 1 + 15) / 16;
    bool ok = false;
#define MDL_STRIP_LAUNCH(T, H, C)                                                                                  \
    if (!ok && (g.dtype == 1) == std::is_same<T, bf16_t>::value && g.hidden == H && g.c_in == C) {                 \
        hipLaunchKernelGGL((k_bwd_strip<T, H, C>), dim3(nwg), dim3(StripCfg<H, C>::THREADS), 0, s, g.canvas_h,     \
                           g.canvas_w, n_strips, segs, static_cast<const T*>(d_dz), static_cast<const T*>(d_x),    \
                           static_cast<const T*>(d_y), static_cast<const T*>(d_wx), d_mask, d_rid,                 \
                           static_cast<T*>(d_dx), d_part);                                                         \
        ok = true;                                                                                                 \
    }
    MDL_STRIP_SHAPES(MDL_STRIP_LAUNCH)
#undef MDL_STRIP_LAUNCH
    if (!ok) return hipErrorInvalidValue;
    const int64_t total = (int64_t)4 * 5 * g.hidden * (g.c_in + 2 * g.hidden + 1);
    int blocks = (int)((total + 255) / 256);
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_strip_reduce, dim3(blocks), dim3(256), 0, s, g.c_in, g.hidden, RT, CT, nwg, d_part, d_dwx,
                       d_du, d_db);
    return hipGetLastError();
}

}  // namespace mdl
