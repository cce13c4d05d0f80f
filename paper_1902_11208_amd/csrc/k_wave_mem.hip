// Wavefronts of the layer with memory-state matrices (Appendix A: three
// matrices per predecessor memory state S1 = c_L and S2 = c_T besides the five
// per hidden state; read as feeding the input gate and the two forget gates):
//     a = Z + U [h_L ; h_T] + [V [c_L ; c_T] ; 0]      (V: 3H x 2H, rows i, f_L, f_T)
// fp32 storage, H = 16 or 32, one workgroup of four waves per (rectangle,
// direction) unit, rectangles up to 64 rows.
//
// Forward, per local anti-diagonal: the contraction M [h_L; h_T; c_L; c_T]
// with M = [U | V'] (5H x 4H, V' = V over the first three gate blocks, zero
// below) runs on 16x16x4 fp32 MFMA for every 16-row tile the diagonal
// crosses, wave w owning gate-row tiles w, w + 4, w + 8 with its rows of M in
// registers and the previous diagonal's states as B operands from LDS; the
// cell update then reads the five pre-activations of its hidden unit from LDS.
// States are double-buffered by diagonal parity (row y of the previous
// diagonal is the left predecessor, row y - 1 the top one); rows not yet
// reached, the row above the first and masked cells hold zeros.
//
// Backward, per diagonal from the last: the cell phase forms dh and dc from
// dY and what the successors passed back (right successor: same row; lower
// successor: row below), writes the gate gradients da (into the workspace,
// as dZ, and to LDS) and the forget-gate part of the state gradients; then
// M^T da on MFMA gives what the cell passes to its predecessors (h_L, h_T,
// c_L, c_T blocks, the memory-state blocks added to dc f_L and dc f_T), and
// dV += da[i, f_L, f_T] x [c_L ; c_T] accumulates in registers over the
// unit's diagonals, written once per unit and summed per direction in unit
// order.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

namespace {

template <int H>
struct MemCfg {
    static constexpr int G = 5 * H;                 // gate rows
    static constexpr int NW = 4, THREADS = 256;
    static constexpr int RT = G / 16;               // gate-row tiles
    static constexpr int RTW = (RT + NW - 1) / NW;  // gate-row tiles per wave (forward)
    static constexpr int KS = H;                    // k-steps of the forward contraction (4H / 4)
    static constexpr int OT = 4 * H / 16;           // output tiles of M^T da
    static constexpr int OTW = (OT + NW - 1) / NW;
    static constexpr int KB = G / 4;                // k-steps of M^T da
    static constexpr int VT = (3 * H / 16) * (2 * H / 16);  // dV tiles
    static constexpr int VTW = (VT + NW - 1) / NW;
    static constexpr int MAXR = 64;
    static constexpr int SP = 2 * H + 4;            // forward state row [h | c] (+ padding)
    static constexpr int AP = G + 4;                // pre-activation / gate-gradient row
    static constexpr int PP = 4 * H + 4;            // backward pass row [dh_left | dc_left | dh_up | dc_up]
    static constexpr int CP = 2 * H + 4;            // backward [c_L | c_T] row
    static_assert(H == 16 || H == 32, "built for H = 16 and 32");
};

__device__ __forceinline__ float sigm(float z) { return 1.0f / (1.0f + __expf(-z)); }

// M[r][k]: U for k < 2H; V for 2H <= k < 4H and gate rows r < 3H; zero otherwise.
template <int H>
__device__ __forceinline__ float m_at(const float* U, const float* V, int d, int r, int k) {
    if (k < 2 * H) return U[((int64_t)d * 5 * H + r) * (2 * H) + k];
    if (r < 3 * H) return V[((int64_t)d * 3 * H + r) * (2 * H) + (k - 2 * H)];
    return 0.0f;
}

}  // namespace

template <int H>
__global__ void __launch_bounds__(256) k_wave_fwd_mem(MemArgs a) {
    using Cf = MemCfg<H>;
    constexpr int G = Cf::G, NW = Cf::NW, RT = Cf::RT, RTW = Cf::RTW, KS = Cf::KS, MAXR = Cf::MAXR;
    __shared__ __attribute__((aligned(16))) float st[2][MAXR + 1][Cf::SP];  // row y at index y + 1
    __shared__ __attribute__((aligned(16))) float sa[MAXR][Cf::AP];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 4, i16 = lane & 15;
    const int unit = a.units[blockIdx.x], d = unit & 3;
    const RectD R = {a.rects[4 * (unit >> 2)], a.rects[4 * (unit >> 2) + 1], a.rects[4 * (unit >> 2) + 2],
                     a.rects[4 * (unit >> 2) + 3]};
    for (int e = tid; e < 2 * (MAXR + 1) * Cf::SP; e += Cf::THREADS) (&st[0][0][0])[e] = 0.0f;
    float am[RTW][KS];
#pragma unroll
    for (int q = 0; q < RTW; ++q) {
        const int rt = wave + q * NW;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) am[q][ks] = rt < RT ? m_at<H>(a.u, a.v, d, rt * 16 + i16, 4 * ks + g) : 0.0f;
    }
    __syncthreads();
    const int h = R.h, w = R.w;
    float* const Z = a.z;
    for (int s = 0; s < h + w - 1; ++s) {
        const int ylo = max(0, s - w + 1), yhi = min(h - 1, s);
        const float(*sp)[Cf::SP] = st[(s + 1) & 1];
        float(*sc)[Cf::SP] = st[s & 1];
        for (int t = ylo >> 4; t <= (yhi >> 4); ++t) {
            floatx4 acc[RTW];
#pragma unroll
            for (int q = 0; q < RTW; ++q) acc[q] = floatx4{0.f, 0.f, 0.f, 0.f};
            const int y = 16 * t + i16;  // B column: the tile's cell on row y
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int k = 4 * ks + g;
                float bv;
                if (4 * ks < H) bv = sp[y + 1][k];                   // h_L: row y
                else if (4 * ks < 2 * H) bv = sp[y][k - H];          // h_T: row y - 1
                else if (4 * ks < 3 * H) bv = sp[y + 1][k - H];      // c_L: row y, c at column H
                else bv = sp[y][k - 2 * H];                          // c_T: row y - 1
#pragma unroll
                for (int q = 0; q < RTW; ++q) acc[q] = mfma_f32(am[q][ks], bv, acc[q]);
            }
#pragma unroll
            for (int q = 0; q < RTW; ++q) {
                const int rt = wave + q * NW;
                if (rt < RT) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) sa[y][rt * 16 + 4 * g + r] = acc[q][r];
                }
            }
        }
        __syncthreads();
        for (int e = tid; e < (yhi - ylo + 1) * H; e += Cf::THREADS) {
            const int y = ylo + e / H, j = e - (e / H) * H, x = s - y;
            const int64_t p = canvas_index(R, d, y, x, a.canvas_w);
            const bool valid = a.mask[p] != 0;
            float* zr = Z + p * (20 * H) + d * G;
            const float ai = sa[y][j] + zr[j], afl = sa[y][H + j] + zr[H + j], aft = sa[y][2 * H + j] + zr[2 * H + j];
            const float ao = sa[y][3 * H + j] + zr[3 * H + j], ag = sa[y][4 * H + j] + zr[4 * H + j];
            const float ig = sigm(ai), fl = sigm(afl), ft = sigm(aft), og = sigm(ao), gg = tanhf(ag);
            const float cl = sp[y + 1][H + j], ct = sp[y][H + j];
            const float c = valid ? ig * gg + fl * cl + ft * ct : 0.0f;
            const float hv = valid ? og * tanhf(c) : 0.0f;
            sc[y + 1][j] = hv;
            sc[y + 1][H + j] = c;
            a.y[p * (4 * H) + d * H + j] = hv;
            a.c[p * (4 * H) + d * H + j] = c;
            zr[j] = ig;
            zr[H + j] = fl;
            zr[2 * H + j] = ft;
            zr[3 * H + j] = og;
            zr[4 * H + j] = gg;
        }
        __syncthreads();
    }
}

template <int H>
__global__ void __launch_bounds__(256) k_wave_bwd_mem(MemArgs a) {
    using Cf = MemCfg<H>;
    constexpr int G = Cf::G, NW = Cf::NW, OT = Cf::OT, OTW = Cf::OTW, KB = Cf::KB, MAXR = Cf::MAXR;
    constexpr int VC = 2 * H / 16, VT = Cf::VT, VTW = Cf::VTW;
    __shared__ __attribute__((aligned(16))) float ps[2][MAXR + 1][Cf::PP];  // row y at index y
    __shared__ __attribute__((aligned(16))) float sda[MAXR][Cf::AP];
    __shared__ __attribute__((aligned(16))) float scm[MAXR][Cf::CP];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 4, i16 = lane & 15;
    const int unit = a.units[blockIdx.x], d = unit & 3;
    const RectD R = {a.rects[4 * (unit >> 2)], a.rects[4 * (unit >> 2) + 1], a.rects[4 * (unit >> 2) + 2],
                     a.rects[4 * (unit >> 2) + 3]};
    for (int e = tid; e < 2 * (MAXR + 1) * Cf::PP; e += Cf::THREADS) (&ps[0][0][0])[e] = 0.0f;
    for (int e = tid; e < MAXR * Cf::AP; e += Cf::THREADS) (&sda[0][0])[e] = 0.0f;
    for (int e = tid; e < MAXR * Cf::CP; e += Cf::THREADS) (&scm[0][0])[e] = 0.0f;
    // A operand of M^T da: output row o (of 4H) x gate row r
    float am[OTW][KB];
#pragma unroll
    for (int q = 0; q < OTW; ++q) {
        const int ot = wave + q * NW;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) am[q][kb] = ot < OT ? m_at<H>(a.u, a.v, d, 4 * kb + g, ot * 16 + i16) : 0.0f;
    }
    floatx4 accv[VTW];
#pragma unroll
    for (int q = 0; q < VTW; ++q) accv[q] = floatx4{0.f, 0.f, 0.f, 0.f};
    __syncthreads();
    const int h = R.h, w = R.w;
    float* const Z = a.z;
    for (int s = h + w - 2; s >= 0; --s) {
        const int ylo = max(0, s - w + 1), yhi = min(h - 1, s);
        const float(*pp)[Cf::PP] = ps[(s + 1) & 1];
        float(*pc)[Cf::PP] = ps[s & 1];
        // cell phase: rows ylo..yhi of this diagonal; every other row up to h
        // is cleared (what it passes on, its gate gradients and states)
        for (int e = tid; e < (h + 1) * H; e += Cf::THREADS) {
            const int y = e / H, j = e - (e / H) * H;
            if (y >= ylo && y <= yhi) {
                const int x = s - y;
                const int64_t p = canvas_index(R, d, y, x, a.canvas_w);
                const bool valid = a.mask[p] != 0;
                float* zr = Z + p * (20 * H) + d * G;
                const float ig = zr[j], fl = zr[H + j], ft = zr[2 * H + j], og = zr[3 * H + j], gg = zr[4 * H + j];
                const float c = a.c[p * (4 * H) + d * H + j];
                const float cl = x > 0 ? a.c[canvas_index(R, d, y, x - 1, a.canvas_w) * (4 * H) + d * H + j] : 0.0f;
                const float ct = y > 0 ? a.c[canvas_index(R, d, y - 1, x, a.canvas_w) * (4 * H) + d * H + j] : 0.0f;
                const float tc = tanhf(c);
                float dh = a.dy[p * (4 * H) + d * H + j] + pp[y][j] + pp[y + 1][2 * H + j];
                float dc = dh * og * (1.0f - tc * tc) + pp[y][H + j] + pp[y + 1][3 * H + j];
                if (!valid) dh = dc = 0.0f;
                const float di = dc * gg * ig * (1.0f - ig), dfl = dc * cl * fl * (1.0f - fl);
                const float dft = dc * ct * ft * (1.0f - ft), dog = dh * tc * og * (1.0f - og);
                const float dgg = dc * ig * (1.0f - gg * gg);
                sda[y][j] = di;
                sda[y][H + j] = dfl;
                sda[y][2 * H + j] = dft;
                sda[y][3 * H + j] = dog;
                sda[y][4 * H + j] = dgg;
                zr[j] = di;
                zr[H + j] = dfl;
                zr[2 * H + j] = dft;
                zr[3 * H + j] = dog;
                zr[4 * H + j] = dgg;
                scm[y][j] = cl;
                scm[y][H + j] = ct;
                pc[y][j] = 0.0f;
                pc[y][H + j] = dc * fl;
                pc[y][2 * H + j] = 0.0f;
                pc[y][3 * H + j] = dc * ft;
            } else {
                pc[y][j] = pc[y][H + j] = pc[y][2 * H + j] = pc[y][3 * H + j] = 0.0f;
                if (y < MAXR) {
#pragma unroll
                    for (int k = 0; k < 5; ++k) sda[y][k * H + j] = 0.0f;
                    scm[y][j] = scm[y][H + j] = 0.0f;
                }
            }
        }
        __syncthreads();
        for (int t = ylo >> 4; t <= (yhi >> 4); ++t) {
            const int y = 16 * t + i16;  // B column: cell on row y
            // M^T da: what the cells pass to their predecessors
#pragma unroll
            for (int q = 0; q < OTW; ++q) {
                const int ot = wave + q * NW;
                if (ot >= OT) continue;
                floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kb = 0; kb < KB; ++kb) acc = mfma_f32(am[q][kb], sda[y][4 * kb + g], acc);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int o = ot * 16 + 4 * g + r, blk = o / H, jj = o - blk * H;
                    // [h_L | h_T | c_L | c_T] -> [dh_left | dh_up | dc_left | dc_up] offsets 0, 2H, H, 3H
                    const int off = blk == 0 ? 0 : (blk == 1 ? 2 * H : (blk == 2 ? H : 3 * H));
                    pc[y][off + jj] += acc[r];
                }
            }
            // dV += da[i, f_L, f_T] x [c_L ; c_T], K = the tile's 16 cells
#pragma unroll
            for (int q = 0; q < VTW; ++q) {
                const int vt = wave + q * NW;
                if (vt >= VT) continue;
                const int vr = vt / VC, vc = vt - vr * VC;
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const int cell = 16 * t + 4 * ks + g;
                    accv[q] = mfma_f32(sda[cell][vr * 16 + i16], scm[cell][vc * 16 + i16], accv[q]);
                }
            }
        }
        __syncthreads();
    }
    float* out = a.dvpart + (int64_t)blockIdx.x * (3 * H) * (2 * H);
#pragma unroll
    for (int q = 0; q < VTW; ++q) {
        const int vt = wave + q * NW;
        if (vt >= VT) continue;
        const int vr = vt / VC, vc = vt - vr * VC;
#pragma unroll
        for (int r = 0; r < 4; ++r) out[(vr * 16 + 4 * g + r) * (2 * H) + vc * 16 + i16] = accv[q][r];
    }
}

// dV[d] = sum over the units of direction d, in launch order, of their partials.
__global__ void k_dv_reduce(int n_units, int per_unit, const int32_t* __restrict__ units,
                            const float* __restrict__ part, float* __restrict__ dv) {
    for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < 4 * per_unit; e += gridDim.x * blockDim.x) {
        const int d = e / per_unit, k = e - d * per_unit;
        float s = 0.0f;
        for (int b = 0; b < n_units; ++b)
            if ((units[b] & 3) == d) s += part[(int64_t)b * per_unit + k];
        dv[e] = s;
    }
}

bool mem_supported(const LayerGeom& g) { return g.dtype == 0 && (g.hidden == 16 || g.hidden == 32); }

size_t mem_partial_bytes(const LayerGeom& g, int n_units) {
    return (size_t)std::max(n_units, 1) * 3 * g.hidden * 2 * g.hidden * sizeof(float);
}

hipError_t launch_wavefront_mem(bool fwd, const LayerGeom& g, int n_units, const MemArgs& a, hipStream_t s) {
    if (n_units == 0) return hipSuccess;
    if (g.hidden == 16) {
        if (fwd) hipLaunchKernelGGL(k_wave_fwd_mem<16>, dim3(n_units), dim3(256), 0, s, a);
        else hipLaunchKernelGGL(k_wave_bwd_mem<16>, dim3(n_units), dim3(256), 0, s, a);
    } else if (g.hidden == 32) {
        if (fwd) hipLaunchKernelGGL(k_wave_fwd_mem<32>, dim3(n_units), dim3(256), 0, s, a);
        else hipLaunchKernelGGL(k_wave_bwd_mem<32>, dim3(n_units), dim3(256), 0, s, a);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_dv_reduce(const LayerGeom& g, int n_units, const int32_t* d_units, const float* d_part, float* d_dv,
                            hipStream_t s) {
    const int per = 3 * g.hidden * 2 * g.hidden;
    hipLaunchKernelGGL(k_dv_reduce, dim3((4 * per + 255) / 256), dim3(256), 0, s, n_units, per, d_units, d_part, d_dv);
    return hipGetLastError();
}

}  // namespace mdl
