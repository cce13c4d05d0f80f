// Input-to-gate projection for all four directions and five gates at once
// (Section IV-B: the gate input activations depend only on the input, so one
// 1x1 convolution with five output groups computes them; here the four
// directions are folded into the same GEMM):
//     Z[p][n] = b_all[n] + sum_k Wx_all[n][k] X[p][k],  n = d*5H + gate*H + j.
// MFMA 16x16 tiles: M = gate columns (A = Wx rows), N = cells (B = X rows),
// K = input channels. Each wave owns 64 cells (four N tiles) and sweeps all
// gate-column tiles, so a lane stores four consecutive gate columns of one
// cell per tile.
#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

// Reduction-slot layouts. fp32: slot g holds k = g*KS + ks (one value per
// K step). bf16: K step ks covers k = 32*ks + 8*g + e, e = 0..7.
template <int KS>
__device__ __forceinline__ void load_slot_f32(const float* __restrict__ row, int g, int C, bool ok, float (&v)[KS]) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        int k = g * KS + ks;
        v[ks] = (ok && k < C) ? row[k] : 0.0f;
    }
}

template <int KS>
__device__ __forceinline__ void load_slot_bf16(const bf16_t* __restrict__ row, int g, int C, bool ok,
                                               bf16x8 (&v)[KS]) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        int k = 32 * ks + 8 * g;
        uint4 u = make_uint4(0, 0, 0, 0);
        if (ok && k < C) u = *reinterpret_cast<const uint4*>(row + k);
        v[ks] = as_bf16x8(u);
    }
}

constexpr int PROJ_CELLS_PER_WAVE = 64;

template <int KS>
__global__ void __launch_bounds__(256)
k_projection_f32(int64_t n_cells, int C, int N, const float* __restrict__ X, const float* __restrict__ Wx,
                 const float* __restrict__ bias, float* __restrict__ Z) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int g = lane >> 4, n16 = lane & 15;
    const int64_t cell0 = ((int64_t)blockIdx.x * 4 + wave) * PROJ_CELLS_PER_WAVE;
    if (cell0 >= n_cells) return;
    float b[4][KS];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        int64_t cell = cell0 + 16 * t + n16;
        load_slot_f32<KS>(X + cell * C, g, C, cell < n_cells, b[t]);
    }
    for (int mt = 0; mt < N / 16; ++mt) {
        float a[KS];
        load_slot_f32<KS>(Wx + (int64_t)(mt * 16 + n16) * C, g, C, true, a);
        floatx4 acc[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[t] = mfma_f32(a[ks], b[t][ks], acc[t]);
        const int col = mt * 16 + 4 * g;
        floatx4 bb = St<float>::ld4(bias + col);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            int64_t cell = cell0 + 16 * t + n16;
            if (cell < n_cells) St<float>::st4(Z + cell * N + col, acc[t] + bb);
        }
    }
}

template <int KS>
__global__ void __launch_bounds__(256)
k_projection_bf16(int64_t n_cells, int C, int N, const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wx,
                  const bf16_t* __restrict__ bias, bf16_t* __restrict__ Z) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int g = lane >> 4, n16 = lane & 15;
    const int64_t cell0 = ((int64_t)blockIdx.x * 4 + wave) * PROJ_CELLS_PER_WAVE;
    if (cell0 >= n_cells) return;
    bf16x8 b[4][KS];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        int64_t cell = cell0 + 16 * t + n16;
        load_slot_bf16<KS>(X + cell * C, g, C, cell < n_cells, b[t]);
    }
    for (int mt = 0; mt < N / 16; ++mt) {
        bf16x8 a[KS];
        load_slot_bf16<KS>(Wx + (int64_t)(mt * 16 + n16) * C, g, C, true, a);
        floatx4 acc[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[t] = mfma_bf16(a[ks], b[t][ks], acc[t]);
        const int col = mt * 16 + 4 * g;
        floatx4 bb = St<bf16_t>::ld4(bias + col);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            int64_t cell = cell0 + 16 * t + n16;
            if (cell < n_cells) St<bf16_t>::st4(Z + cell * N + col, acc[t] + bb);
        }
    }
}

hipError_t launch_projection(const LayerGeom& g, const void* d_x, const void* d_wx, const void* d_b, void* d_z,
                             hipStream_t s) {
    const int N = 20 * g.hidden;
    const int64_t waves = (g.n_cells + PROJ_CELLS_PER_WAVE - 1) / PROJ_CELLS_PER_WAVE;
    const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
    if (g.n_cells == 0) return hipSuccess;
    if (g.dtype == 0) {
        const int ks = (g.c_in + 3) / 4;
        auto X = static_cast<const float*>(d_x);
        auto W = static_cast<const float*>(d_wx);
        auto B = static_cast<const float*>(d_b);
        auto Z = static_cast<float*>(d_z);
        if (ks <= 1) hipLaunchKernelGGL(k_projection_f32<1>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else if (ks <= 2) hipLaunchKernelGGL(k_projection_f32<2>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else if (ks <= 4) hipLaunchKernelGGL(k_projection_f32<4>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else if (ks <= 8) hipLaunchKernelGGL(k_projection_f32<8>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else if (ks <= 16) hipLaunchKernelGGL(k_projection_f32<16>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else if (ks <= 32) hipLaunchKernelGGL(k_projection_f32<32>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else if (ks <= 64) hipLaunchKernelGGL(k_projection_f32<64>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else return hipErrorInvalidValue;
    } else {
        const int ks = (g.c_in + 31) / 32;
        auto X = static_cast<const bf16_t*>(d_x);
        auto W = static_cast<const bf16_t*>(d_wx);
        auto B = static_cast<const bf16_t*>(d_b);
        auto Z = static_cast<bf16_t*>(d_z);
        if (ks <= 1) hipLaunchKernelGGL(k_projection_bf16<1>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else if (ks <= 2) hipLaunchKernelGGL(k_projection_bf16<2>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else if (ks <= 4) hipLaunchKernelGGL(k_projection_bf16<4>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else if (ks <= 8) hipLaunchKernelGGL(k_projection_bf16<8>, grid, block, 0, s, g.n_cells, g.c_in, N, X, W, B, Z);
        else return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace mdl
