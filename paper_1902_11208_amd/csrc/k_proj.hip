// Input-to-gate projection for all four directions and five gates at once
// (Section IV-B: the gate input activations depend only on the input, so one
// 1x1 convolution with five output groups computes them; here the four
// directions are folded into the same GEMM):
//     Z[p][n] = b_all[n] + sum_k Wx_all[n][k] X[p][k],  n = d*5H + gate*H + j.
// MFMA 16x16 tiles: M = gate columns (A = Wx rows), N = cells (B = X rows),
// K = input channels. A workgroup stages a chunk of Wx rows (gate columns) in
// LDS once and then loops over blocks of 256 cells (its four waves take 64
// cells each, B operands in registers, the next block's loaded while the
// current one is stored). The stores are write-bandwidth bound: every 16-cell x 64-column
// output block passes through a small per-wave LDS tile so that one store
// instruction writes four cells x 64 contiguous columns instead of sixteen
// cells x 4 columns.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

namespace {

constexpr int PCELLS = 64;             // cells per wave
constexpr int PW_LDS = 48 * 1024;      // LDS bytes for the Wx chunk

template <typename T>
struct PK;
template <>
struct PK<float> {  // 16x16x4 f32: K step ks, slot g holds k = g*KS + ks
    using Op = float;
    static constexpr int PERK = 4;  // k values per K step
    static constexpr int PAD = 4;   // LDS row padding (elements)
    static __device__ __forceinline__ int koff(int g, int ks, int KS) { return g * KS + ks; }
    static __device__ __forceinline__ Op lds(const float* p) { return *p; }
    static __device__ __forceinline__ Op gload(const float* row, int k, int C) { return k < C ? row[k] : 0.0f; }
    static __device__ __forceinline__ floatx4 mma(Op a, Op b, floatx4 c) { return mfma_f32(a, b, c); }
    // non-temporal: Z is far larger than the caches and is next read by the
    // wavefront; streaming it past them measured faster for the whole step
    static __device__ __forceinline__ void st4(float* p, floatx4 v) {
        __builtin_nontemporal_store(v, reinterpret_cast<floatx4*>(p));
    }
};
template <>
struct PK<bf16_t> {  // 16x16x32 bf16: K step ks, slot g holds k = 32 ks + 8 g + e
    using Op = bf16x8;
    static constexpr int PERK = 32;
    static constexpr int PAD = 8;
    static __device__ __forceinline__ int koff(int g, int ks, int) { return 32 * ks + 8 * g; }
    static __device__ __forceinline__ Op lds(const bf16_t* p) { return as_bf16x8(*reinterpret_cast<const uint4*>(p)); }
    static __device__ __forceinline__ Op gload(const bf16_t* row, int k, int C) {
        return as_bf16x8(k < C ? *reinterpret_cast<const uint4*>(row + k) : make_uint4(0, 0, 0, 0));
    }
    static __device__ __forceinline__ floatx4 mma(Op a, Op b, floatx4 c) { return mfma_bf16(a, b, c); }
    // non-temporal, as for fp32: four bf16 values as one 8-byte store
    static __device__ __forceinline__ void st4(bf16_t* p, floatx4 v) {
        const uint64_t lo = f2bf2(v[0], v[1]);
        const uint64_t hi = f2bf2(v[2], v[3]);
        __builtin_nontemporal_store(lo | (hi << 32), reinterpret_cast<uint64_t*>(p));
    }
};

}  // namespace

template <typename T, int KS>
__global__ void __launch_bounds__(256)
k_projection(int64_t n_cells, int64_t n_blocks, int C, int N, int nch, const T* __restrict__ X,
             const T* __restrict__ Wx, const T* __restrict__ bias, const int32_t* __restrict__ rid,
             T* __restrict__ Z) {
    using K = PK<T>;
    using Op = typename K::Op;
    constexpr int RW = K::PERK * KS;  // staged k values per row
    constexpr int P = RW + K::PAD;    // LDS row pitch (elements); the pad spreads rows over banks
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    T* sW = reinterpret_cast<T*>(smem);
    __shared__ __attribute__((aligned(16))) float sO[4][16][64 + 4];

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int g = lane >> 4, n16 = lane & 15;
    const int n0 = blockIdx.y * nch, nc = min(nch, N - n0);
    for (int i = threadIdx.x; i < nc * RW; i += 256) {
        const int r = i / RW, k = i - r * RW;
        sW[r * P + k] = k < C ? Wx[(int64_t)(n0 + r) * C + k] : T(0);
    }
    __syncthreads();
    float(*so)[64 + 4] = sO[wave];
    const int ntiles = nc / 16;
    // B operands of a block's 64 cells of this wave (rows past the canvas
    // re-read its last cell; their results are not stored)
    Op b[4][KS];
    // rectangle id of the lane's cell of the block: a wave whose 64 cells all
    // lie outside the rectangles (row slack, separators) skips the block; no
    // later step reads their pre-activations
    int32_t rv = 0;
    auto load_b = [&](int64_t blk) {
        const int64_t cell0 = (blk * 4 + wave) * PCELLS;
        rv = rid ? rid[min(cell0 + lane, n_cells - 1)] : 0;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const T* row = X + min(cell0 + 16 * t + n16, n_cells - 1) * C;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) b[t][ks] = K::gload(row, K::koff(g, ks, KS), C);
        }
    };
    load_b(blockIdx.x);
    for (int64_t blk = blockIdx.x; blk < n_blocks; blk += gridDim.x) {
        const int64_t cell0 = (blk * 4 + wave) * PCELLS;
        if (__ballot(rv >= 0 && cell0 + lane < n_cells) == 0) {
            load_b(min(blk + (int64_t)gridDim.x, n_blocks - 1));
            continue;
        }
        for (int mg = 0; mg * 4 < ntiles; ++mg) {
            const int mc = min(4, ntiles - 4 * mg);  // column tiles in this group
            floatx4 acc[4][4];
    #pragma unroll
            for (int m = 0; m < 4; ++m) {
    #pragma unroll
                for (int t = 0; t < 4; ++t) acc[m][t] = floatx4{0.f, 0.f, 0.f, 0.f};
                if (m < mc) {
                    Op a[KS];
                    const T* ar = sW + ((mg * 4 + m) * 16 + n16) * P;
    #pragma unroll
                    for (int ks = 0; ks < KS; ++ks) a[ks] = K::lds(ar + K::koff(g, ks, KS));
    #pragma unroll
                    for (int ks = 0; ks < KS; ++ks)
    #pragma unroll
                        for (int t = 0; t < 4; ++t) acc[m][t] = K::mma(a[ks], b[t][ks], acc[m][t]);
                }
            }
            // lane (r, c) of the store pass writes cell 4 r' + lane/16 of the tile,
            // columns 4 (lane % 16) .. + 3 of the group
            // the last column group's MFMAs are issued: load the next block's operands
            if (mg * 4 + 4 >= ntiles) load_b(min(blk + (int64_t)gridDim.x, n_blocks - 1));
            const int c4 = 4 * (lane & 15);
            const int colb = n0 + mg * 64;
            const bool colok = c4 < 16 * mc;
            const floatx4 bb = colok ? St<T>::ld4(bias + colb + c4) : floatx4{0.f, 0.f, 0.f, 0.f};
    #pragma unroll
            for (int t = 0; t < 4; ++t) {
    #pragma unroll
                for (int m = 0; m < 4; ++m) *reinterpret_cast<floatx4*>(&so[n16][m * 16 + 4 * g]) = acc[m][t];
                __builtin_amdgcn_wave_barrier();
    #pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int cl = 4 * r + (lane >> 4);
                    const floatx4 v = *reinterpret_cast<const floatx4*>(&so[cl][c4]) + bb;
                    const int64_t cell = cell0 + 16 * t + cl;
                    if (colok && cell < n_cells) K::st4(Z + cell * N + colb + c4, v);
                }
                __builtin_amdgcn_wave_barrier();
            }
        }
    }
}

template <typename T, int KS>
static hipError_t launch_proj(const LayerGeom& g, const T* X, const T* W, const T* B, const int32_t* rid, T* Z,
                              hipStream_t s) {
    constexpr int RW = PK<T>::PERK * KS, P = RW + PK<T>::PAD;
    const int N = 20 * g.hidden;
    // columns per workgroup: as many as the LDS budget holds (a multiple of 16,
    // of 64 when possible), split evenly over the chunks
    const int cap = PW_LDS / (P * (int)sizeof(T)) / 16 * 16;
    const int unit = cap >= 64 ? 64 : 16;
    const int nchunks = (N + cap / unit * unit - 1) / (cap / unit * unit);
    int nch = ((N + nchunks - 1) / nchunks + unit - 1) / unit * unit;
    nch = std::min(std::min(nch, cap / unit * unit), N);
    const int64_t waves = (g.n_cells + PCELLS - 1) / PCELLS;
    const int64_t blocks = (waves + 3) / 4;
    const int nchunks_col = (N + nch - 1) / nch;
    // workgroups that loop over the cell blocks: as many as fit on the CUs at
    // once (LDS-limited, at most four per CU)
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
        cus = 256;
        (void)hipGetLastError();  // not reported for the launch below
    }
    const size_t lds = (size_t)nch * P * sizeof(T) + 4 * 16 * (64 + 4) * sizeof(float);
    const int per_cu = (int)std::max<size_t>(1, std::min<size_t>(4, 160 * 1024 / lds));
    const int64_t want = std::max<int64_t>(1, (int64_t)per_cu * std::max(cus, 1) / nchunks_col);
    const dim3 grid((unsigned)std::min<int64_t>(blocks, want), (unsigned)nchunks_col), block(256);
    hipLaunchKernelGGL((k_projection<T, KS>), grid, block, (size_t)nch * P * sizeof(T), s, g.n_cells, blocks, g.c_in,
                       N, nch, X, W, B, rid, Z);
    return hipGetLastError();
}

hipError_t launch_projection(const LayerGeom& g, const void* d_x, const void* d_wx, const void* d_b,
                             const int32_t* d_rid, void* d_z, hipStream_t s) {
    if (g.n_cells == 0) return hipSuccess;
    if (g.dtype == 0) {
        const int ks = (g.c_in + 3) / 4;
        auto X = static_cast<const float*>(d_x);
        auto W = static_cast<const float*>(d_wx);
        auto B = static_cast<const float*>(d_b);
        auto Z = static_cast<float*>(d_z);
        if (ks <= 1) return launch_proj<float, 1>(g, X, W, B, d_rid, Z, s);
        if (ks <= 2) return launch_proj<float, 2>(g, X, W, B, d_rid, Z, s);
        if (ks <= 4) return launch_proj<float, 4>(g, X, W, B, d_rid, Z, s);
        if (ks <= 8) return launch_proj<float, 8>(g, X, W, B, d_rid, Z, s);
        if (ks <= 16) return launch_proj<float, 16>(g, X, W, B, d_rid, Z, s);
        if (ks <= 32) return launch_proj<float, 32>(g, X, W, B, d_rid, Z, s);
        if (ks <= 64) return launch_proj<float, 64>(g, X, W, B, d_rid, Z, s);
        return hipErrorInvalidValue;
    }
    const int ks = (g.c_in + 31) / 32;
    auto X = static_cast<const bf16_t*>(d_x);
    auto W = static_cast<const bf16_t*>(d_wx);
    auto B = static_cast<const bf16_t*>(d_b);
    auto Z = static_cast<bf16_t*>(d_z);
    if (ks <= 1) return launch_proj<bf16_t, 1>(g, X, W, B, d_rid, Z, s);
    if (ks <= 2) return launch_proj<bf16_t, 2>(g, X, W, B, d_rid, Z, s);
    if (ks <= 4) return launch_proj<bf16_t, 4>(g, X, W, B, d_rid, Z, s);
    if (ks <= 8) return launch_proj<bf16_t, 8>(g, X, W, B, d_rid, Z, s);
    return hipErrorInvalidValue;
}

// Fill of n 32-bit words with one pattern (the poisoned-workspace debug mode).
__global__ void k_fill_u32(uint32_t* __restrict__ d, int64_t n, uint32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        d[i] = v;
}

hipError_t launch_fill_u32(void* d, int64_t n_words, uint32_t v, hipStream_t s) {
    if (n_words <= 0) return hipSuccess;
    const int blocks = (int)std::min<int64_t>((n_words + 255) / 256, 4096);
    hipLaunchKernelGGL(k_fill_u32, dim3(blocks), dim3(256), 0, s, static_cast<uint32_t*>(d), n_words, v);
    return hipGetLastError();
}

// Number of NaN and infinite values among the rows of the cells whose mask
// byte is set (row values per cell each), added to *count: a wave reduction
// and one atomic per wave.
template <typename T>
__global__ void k_count_nonfinite(const T* __restrict__ p, int64_t n_cells, int row, const uint8_t* __restrict__ mask,
                                  unsigned long long* __restrict__ count) {
    unsigned local = 0;
    const int64_t n = n_cells * row;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        if (!mask[i / row]) continue;
        const float v = St<T>::ld1(p + i);
        local += (v - v) != 0.0f ? 1u : 0u;  // NaN or +-inf
    }
    for (int o = 32; o > 0; o >>= 1) local += __shfl_xor(local, o);
    if ((threadIdx.x & 63) == 0 && local) atomicAdd(count, (unsigned long long)local);
}

hipError_t launch_count_nonfinite(const void* d, int64_t n_cells, int row, const uint8_t* d_mask, int dtype,
                                  unsigned long long* d_count, hipStream_t s) {
    if (n_cells <= 0 || row <= 0) return hipSuccess;
    const int blocks = (int)std::min<int64_t>((n_cells * row + 255) / 256, 4096);
    if (dtype == 0)
        hipLaunchKernelGGL(k_count_nonfinite<float>, dim3(blocks), dim3(256), 0, s, static_cast<const float*>(d),
                           n_cells, row, d_mask, d_count);
    else
        hipLaunchKernelGGL(k_count_nonfinite<bf16_t>, dim3(blocks), dim3(256), 0, s, static_cast<const bf16_t*>(d),
                           n_cells, row, d_mask, d_count);
    return hipGetLastError();
}

}  // namespace mdl
