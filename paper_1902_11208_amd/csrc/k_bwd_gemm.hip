// Input and weight gradients of the MDLSTM layer from dZ (the gradient of the
// gate pre-activations, written by the backward wavefront):
//   dX[p]      = valid(p) * sum_n dZ[p][n] Wx_all[n][:]
//   dW_d       = sum_p valid(p) dZ[p][d*5H : d*5H+5H] (x) [X[p] ; h_L,d(p) ; h_T,d(p) ; 1]
// where h_L,d(p) / h_T,d(p) are the hidden states of p's left / top
// predecessor in direction d's frame (zero when the predecessor is outside
// p's rectangle or masked). The predecessor operand is the layer output
// shifted by one cell, the way Appendix A shifts the recurrent activations so
// that left and top contributions line up; dWx, dU and db come out of one
// product per direction as column blocks.
//
// Both products run on 16x16x4 fp32 MFMA (bf16 storage is widened on load).
// The weight-gradient reduction over cells is split into fixed chunks; a
// second kernel sums the chunk partials in a fixed order, so results are
// deterministic.
#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

template <typename T>
__device__ __forceinline__ float ldf(const T* p) {
    return St<T>::ld1(p);
}

__device__ __forceinline__ bool cell_valid(const uint8_t* mask, const int32_t* rid, int64_t p) {
    return mask[p] != 0 && rid[p] >= 0;
}

// ---------------------------------------------------------------------------
// dX: M = input channels (A = Wx_all^T), N = cells (B = dZ^T), K = 20H.
// K step ks covers n = 4 ks + g. Each wave owns 64 cells (four N tiles) and all
// channel tiles (at most 4, i.e. c_in <= 64 per pass; larger c_in loops).
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256)
k_dx(int64_t n_cells, int C, int N, const T* __restrict__ dZ, const T* __restrict__ Wx,
     const uint8_t* __restrict__ mask, const int32_t* __restrict__ rid, T* __restrict__ dX) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int64_t cell0 = ((int64_t)blockIdx.x * 4 + wave) * 64;
    if (cell0 >= n_cells) return;
    bool ok[4];
    int64_t cell[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        cell[t] = cell0 + 16 * t + i16;
        ok[t] = cell[t] < n_cells && cell_valid(mask, rid, cell[t]);
    }
    for (int mt0 = 0; mt0 < (C + 15) / 16; mt0 += 4) {
        floatx4 acc[4][4];
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[m][t] = floatx4{0.f, 0.f, 0.f, 0.f};
        const int nmt = min(4, (C + 15) / 16 - mt0);
        for (int ks = 0; ks < N / 4; ++ks) {
            const int n = 4 * ks + g;
            float b[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) b[t] = ok[t] ? ldf(dZ + cell[t] * N + n) : 0.0f;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                if (m < nmt) {
                    const int ch = (mt0 + m) * 16 + i16;
                    const float av = ch < C ? ldf(Wx + (int64_t)n * C + ch) : 0.0f;
#pragma unroll
                    for (int t = 0; t < 4; ++t) acc[m][t] = mfma_f32(av, b[t], acc[m][t]);
                }
            }
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            if (m >= nmt) continue;
            const int ch = (mt0 + m) * 16 + 4 * g;
            if (ch >= C) continue;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                int64_t c = cell0 + 16 * t + i16;
                if (c < n_cells) St<T>::st4(dX + c * C + ch, ok[t] ? acc[m][t] : floatx4{0.f, 0.f, 0.f, 0.f});
            }
        }
    }
}

hipError_t launch_dx(const LayerGeom& g, const void* d_dz, const void* d_wx, const uint8_t* d_mask,
                     const int32_t* d_rid, void* d_dx, hipStream_t s) {
    if (g.n_cells == 0) return hipSuccess;
    const int N = 20 * g.hidden;
    const int64_t waves = (g.n_cells + 63) / 64;
    const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
    if (g.dtype == 0)
        hipLaunchKernelGGL(k_dx<float>, grid, block, 0, s, g.n_cells, g.c_in, N, static_cast<const float*>(d_dz),
                           static_cast<const float*>(d_wx), d_mask, d_rid, static_cast<float*>(d_dx));
    else
        hipLaunchKernelGGL(k_dx<bf16_t>, grid, block, 0, s, g.n_cells, g.c_in, N, static_cast<const bf16_t*>(d_dz),
                           static_cast<const bf16_t*>(d_wx), d_mask, d_rid, static_cast<bf16_t*>(d_dx));
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight gradients. Per direction d the product O_d[5H][NB] with
// NB = c_in + 2H + 1 columns: [0, c_in) input, [c_in, c_in+H) left predecessor
// hidden state, [c_in+H, c_in+2H) top predecessor hidden state, c_in+2H bias.
// A = dZ^T (rows r = gate rows of direction d), B = the column operand, K = cells.
// A workgroup = 4 waves, each owning a block of up to 4 x 4 output tiles;
// grid = (cell chunks, tile groups, 4 directions).
// ---------------------------------------------------------------------------
constexpr int DW_TB = 4;  // tiles per wave block side

struct DwGeom {
    int RT, CT, NB, NBP, groups, chunks;
    int64_t chunk_cells;
};

static DwGeom dw_geom(const LayerGeom& g) {
    DwGeom q;
    q.RT = (5 * g.hidden + 15) / 16;
    q.NB = g.c_in + 2 * g.hidden + 1;
    q.CT = (q.NB + 15) / 16;
    q.NBP = q.CT * 16;
    const int blocks = ((q.RT + DW_TB - 1) / DW_TB) * ((q.CT + DW_TB - 1) / DW_TB);
    q.groups = (blocks + 3) / 4;
    int64_t target = 2048 / (4 * (int64_t)q.groups);  // aim for ~2048 workgroups in flight
    if (target < 1) target = 1;
    int64_t by_size = (g.n_cells + 255) / 256;  // at least 256 cells per chunk
    int64_t ch = target < by_size ? target : by_size;
    if (ch < 1) ch = 1;
    q.chunks = (int)ch;
    q.chunk_cells = (g.n_cells + ch - 1) / ch;
    q.chunk_cells = (q.chunk_cells + 3) / 4 * 4;
    return q;
}

int dw_chunks(const LayerGeom& g) { return dw_geom(g).chunks; }

size_t dw_partial_bytes(const LayerGeom& g) {
    DwGeom q = dw_geom(g);
    return (size_t)4 * q.chunks * q.RT * 16 * q.NBP * sizeof(float);
}

template <typename T>
__global__ void __launch_bounds__(256)
k_dw_partial(int64_t n_cells, int canvas_h, int canvas_w, int C, int H, DwGeom q, const T* __restrict__ dZ,
             const T* __restrict__ X, const T* __restrict__ Y, const uint8_t* __restrict__ mask,
             const int32_t* __restrict__ rid, float* __restrict__ part) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int chunk = blockIdx.x, d = blockIdx.z;
    const int bcols = (q.CT + DW_TB - 1) / DW_TB;
    const int blk = blockIdx.y * 4 + wave;
    const int nblocks = ((q.RT + DW_TB - 1) / DW_TB) * bcols;
    if (blk >= nblocks) return;
    const int rt0 = (blk / bcols) * DW_TB, ct0 = (blk % bcols) * DW_TB;
    const int G = 5 * H, N = 20 * H;
    const int64_t c_begin = (int64_t)chunk * q.chunk_cells;
    const int64_t c_end = min(n_cells, c_begin + q.chunk_cells);

    // column kind per owned column tile: 0 input, 1 left, 2 top, 3 one, 4 zero
    int kind[DW_TB], off[DW_TB];
#pragma unroll
    for (int ct = 0; ct < DW_TB; ++ct) {
        const int col = (ct0 + ct) * 16 + i16;
        if (col < C) { kind[ct] = 0; off[ct] = col; }
        else if (col < C + H) { kind[ct] = 1; off[ct] = d * H + (col - C); }
        else if (col < C + 2 * H) { kind[ct] = 2; off[ct] = d * H + (col - C - H); }
        else if (col == C + 2 * H) { kind[ct] = 3; off[ct] = 0; }
        else { kind[ct] = 4; off[ct] = 0; }
    }
    // predecessor offsets in canvas coordinates for direction d
    const int dxL = (d & 1) ? 1 : -1;  // left predecessor column step
    const int dyT = (d & 2) ? 1 : -1;  // top predecessor row step

    floatx4 acc[DW_TB][DW_TB];
#pragma unroll
    for (int a = 0; a < DW_TB; ++a)
#pragma unroll
        for (int b = 0; b < DW_TB; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    for (int64_t kb = c_begin; kb < c_end; kb += 4) {
        const int64_t p = kb + g;
        bool v = p < c_end && cell_valid(mask, rid, p);
        int64_t pL = -1, pT = -1;
        if (v) {
            const int cy = (int)(p / canvas_w), cx = (int)(p - (int64_t)cy * canvas_w);
            const int r = rid[p];
            const int lx = cx + dxL, ty = cy + dyT;
            if (lx >= 0 && lx < canvas_w) {
                int64_t pp = (int64_t)cy * canvas_w + lx;
                if (rid[pp] == r && mask[pp]) pL = pp;
            }
            if (ty >= 0 && ty < canvas_h) {
                int64_t pp = (int64_t)ty * canvas_w + cx;
                if (rid[pp] == r && mask[pp]) pT = pp;
            }
        }
        float av[DW_TB], bv[DW_TB];
#pragma unroll
        for (int a = 0; a < DW_TB; ++a) {
            const int r = (rt0 + a) * 16 + i16;
            av[a] = (v && r < G) ? ldf(dZ + p * N + d * G + r) : 0.0f;
        }
#pragma unroll
        for (int b = 0; b < DW_TB; ++b) {
            float x = 0.0f;
            if (v) {
                switch (kind[b]) {
                    case 0: x = ldf(X + p * C + off[b]); break;
                    case 1: x = pL >= 0 ? ldf(Y + pL * (4 * H) + off[b]) : 0.0f; break;
                    case 2: x = pT >= 0 ? ldf(Y + pT * (4 * H) + off[b]) : 0.0f; break;
                    case 3: x = 1.0f; break;
                    default: x = 0.0f;
                }
            }
            bv[b] = x;
        }
#pragma unroll
        for (int a = 0; a < DW_TB; ++a)
#pragma unroll
            for (int b = 0; b < DW_TB; ++b) acc[a][b] = mfma_f32(av[a], bv[b], acc[a][b]);
    }
    // partial layout: [d][chunk][RT*16][NBP]
    float* out = part + ((int64_t)d * q.chunks + chunk) * (int64_t)(q.RT * 16) * q.NBP;
#pragma unroll
    for (int a = 0; a < DW_TB; ++a) {
        if (rt0 + a >= q.RT) continue;
#pragma unroll
        for (int b = 0; b < DW_TB; ++b) {
            if (ct0 + b >= q.CT) continue;
            const int col = (ct0 + b) * 16 + i16;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = (rt0 + a) * 16 + 4 * g + r;
                out[(int64_t)row * q.NBP + col] = acc[a][b][r];
            }
        }
    }
}

// Fixed-order sum of the chunk partials, scattered into dWx, dU, db.
__global__ void k_dw_reduce(int C, int H, DwGeom q, const float* __restrict__ part, float* __restrict__ dwx,
                            float* __restrict__ du, float* __restrict__ db) {
    const int G = 5 * H;
    const int64_t total = (int64_t)4 * G * q.NB;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int d = (int)(idx / ((int64_t)G * q.NB));
        const int rem = (int)(idx - (int64_t)d * G * q.NB);
        const int r = rem / q.NB, col = rem - r * q.NB;
        const float* src = part + (int64_t)d * q.chunks * (q.RT * 16) * q.NBP + (int64_t)r * q.NBP + col;
        float s = 0.0f;
        for (int c = 0; c < q.chunks; ++c) s += src[(int64_t)c * (q.RT * 16) * q.NBP];
        if (col < C) dwx[((int64_t)d * G + r) * C + col] = s;
        else if (col < C + 2 * H) du[((int64_t)d * G + r) * (2 * H) + (col - C)] = s;
        else db[(int64_t)d * G + r] = s;
    }
}

hipError_t launch_dw(const LayerGeom& g, const void* d_dz, const void* d_x, const void* d_y, const uint8_t* d_mask,
                     const int32_t* d_rid, float* d_part, float* d_dwx, float* d_du, float* d_db, hipStream_t s) {
    DwGeom q = dw_geom(g);
    const dim3 grid(q.chunks, q.groups, 4), block(256);
    // chunks past the last cell (or an empty canvas) write zero partials
    if (g.dtype == 0)
        hipLaunchKernelGGL(k_dw_partial<float>, grid, block, 0, s, g.n_cells, g.canvas_h, g.canvas_w, g.c_in,
                           g.hidden, q, static_cast<const float*>(d_dz), static_cast<const float*>(d_x),
                           static_cast<const float*>(d_y), d_mask, d_rid, d_part);
    else
        hipLaunchKernelGGL(k_dw_partial<bf16_t>, grid, block, 0, s, g.n_cells, g.canvas_h, g.canvas_w, g.c_in,
                           g.hidden, q, static_cast<const bf16_t*>(d_dz), static_cast<const bf16_t*>(d_x),
                           static_cast<const bf16_t*>(d_y), d_mask, d_rid, d_part);
    const int64_t total = (int64_t)4 * 5 * g.hidden * q.NB;
    int blocks = (int)((total + 255) / 256);
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_dw_reduce, dim3(blocks), dim3(256), 0, s, g.c_in, g.hidden, q, d_part, d_dwx, d_du, d_db);
    return hipGetLastError();
}

}  // namespace mdl
