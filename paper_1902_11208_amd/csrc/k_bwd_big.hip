// Input and weight gradients for the shapes the fused strip kernel does not
// cover (hidden sizes 64 and 128, other c_in), as two tiled MFMA products:
//   dX[p]  = valid(p) * sum_n dZ[p][n] Wx_all[n][:]                (K = 20H)
//   dW_d   = sum_p valid(p) dZ_d[p] (x) [X[p] ; h_L,d(p) ; h_T,d(p)]  (K = cells)
//   db_d   = sum_p valid(p) dZ_d[p]
// with h_L,d / h_T,d the layer output at p's left / top predecessor in
// direction d's frame, zero when that predecessor is outside p's rectangle or
// masked (the shifted recurrent operand of Appendix A).
//
// bf16 storage runs 16x16x32 bf16 MFMAs, fp32 storage 16x16x4 fp32 MFMAs;
// both accumulate in fp32. A validity byte per cell (bit 0 valid, bits 1-4
// left / right / up / down neighbour in the same rectangle and unmasked) is
// computed once per call.
//
// dX: A = Wx_all^T (rows = channels, from a transposed copy), B = dZ rows
// (cells), K = 20H; a wave owns 64 cells x 64 channels.
// dW: per direction, a workgroup owns a 128 x 128 block of [5H] x [c_in + 2H]
// for one chunk of cells; each step stages 32 cells of dZ and of the column
// operand in LDS transposed (cells contiguous), so that an MFMA operand is
// one 16-byte LDS read; the next step's loads are in flight meanwhile. The
// chunks' partial products are summed in a fixed order.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

namespace {

// 16-byte chunk: E elements of storage type T.
template <typename T>
struct BigT;
template <>
struct BigT<float> {
    static constexpr int E = 4;       // elements per 16 bytes
    static constexpr int KSTEP = 16;  // reduction values per operand read (4 MFMAs of K = 4)
};
template <>
struct BigT<bf16_t> {
    static constexpr int E = 8;
    static constexpr int KSTEP = 32;  // one 16x16x32 MFMA
};

__device__ __forceinline__ u32x4 zero4() { return u32x4{0u, 0u, 0u, 0u}; }

// acc += A * B over one 16-byte operand pair: bf16, one 16x16x32 MFMA; fp32,
// four 16x16x4 MFMAs (element j of both operands in MFMA j).
template <typename T>
__device__ __forceinline__ floatx4 mma16(u32x4 a, u32x4 b, floatx4 acc) {
    if constexpr (std::is_same<T, float>::value) {
#pragma unroll
        for (int j = 0; j < 4; ++j) acc = mfma_f32(__uint_as_float(a[j]), __uint_as_float(b[j]), acc);
        return acc;
    } else {
        bf16x8 av, bv;
        __builtin_memcpy(&av, &a, 16);
        __builtin_memcpy(&bv, &b, 16);
        return mfma_bf16(av, bv, acc);
    }
}

}  // namespace

// --- validity byte per cell ------------------------------------------------
__global__ void k_cell_flags(int canvas_h, int canvas_w, const uint8_t* __restrict__ mask,
                             const int32_t* __restrict__ rid, uint8_t* __restrict__ flags) {
    const int64_t n = (int64_t)canvas_h * canvas_w;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += (int64_t)gridDim.x * blockDim.x) {
        const int cy = (int)(p / canvas_w), cx = (int)(p - (int64_t)cy * canvas_w);
        const int r = rid[p];
        uint8_t f = 0;
        if (mask[p] && r >= 0) {
            f = 1;
            if (cx > 0 && rid[p - 1] == r && mask[p - 1]) f |= 2;
            if (cx + 1 < canvas_w && rid[p + 1] == r && mask[p + 1]) f |= 4;
            if (cy > 0 && rid[p - canvas_w] == r && mask[p - canvas_w]) f |= 8;
            if (cy + 1 < canvas_h && rid[p + canvas_w] == r && mask[p + canvas_w]) f |= 16;
        }
        flags[p] = f;
    }
}

// --- Wx_all [N][C] -> WxT [C][N] ---------------------------------------------
template <typename T>
__global__ void k_transpose(int rows, int cols, const T* __restrict__ src, T* __restrict__ dst) {
    const int64_t n = (int64_t)rows * cols;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int r = (int)(i / cols), c = (int)(i - (int64_t)r * cols);
        dst[(int64_t)c * rows + r] = src[i];
    }
}

// --- dX ------------------------------------------------------------------------
// Wave: 64 cells (four N tiles) x up to 64 channels (four M tiles) of one
// channel group (blockIdx.y). Lane (g, i16) reads, per reduction step, the
// 16 bytes of row k0 + E g of its channel (WxT) and of its cell (dZ).
template <typename T>
__global__ void __launch_bounds__(256)
k_dx_big(int64_t n_cells, int C, int N, const T* __restrict__ dZ, const T* __restrict__ WxT,
         const uint8_t* __restrict__ flags, T* __restrict__ dX) {
    using B = BigT<T>;
    constexpr int E = B::E, KS = B::KSTEP;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int64_t cell0 = ((int64_t)blockIdx.x * 4 + wave) * 64;
    if (cell0 >= n_cells) return;
    const int ch0 = blockIdx.y * 64;
    const int nmt = min(4, (C - ch0 + 15) / 16);
    const char* Zb = reinterpret_cast<const char*>(dZ);
    const char* Wb = reinterpret_cast<const char*>(WxT);
    int64_t cl[4];
    bool ok[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int64_t c = cell0 + 16 * t + i16;
        ok[t] = c < n_cells && (flags[min(c, n_cells - 1)] & 1);
        cl[t] = min(c, n_cells - 1);
    }
    int chl[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) chl[m] = min(ch0 + 16 * m + i16, C - 1);
    floatx4 acc[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[m][t] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int64_t rb = (int64_t)N * sizeof(T);
    const int koff = E * g * (int)sizeof(T);
    for (int k0 = 0; k0 < N; k0 += KS) {
        u32x4 a[4], b[4];
#pragma unroll
        for (int m = 0; m < 4; ++m)
            a[m] = *reinterpret_cast<const u32x4*>(Wb + chl[m] * rb + (int64_t)k0 * sizeof(T) + koff);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(Zb + cl[t] * rb + (int64_t)k0 * sizeof(T) + koff);
            b[t] = ok[t] ? v : zero4();
        }
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[m][t] = mma16<T>(a[m], b[t], acc[m][t]);
    }
    // lane (q, n) holds channels 4 q .. 4 q + 3 of cell n of every tile pair
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const int ch = ch0 + 16 * m + 4 * g;
        if (m >= nmt || ch >= C) continue;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int64_t c = cell0 + 16 * t + i16;
            if (c < n_cells) St<T>::st4(dX + c * C + ch, acc[m][t]);
        }
    }
}

// --- dW --------------------------------------------------------------------------
constexpr int BW_KC = 32;    // cells per step
constexpr int BW_RB = 128;   // gate rows per workgroup
constexpr int BW_CB = 128;   // columns per workgroup
constexpr int BW_TARGET = 512;  // workgroups aimed for

struct BigDw {
    int G, NB, rblocks, cblocks, chunks, PP;
    int64_t chunk_cells;
};

static BigDw big_dw(const LayerGeom& g) {
    BigDw q;
    q.G = 5 * g.hidden;
    q.NB = g.c_in + 2 * g.hidden;
    q.rblocks = (q.G + BW_RB - 1) / BW_RB;
    q.cblocks = (q.NB + BW_CB - 1) / BW_CB;
    q.PP = q.NB + 1;  // partial row: the columns, then the bias
    const int per_chunk = q.rblocks * q.cblocks * 4;
    int64_t ch = (BW_TARGET + per_chunk - 1) / per_chunk;
    const int64_t by_size = std::max<int64_t>(1, g.n_cells / (16 * BW_KC));  // at least 16 steps per chunk
    ch = std::max<int64_t>(1, std::min(ch, by_size));
    q.chunk_cells = (g.n_cells + ch - 1) / ch;
    q.chunk_cells = (q.chunk_cells + BW_KC - 1) / BW_KC * BW_KC;
    q.chunks = (int)((g.n_cells + q.chunk_cells - 1) / q.chunk_cells);
    if (q.chunks < 1) q.chunks = 1;
    return q;
}

// Workgroup (row block, column block, direction) x chunk. LDS holds the
// step's operands transposed: sA[row][cell], sB[col][cell] (pitch KC + 8
// elements). Wave w owns rows 32 w .. 32 w + 31 (two M tiles) and all eight
// N tiles of the column block. Thread t stages cell t % KC: the 16-byte
// chunks (t / KC) + 8 j of the cell's dZ rows and of its column operand.
template <typename T>
__global__ void __launch_bounds__(256)
k_dw_big(int64_t n_cells, int canvas_w, int C, int H, BigDw q, const T* __restrict__ dZ, const T* __restrict__ X,
         const T* __restrict__ Y, const uint8_t* __restrict__ flags, float* __restrict__ part) {
    using B = BigT<T>;
    constexpr int E = B::E;
    constexpr int KC = BW_KC, PIT = KC + 8;
    constexpr int CPC = BW_RB / E;            // 16-byte chunks per cell row of a block
    constexpr int NJ = CPC / 8;               // chunks per thread (8 threads per cell)
    __shared__ __attribute__((aligned(16))) T sA[BW_RB][PIT];
    __shared__ __attribute__((aligned(16))) T sB[BW_CB][PIT];

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int rb = blockIdx.x % q.rblocks, cb = (blockIdx.x / q.rblocks) % q.cblocks, d = blockIdx.x / (q.rblocks * q.cblocks);
    const int chunk = blockIdx.y;
    const int G = q.G, N = 20 * H;
    const int r0 = rb * BW_RB, c0 = cb * BW_CB;
    const int64_t k_begin = (int64_t)chunk * q.chunk_cells;
    const int64_t k_end = min(n_cells, k_begin + q.chunk_cells);
    const int lstep = (d & 1) ? 1 : -1;                // left predecessor: cell + lstep
    const int64_t tstep = (d & 2) ? canvas_w : -(int64_t)canvas_w;  // top predecessor
    const uint8_t lbit = (d & 1) ? 4 : 2, tbit = (d & 2) ? 16 : 8;

    const int cs = tid % KC, cq = tid / KC;  // staging: cell slot, chunk phase
    // source of column chunk k (k = cq + 8 j): 0 X, 1 left, 2 top, 3 none; element offset in its row
    int ksrc[NJ], koff[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int col = c0 + E * (cq + 8 * j);
        if (col < C) { ksrc[j] = 0; koff[j] = col; }
        else if (col < C + H) { ksrc[j] = 1; koff[j] = d * H + col - C; }
        else if (col < C + 2 * H) { ksrc[j] = 2; koff[j] = d * H + col - C - H; }
        else { ksrc[j] = 3; koff[j] = 0; }
    }
    const int rlim = min(BW_RB, G - r0);  // rows of this block inside the direction
    u32x4 va[NJ], vb[NJ];
    uint32_t vf;
    auto issue = [&](int64_t kb) {
        const int64_t p = kb + cs;
        const bool in = p < k_end;
        const int64_t pc = in ? p : k_end - 1;
        vf = in ? flags[pc] : 0u;
        const int64_t pl = min(max(pc + lstep, (int64_t)0), n_cells - 1);
        const int64_t pt = min(max(pc + tstep, (int64_t)0), n_cells - 1);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int rr = E * (cq + 8 * j);
            va[j] = *reinterpret_cast<const u32x4*>(dZ + pc * N + d * G + r0 + min(rr, max(rlim - E, 0)));
            const T* src = ksrc[j] == 0 ? X + pc * C : (ksrc[j] == 1 ? Y + pl * (4 * H) : Y + pt * (4 * H));
            vb[j] = *reinterpret_cast<const u32x4*>(src + koff[j]);
        }
    };
    auto commit = [&]() {
        const bool v = vf & 1, vl = vf & lbit, vt = vf & tbit;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int rr = E * (cq + 8 * j);
            const bool oka = v && rr < rlim;
            const bool okb = v && (ksrc[j] == 0 || (ksrc[j] == 1 && vl) || (ksrc[j] == 2 && vt));
            const u32x4 a = oka ? va[j] : zero4();
            const u32x4 b = okb ? vb[j] : zero4();
            const T* ae = reinterpret_cast<const T*>(&a);
            const T* be = reinterpret_cast<const T*>(&b);
#pragma unroll
            for (int e = 0; e < E; ++e) {
                sA[rr + e][cs] = ae[e];
                sB[rr + e][cs] = be[e];
            }
        }
    };

    floatx4 acc[2][8];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int n = 0; n < 8; ++n) acc[m][n] = floatx4{0.f, 0.f, 0.f, 0.f};
    // bias (column block 0 only): thread t sums row t / 2, cells of half t % 2
    float bsum = 0.0f;
    const bool do_bias = cb == 0;

    if (k_begin < k_end) issue(k_begin);
    for (int64_t kb = k_begin; kb < k_end; kb += KC) {
        commit();
        lds_barrier();
        issue(kb + KC);  // past the chunk's end the loads re-read its last cell (flags 0)
        if (do_bias) {
            const int row = tid >> 1, h = tid & 1;
#pragma unroll 8
            for (int c = 0; c < KC / 2; ++c) bsum += St<T>::ld1(&sA[row][h * (KC / 2) + c]);
        }
        // MFMA: lane (g, i16) reads row 32 w + 16 m + i16 of sA and column 16 n + i16 of sB,
        // cells KS-blocks: fp32 cells 16 s + 4 g .. + 3; bf16 cells 8 g .. 8 g + 7
        constexpr int KS = B::KSTEP;
#pragma unroll
        for (int s = 0; s < KC / KS; ++s) {
            u32x4 a[2], b[8];
#pragma unroll
            for (int m = 0; m < 2; ++m) a[m] = *reinterpret_cast<const u32x4*>(&sA[32 * wave + 16 * m + i16][KS * s + E * g]);
#pragma unroll
            for (int n = 0; n < 8; ++n) b[n] = *reinterpret_cast<const u32x4*>(&sB[16 * n + i16][KS * s + E * g]);
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int n = 0; n < 8; ++n) acc[m][n] = mma16<T>(a[m], b[n], acc[m][n]);
        }
        lds_barrier();
    }

    // partial [chunk][d][G][PP]: columns then the bias; lane (q, n) holds rows 4 q + r of tile (m, n)
    float* out = part + ((int64_t)chunk * 4 + d) * (int64_t)G * q.PP;
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int n = 0; n < 8; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = r0 + 32 * wave + 16 * m + 4 * g + r, col = c0 + 16 * n + i16;
                if (row < G && col < q.NB) out[(int64_t)row * q.PP + col] = acc[m][n][r];
            }
    if (do_bias) {
        bsum += __shfl_xor(bsum, 1);
        const int row = r0 + (tid >> 1);
        if ((tid & 1) == 0 && row < G) out[(int64_t)row * q.PP + q.NB] = bsum;
    }
}

// Fixed-order sum of the chunk partials into dWx, dU, db.
__global__ void k_dw_big_reduce(int C, int H, BigDw q, const float* __restrict__ part, float* __restrict__ dwx,
                                float* __restrict__ du, float* __restrict__ db) {
    const int G = q.G;
    const int64_t total = (int64_t)4 * G * q.PP;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int d = (int)(idx / ((int64_t)G * q.PP));
        const int rem = (int)(idx - (int64_t)d * G * q.PP);
        const int r = rem / q.PP, col = rem - r * q.PP;
        const float* src = part + (int64_t)d * G * q.PP + (int64_t)r * q.PP + col;
        float s = 0.0f;
        for (int c = 0; c < q.chunks; ++c) s += src[(int64_t)c * 4 * G * q.PP];
        if (col < C) dwx[((int64_t)d * G + r) * C + col] = s;
        else if (col < C + 2 * H) du[((int64_t)d * G + r) * (2 * H) + (col - C)] = s;
        else db[(int64_t)d * G + r] = s;
    }
}

// --- host --------------------------------------------------------------------------
size_t big_flags_bytes(const LayerGeom& g) { return (size_t)(g.n_cells > 0 ? g.n_cells : 1); }
size_t big_wxt_bytes(const LayerGeom& g) {
    return (size_t)g.c_in * 20 * g.hidden * (g.dtype == 0 ? 4 : 2);
}
size_t big_partial_bytes(const LayerGeom& g) {
    const BigDw q = big_dw(g);
    return (size_t)q.chunks * 4 * q.G * q.PP * sizeof(float);
}

hipError_t launch_bwd_big(const LayerGeom& g, const void* d_dz, const void* d_x, const void* d_y, const void* d_wx,
                          const uint8_t* d_mask, const int32_t* d_rid, void* d_dx, uint8_t* d_flags, void* d_wxt,
                          float* d_part, float* d_dwx, float* d_du, float* d_db, hipStream_t s) {
    if (g.n_cells == 0) return hipSuccess;
    const int N = 20 * g.hidden;
    int fb = (int)std::min<int64_t>((g.n_cells + 255) / 256, 4096);
    hipLaunchKernelGGL(k_cell_flags, dim3(fb), dim3(256), 0, s, g.canvas_h, g.canvas_w, d_mask, d_rid, d_flags);
    const int64_t nw = (int64_t)N * g.c_in;
    const int tb = (int)std::min<int64_t>((nw + 255) / 256, 4096);
    const BigDw q = big_dw(g);
    const dim3 gx((unsigned)(((g.n_cells + 63) / 64 + 3) / 4), (unsigned)((g.c_in + 63) / 64));
    const dim3 gw((unsigned)(q.rblocks * q.cblocks * 4), (unsigned)q.chunks);
    const int64_t total = (int64_t)4 * q.G * q.PP;
    const int rbk = (int)std::min<int64_t>((total + 255) / 256, 4096);
    if (g.dtype == 0) {
        using T = float;
        hipLaunchKernelGGL(k_transpose<T>, dim3(tb), dim3(256), 0, s, N, g.c_in, static_cast<const T*>(d_wx),
                           static_cast<T*>(d_wxt));
        hipLaunchKernelGGL(k_dx_big<T>, gx, dim3(256), 0, s, g.n_cells, g.c_in, N, static_cast<const T*>(d_dz),
                           static_cast<const T*>(d_wxt), d_flags, static_cast<T*>(d_dx));
        hipLaunchKernelGGL(k_dw_big<T>, gw, dim3(256), 0, s, g.n_cells, g.canvas_w, g.c_in, g.hidden, q,
                           static_cast<const T*>(d_dz), static_cast<const T*>(d_x), static_cast<const T*>(d_y),
                           d_flags, d_part);
    } else {
        using T = bf16_t;
        hipLaunchKernelGGL(k_transpose<T>, dim3(tb), dim3(256), 0, s, N, g.c_in, static_cast<const T*>(d_wx),
                           static_cast<T*>(d_wxt));
        hipLaunchKernelGGL(k_dx_big<T>, gx, dim3(256), 0, s, g.n_cells, g.c_in, N, static_cast<const T*>(d_dz),
                           static_cast<const T*>(d_wxt), d_flags, static_cast<T*>(d_dx));
        hipLaunchKernelGGL(k_dw_big<T>, gw, dim3(256), 0, s, g.n_cells, g.canvas_w, g.c_in, g.hidden, q,
                           static_cast<const T*>(d_dz), static_cast<const T*>(d_x), static_cast<const T*>(d_y),
                           d_flags, d_part);
    }
    hipLaunchKernelGGL(k_dw_big_reduce, dim3(rbk), dim3(256), 0, s, g.c_in, g.hidden, q, d_part, d_dwx, d_du, d_db);
    return hipGetLastError();
}

}  // namespace mdl
