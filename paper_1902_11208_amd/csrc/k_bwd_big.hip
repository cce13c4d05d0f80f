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
// dW: per direction, a workgroup owns a 320 x 160 block of [5H] x [c_in + 2H]
// for one chunk of cells. fp32 (k_dw_big): each step stages 32 cells of dZ
// and of the column operand in LDS transposed (cells contiguous) through
// registers, so that an MFMA operand is one 16-byte LDS read; the next
// step's loads are in flight meanwhile. bf16 (k_dw_tr): the steps are copied
// to LDS directly, cell-major as in memory, and the MFMA operands are read
// with the LDS transpose read. The chunks' partial products are summed in a
// fixed order.
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
// 16 bytes of row k0 + E g of its channel (WxT) and of its cell (dZ). When
// there are too few cells to fill the CUs with such waves (SPLIT), the four
// waves of a workgroup take 16 cells together, each a quarter of the
// reduction steps, and their sums are added in LDS in wave order.
template <typename T, bool SPLIT>
__global__ void __launch_bounds__(256)
k_dx_big(int64_t n_cells, int C, int N, const T* __restrict__ dZ, const T* __restrict__ WxT,
         const uint8_t* __restrict__ flags, T* __restrict__ dX) {
    using B = BigT<T>;
    constexpr int E = B::E, KS = B::KSTEP, CT = SPLIT ? 1 : 4;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int64_t cell0 = SPLIT ? (int64_t)blockIdx.x * 16 : ((int64_t)blockIdx.x * 4 + wave) * 64;
    if (cell0 >= n_cells) return;
    const int ch0 = blockIdx.y * 64;
    const int nmt = min(4, (C - ch0 + 15) / 16);
    const char* Zb = reinterpret_cast<const char*>(dZ);
    const char* Wb = reinterpret_cast<const char*>(WxT);
    int64_t cl[CT];
    bool ok[CT];
#pragma unroll
    for (int t = 0; t < CT; ++t) {
        const int64_t c = cell0 + 16 * t + i16;
        ok[t] = c < n_cells && (flags[min(c, n_cells - 1)] & 1);
        cl[t] = min(c, n_cells - 1);
    }
    int chl[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) chl[m] = min(ch0 + 16 * m + i16, C - 1);
    floatx4 acc[4][CT];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int t = 0; t < CT; ++t) acc[m][t] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int64_t rb = (int64_t)N * sizeof(T);
    const int koff = E * g * (int)sizeof(T);
    const int nsteps = (N + KS - 1) / KS;
    const int k_begin = SPLIT ? KS * (nsteps * wave / 4) : 0;
    const int k_end = SPLIT ? min(N, KS * (nsteps * (wave + 1) / 4)) : N;
    for (int k0 = k_begin; k0 < k_end; k0 += KS) {
        u32x4 a[4], b[CT];
#pragma unroll
        for (int m = 0; m < 4; ++m)
            a[m] = *reinterpret_cast<const u32x4*>(Wb + chl[m] * rb + (int64_t)k0 * sizeof(T) + koff);
#pragma unroll
        for (int t = 0; t < CT; ++t) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(Zb + cl[t] * rb + (int64_t)k0 * sizeof(T) + koff);
            b[t] = ok[t] ? v : zero4();
        }
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int t = 0; t < CT; ++t) acc[m][t] = mma16<T>(a[m], b[t], acc[m][t]);
    }
    if constexpr (SPLIT) {
        __shared__ floatx4 part[3][4][64];
        if (wave > 0) {
#pragma unroll
            for (int m = 0; m < 4; ++m) part[wave - 1][m][lane] = acc[m][0];
        }
        __syncthreads();
        if (wave > 0) return;
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int w = 0; w < 3; ++w) acc[m][0] += part[w][m][lane];
    }
    // lane (q, n) holds channels 4 q .. 4 q + 3 of cell n of every tile pair
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const int ch = ch0 + 16 * m + 4 * g;
        if (m >= nmt || ch >= C) continue;
#pragma unroll
        for (int t = 0; t < CT; ++t) {
            const int64_t c = cell0 + 16 * t + i16;
            if (c < n_cells) St<T>::st4(dX + c * C + ch, acc[m][t]);
        }
    }
}

// --- dX, bf16: direct-to-LDS staging --------------------------------------------
// A workgroup of eight waves takes blocks of 128 cells in turn; each wave
// owns 16 of them (one N tile) and every channel tile, so that one staged
// copy of the WxT rows serves 128 cells. The reduction over the 20H gate rows
// runs in stages of KC (128 values, 64 for inputs wider than 128): the
// stage's dZ rows of the block's cells (256 contiguous bytes of each; HBM
// serves such runs far better than 64-byte pieces of many rows) and the
// WxT rows (channels, padded to a multiple of 64 with re-read rows) are
// copied by direct global-to-LDS loads, the next stage's copy in flight
// during the current one's MFMAs (one stream across blocks). A staged row's
// 16-byte chunk j sits at j ^ (r & 15) within aligned groups of sixteen (of
// eight at KC = 64), so the sixteen rows one operand read touches fall on
// distinct banks. The dX rows of invalid cells are written as zero.
namespace {
constexpr int DX_CELLS = 128;
constexpr int NWV = DX_CELLS / 16;
// LDS-only barrier without a fence, so that the direct-to-LDS loads of the
// next stage (into the other buffers) are not waited for
__device__ __forceinline__ void dx_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
// The operands of one reduction step, 1 + MT 16-byte LDS reads, issued and
// waited for in one asm statement (MT <= 4): the compiler does not know
// which buffer the direct loads in flight fill, and before its own LDS reads
// it would wait for the next stage's loads as well. The values are complete
// when the statement ends.
template <int MT>
__device__ __forceinline__ void dx_read_ops(uint32_t pb, const uint32_t (&pa)[MT], uint4& b, uint4 (&a)[MT]) {
#if defined(__HIP_DEVICE_COMPILE__)
    static_assert(MT >= 1 && MT <= 4, "batched reads up to four channel tiles");
    if constexpr (MT == 1)
        asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %3\n\ts_waitcnt lgkmcnt(0)"
                     : "=&v"(b), "=&v"(a[0]) : "v"(pb), "v"(pa[0]) : "memory");
    else if constexpr (MT == 2)
        asm volatile("ds_read_b128 %0, %3\n\tds_read_b128 %1, %4\n\tds_read_b128 %2, %5\n\ts_waitcnt lgkmcnt(0)"
                     : "=&v"(b), "=&v"(a[0]), "=&v"(a[1]) : "v"(pb), "v"(pa[0]), "v"(pa[1]) : "memory");
    else if constexpr (MT == 3)
        asm volatile(
            "ds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\tds_read_b128 %2, %6\n\tds_read_b128 %3, %7\n\t"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(b), "=&v"(a[0]), "=&v"(a[1]), "=&v"(a[2]) : "v"(pb), "v"(pa[0]), "v"(pa[1]), "v"(pa[2])
            : "memory");
    else
        asm volatile(
            "ds_read_b128 %0, %5\n\tds_read_b128 %1, %6\n\tds_read_b128 %2, %7\n\tds_read_b128 %3, %8\n\t"
            "ds_read_b128 %4, %9\n\ts_waitcnt lgkmcnt(0)"
            : "=&v"(b), "=&v"(a[0]), "=&v"(a[1]), "=&v"(a[2]), "=&v"(a[3])
            : "v"(pb), "v"(pa[0]), "v"(pa[1]), "v"(pa[2]), "v"(pa[3])
            : "memory");
#else
    (void)pb;
    (void)pa;
    b = make_uint4(0u, 0u, 0u, 0u);
    for (int m = 0; m < MT; ++m) a[m] = b;
#endif
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }
// one dword LDS read, complete when the statement ends (as above)
__device__ __forceinline__ uint32_t dx_read_u32(uint32_t p) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t v;
    asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=&v"(v) : "v"(p) : "memory");
    return v;
#else
    (void)p;
    return 0u;
#endif
}
template <int KC>
__device__ __forceinline__ int dx_chunk(int r, int j) {
    return j ^ (r & (KC / 8 >= 16 ? 15 : 7));
}
template <int MT>
struct DxCfg {
    static constexpr int WI = (MT * 16 + 63) / 64;           // 64-row groups of staged WxT
    static constexpr int KC = MT <= 8 ? 128 : 64;
    static constexpr int SZ = DX_CELLS * KC, SW = 64 * WI * KC;  // staged elements per buffer
    static constexpr int ZI = SZ / 8 / 64 / NWV, WLI = SW / 8 / 64 / NWV;  // load instructions per wave and stage
    static_assert(SZ % (8 * 64 * NWV) == 0 && SW % (8 * 64 * NWV) == 0, "whole instructions on every wave");
};
}  // namespace

template <int MT>
__global__ void __launch_bounds__(64 * NWV)
k_dx_tr(int64_t n_cells, int C, int N, int64_t n_blocks, const bf16_t* __restrict__ dZ,
        const bf16_t* __restrict__ WxT, const uint8_t* __restrict__ flags, bf16_t* __restrict__ dX) {
    using Cf = DxCfg<MT>;
    constexpr int KC = Cf::KC, SZ = Cf::SZ, SW = Cf::SW, ZI = Cf::ZI, WLI = Cf::WLI;
    constexpr int RG = KC / 8;  // 16-byte chunks per staged row
    // two buffer sets, as separate arrays so that reads of one are not
    // ordered behind the direct loads into the other
    __shared__ __attribute__((aligned(16))) bf16_t szA[SZ], szB[SZ];
    __shared__ __attribute__((aligned(16))) bf16_t swA[SW], swB[SW];
    // per wave: the flag bytes of its sixteen cells in the first four dwords
    __shared__ __attribute__((aligned(16))) uint32_t sfA[NWV * 64], sfB[NWV * 64];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int nk = N / KC;

    // the lane's chunk of every stage: instruction j of the wave fills chunks
    // (wave + 4 j) * 64 + lane of the buffer
    int zrow[ZI], zoff[ZI], wrow[WLI], woff[WLI];
#pragma unroll
    for (int j = 0; j < ZI; ++j) {
        const int P = (wave + NWV * j) * 64 + lane, r = P / RG, pos = P - r * RG;
        zrow[j] = r;
        zoff[j] = 8 * dx_chunk<KC>(r, pos);
    }
#pragma unroll
    for (int j = 0; j < WLI; ++j) {
        const int P = (wave + NWV * j) * 64 + lane, r = P / RG, pos = P - r * RG;
        wrow[j] = min(r, C - 1);  // padded channels re-read the last one (results not stored)
        woff[j] = 8 * dx_chunk<KC>(r, pos);
    }
    auto issue = [&](int64_t blk, int kc, bf16_t* zb, bf16_t* wb, uint32_t* fb) __attribute__((always_inline)) {
        const int64_t cell0 = blk * DX_CELLS;
        const int k0 = kc * KC;
        // flags of the wave's cells, four per lane in lanes 0-3 (the array is
        // padded past the last cell; every stage loads them, so that every
        // stage has the same loads)
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(flags + cell0 + 16 * wave + 4 * min(lane, 3)),
                                         static_cast<void*>(fb + wave * 64), 4, 0, 0);
#pragma unroll
        for (int j = 0; j < ZI; ++j) {
            const int64_t cell = min(cell0 + zrow[j], n_cells - 1);
            __builtin_amdgcn_global_load_lds(static_cast<const void*>(dZ + cell * N + k0 + zoff[j]),
                                             static_cast<void*>(zb + (wave + NWV * j) * 512), 16, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < WLI; ++j)
            __builtin_amdgcn_global_load_lds(static_cast<const void*>(WxT + (int64_t)wrow[j] * N + k0 + woff[j]),
                                             static_cast<void*>(wb + (wave + NWV * j) * 512), 16, 0, 0);
    };
    floatx4 acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = floatx4{0.f, 0.f, 0.f, 0.f};

    int64_t blk = blockIdx.x;
    int kc = 0;
    // one stage from buffers (zb, wb), the next one's loads into (zn, wn);
    // false once the last stage is done
    auto stage = [&](const bf16_t* zb, const bf16_t* wb, const uint32_t* fb, bf16_t* zn, bf16_t* wn, uint32_t* fn)
                     __attribute__((always_inline)) {
        int64_t nblk = blk;
        int nkc = kc + 1;
        if (nkc == nk) {
            nkc = 0;
            nblk += gridDim.x;
        }
        if (nblk < n_blocks) {
            issue(nblk, nkc, zn, wn, fn);
            // the next stage's loads stay in flight (vmcnt: bits 3:0 and 15:14)
            constexpr int n = ZI + WLI + 1;
            static_assert(n < 64, "vmcnt range");
            __builtin_amdgcn_s_waitcnt(0x0f70 | (n & 15) | ((n >> 4) << 14));
        } else {
            __builtin_amdgcn_s_waitcnt(0x0f70);
        }
        dx_barrier();
        const int rz = 16 * wave + i16;
#pragma unroll 4
        for (int ks = 0; ks < KC / 32; ++ks) {
            if constexpr (MT <= 4) {
                uint32_t pa[MT];
                uint4 bo, ao[MT];
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const int r = 16 * m + i16;
                    pa[m] = lds_addr(&wb[r * KC + 8 * dx_chunk<KC>(r, 4 * ks + g)]);
                }
                dx_read_ops<MT>(lds_addr(&zb[rz * KC + 8 * dx_chunk<KC>(rz, 4 * ks + g)]), pa, bo, ao);
#pragma unroll
                for (int m = 0; m < MT; ++m) acc[m] = mfma_bf16(as_bf16x8(ao[m]), as_bf16x8(bo), acc[m]);
            } else {
                const bf16x8 bo =
                    as_bf16x8(*reinterpret_cast<const uint4*>(&zb[rz * KC + 8 * dx_chunk<KC>(rz, 4 * ks + g)]));
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const int r = 16 * m + i16;
                    const bf16x8 ao =
                        as_bf16x8(*reinterpret_cast<const uint4*>(&wb[r * KC + 8 * dx_chunk<KC>(r, 4 * ks + g)]));
                    acc[m] = mfma_bf16(ao, bo, acc[m]);
                }
            }
        }
        dx_barrier();  // every wave is done with these buffers before the next stage's issue refills them
        if (kc == nk - 1) {
            // lane (g, i16) holds channels 16 m + 4 g .. + 3 of cell 16 wave + i16;
            // the wave's sixteen flag bytes were staged with the stage's loads
            const int64_t cell = blk * DX_CELLS + 16 * wave + i16;
            const uint32_t fw = dx_read_u32(lds_addr(&fb[wave * 64 + (i16 >> 2)]));
            if (cell < n_cells) {
                const bool ok = (fw >> (8 * (i16 & 3))) & 1;
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const int ch = 16 * m + 4 * g;
                    if (ch < C) St<bf16_t>::st4(dX + cell * C + ch, ok ? acc[m] : floatx4{0.f, 0.f, 0.f, 0.f});
                }
            }
#pragma unroll
            for (int m = 0; m < MT; ++m) acc[m] = floatx4{0.f, 0.f, 0.f, 0.f};
        }
        blk = nblk;
        kc = nkc;
        return blk < n_blocks;
    };
    if (blk < n_blocks) {
        issue(blk, 0, szA, swA, sfA);
        while (stage(szA, swA, sfA, szB, swB, sfB) && stage(szB, swB, sfB, szA, swA, sfA)) {
        }
    }
}

// false when the stage length does not divide 20H (H = 32 with c_in up to
// 64): the caller takes k_dx_big
template <int MT>
static bool launch_dx_tr(const LayerGeom& g, const bf16_t* dz, const bf16_t* wxt, const uint8_t* flags, bf16_t* dx,
                         hipStream_t s) {
    using Cf = DxCfg<MT>;
    if ((20 * g.hidden) % Cf::KC != 0) return false;
    constexpr size_t lds = 2 * ((size_t)Cf::SZ + Cf::SW) * sizeof(bf16_t);
    static_assert(lds <= 160 * 1024, "LDS of a CU");
    const int64_t n_blocks = (g.n_cells + DX_CELLS - 1) / DX_CELLS;
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
        cus = 256;
        (void)hipGetLastError();  // not reported for the launch below
    }
    const int per_cu = (int)std::max<size_t>(1, (160 * 1024) / lds);
    const unsigned grid = (unsigned)std::max<int64_t>(1, std::min<int64_t>(n_blocks, (int64_t)per_cu * cus));
    hipLaunchKernelGGL(k_dx_tr<MT>, dim3(grid), dim3(64 * NWV), 0, s, g.n_cells, g.c_in, 20 * g.hidden, n_blocks, dz, wxt,
                       flags, dx);
    return true;
}

// --- dW --------------------------------------------------------------------------
constexpr int BW_KC = 32;         // cells per step
constexpr int BW_RB = 320;        // gate rows per workgroup
constexpr int BW_CB = 160;        // columns per workgroup
constexpr int BW_THREADS = 512;   // 8 waves: 4 along the rows x 2 along the columns, 80 x 80 each
constexpr int BW_TARGET = 256;    // workgroups aimed for (one per CU)

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
    const int64_t by_size = std::max<int64_t>(1, g.n_cells / (4 * BW_KC));  // at least 4 steps per chunk
    ch = std::max<int64_t>(1, std::min(ch, by_size));
    q.chunk_cells = (g.n_cells + ch - 1) / ch;
    q.chunk_cells = std::max<int64_t>(BW_KC, (q.chunk_cells + BW_KC - 1) / BW_KC * BW_KC);  // an empty canvas: one chunk
    q.chunks = (int)((g.n_cells + q.chunk_cells - 1) / q.chunk_cells);
    if (q.chunks < 1) q.chunks = 1;
    return q;
}

// Workgroup = (row block, column block) of one direction and one chunk of
// cells. The blocks of a (direction, chunk) read the same dZ rows and column
// operands, so they are placed on one XCD (workgroups are dealt to the XCDs
// in turn) to share its L2. Each step stages 32 cells of dZ and of the column
// operand in LDS transposed (cells contiguous; a thread writes the values of
// two adjacent cells together), so that an MFMA operand is one 16-byte LDS
// read; the loads of the next PD steps are in flight meanwhile. The bias
// gradient is summed from the staged dZ values in registers. Launched for
// fp32 storage (bf16 takes k_dw_tr below); the kernel itself handles both.
template <typename T, int PD>
__global__ void __launch_bounds__(BW_THREADS)
k_dw_big(int64_t n_cells, int canvas_w, int C, int H, BigDw q, const T* __restrict__ dZ, const T* __restrict__ X,
         const T* __restrict__ Y, const uint8_t* __restrict__ flags, float* __restrict__ part) {
    using B = BigT<T>;
    constexpr int E = B::E;
    constexpr int KC = BW_KC, PIT = KC + 8;
    constexpr int CA = BW_RB / E, CBK = BW_CB / E;  // 16-byte chunks per cell: dZ rows, columns
    constexpr int NP = KC / 2;                      // cell pairs per step
    constexpr int NITEM = (CA + CBK) * NP;          // staging items (chunk, cell pair)
    constexpr int NPASS = (NITEM + BW_THREADS - 1) / BW_THREADS;
    static_assert(BW_THREADS % NP == 0, "a thread keeps its cell pair in every pass");
    __shared__ __attribute__((aligned(16))) T sA[BW_RB][PIT];
    __shared__ __attribute__((aligned(16))) T sB[BW_CB][PIT];

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int wr = wave >> 1, wc = wave & 1;
    const int M = q.rblocks * q.cblocks, L = blockIdx.x;
    int gi, mem;
    if ((4 * q.chunks) % 8 == 0) {
        const int slot = L >> 3;
        gi = (slot / M) * 8 + (L & 7);
        mem = slot % M;
    } else {
        gi = L / M;
        mem = L % M;
    }
    const int rb = mem % q.rblocks, cb = mem / q.rblocks, d = gi & 3, chunk = gi >> 2;
    const int G = q.G, N = 20 * H;
    const int r0 = rb * BW_RB, c0 = cb * BW_CB;
    const int64_t k_begin = (int64_t)chunk * q.chunk_cells;
    const int64_t k_end = min(n_cells, k_begin + q.chunk_cells);
    const int lstep = (d & 1) ? 1 : -1;                              // left predecessor: cell + lstep
    const int64_t tstep = (d & 2) ? canvas_w : -(int64_t)canvas_w;  // top predecessor
    const uint8_t lbit = (d & 1) ? 4 : 2, tbit = (d & 2) ? 16 : 8;
    const int rlim = min(BW_RB, G - r0);  // rows of this block inside the direction
    const int p2 = 2 * (tid % NP);        // first cell of the thread's pair

    // Items of the thread, pass by pass: source 0 dZ, 1 X, 2 left Y, 3 top Y,
    // 4 zero columns, 5 idle; element offset in the source row; LDS row.
    int isrc[NPASS], ioff[NPASS], irow[NPASS];
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
        const int i = ps * BW_THREADS + tid;
        if (i < CA * NP) {
            const int rr = E * (i / NP);
            isrc[ps] = 0;
            ioff[ps] = d * G + r0 + min(rr, max(rlim - E, 0));
            irow[ps] = rr;
        } else if (i < NITEM) {
            const int kk = E * ((i - CA * NP) / NP), col = c0 + kk;
            irow[ps] = kk;
            if (col < C) { isrc[ps] = 1; ioff[ps] = col; }
            else if (col < C + H) { isrc[ps] = 2; ioff[ps] = d * H + col - C; }
            else if (col < C + 2 * H) { isrc[ps] = 3; ioff[ps] = d * H + col - C - H; }
            else { isrc[ps] = 4; ioff[ps] = 0; }
        } else {
            isrc[ps] = 5;
            ioff[ps] = 0;
            irow[ps] = 0;
        }
    }
    u32x4 va[PD][NPASS][2];
    uint32_t vf[PD][2];
    // Loads of the step at cell kb into register set k: the pair's flags and,
    // per pass, the item's 16-byte chunk of both cells (cells past the
    // chunk's end read its last cell and get flags 0).
    auto issue = [&](int64_t kb, int k) {
        int64_t pc[2], pl[2], pt[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int64_t p = kb + p2 + c;
            const bool in = p < k_end;
            pc[c] = in ? p : k_end - 1;
            vf[k][c] = in ? flags[pc[c]] : 0u;
            pl[c] = min(max(pc[c] + lstep, (int64_t)0), n_cells - 1);
            pt[c] = min(max(pc[c] + tstep, (int64_t)0), n_cells - 1);
        }
#pragma unroll
        for (int ps = 0; ps < NPASS; ++ps)
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const T* src = isrc[ps] == 0   ? dZ + pc[c] * N
                               : isrc[ps] == 2 ? Y + pl[c] * (4 * H)
                               : isrc[ps] == 3 ? Y + pt[c] * (4 * H)
                                               : X + pc[c] * C;
                va[k][ps][c] = *reinterpret_cast<const u32x4*>(src + ioff[ps]);
            }
    };
    // bias partial sums of the thread's dZ items (column block 0 only)
    float bsum[NPASS][E];
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps)
#pragma unroll
        for (int e = 0; e < E; ++e) bsum[ps][e] = 0.0f;
    const bool do_bias = cb == 0;
    auto commit = [&](int k) {
        bool ok[NPASS][2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const uint32_t f = vf[k][c];
            const bool v = f & 1, vl = f & lbit, vt = f & tbit;
#pragma unroll
            for (int ps = 0; ps < NPASS; ++ps)
                ok[ps][c] = v && ((isrc[ps] == 0 && irow[ps] < rlim) || isrc[ps] == 1 || (isrc[ps] == 2 && vl) ||
                                  (isrc[ps] == 3 && vt));
        }
#pragma unroll
        for (int ps = 0; ps < NPASS; ++ps) {
            if (isrc[ps] == 5) continue;
            const u32x4 a = ok[ps][0] ? va[k][ps][0] : zero4();
            const u32x4 b = ok[ps][1] ? va[k][ps][1] : zero4();
            T* dst = isrc[ps] == 0 ? &sA[irow[ps]][p2] : &sB[irow[ps]][p2];
            if constexpr (std::is_same<T, float>::value) {
#pragma unroll
                for (int e = 0; e < E; ++e)
                    *reinterpret_cast<uint2*>(dst + e * PIT) = make_uint2(a[e], b[e]);
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const uint32_t lo = (e & 1) ? a[e >> 1] >> 16 : a[e >> 1] & 0xffffu;
                    const uint32_t hi = (e & 1) ? b[e >> 1] & 0xffff0000u : b[e >> 1] << 16;
                    *reinterpret_cast<uint32_t*>(dst + e * PIT) = lo | hi;
                }
            }
            if (do_bias && isrc[ps] == 0) {
                const T* ae = reinterpret_cast<const T*>(&a);
                const T* be = reinterpret_cast<const T*>(&b);
#pragma unroll
                for (int e = 0; e < E; ++e) bsum[ps][e] += St<T>::ld1(ae + e) + St<T>::ld1(be + e);
            }
        }
    };

    floatx4 acc[5][5];
#pragma unroll
    for (int m = 0; m < 5; ++m)
#pragma unroll
        for (int n = 0; n < 5; ++n) acc[m][n] = floatx4{0.f, 0.f, 0.f, 0.f};

    auto step = [&](int64_t kb, int k) {
        commit(k);
        lds_barrier();
        issue(kb + PD * KC, k);  // past the chunk's end the loads re-read its last cell (flags 0)
        // MFMA: lane (g, i16) reads row 80 wr + 16 m + i16 of sA and column
        // 80 wc + 16 n + i16 of sB at cells KS s + E g .. + E - 1
        constexpr int KS = B::KSTEP;
#pragma unroll
        for (int s = 0; s < KC / KS; ++s) {
            u32x4 a[5], b[5];
#pragma unroll
            for (int m = 0; m < 5; ++m)
                a[m] = *reinterpret_cast<const u32x4*>(&sA[80 * wr + 16 * m + i16][KS * s + E * g]);
#pragma unroll
            for (int n = 0; n < 5; ++n)
                b[n] = *reinterpret_cast<const u32x4*>(&sB[80 * wc + 16 * n + i16][KS * s + E * g]);
#pragma unroll
            for (int m = 0; m < 5; ++m)
#pragma unroll
                for (int n = 0; n < 5; ++n) acc[m][n] = mma16<T>(a[m], b[n], acc[m][n]);
        }
        lds_barrier();
    };
    if (k_begin < k_end) {
#pragma unroll
        for (int k = 0; k < PD; ++k) issue(k_begin + k * KC, k);
    }
    for (int64_t kb = k_begin; kb < k_end; kb += PD * KC) {
        step(kb, 0);
        if constexpr (PD == 2) {
            if (kb + KC >= k_end) break;
            step(kb + KC, 1);
        }
    }

    // partial [chunk][d][G][PP]: columns then the bias; lane (g, i16) holds rows 4 g + r of tile (m, n)
    float* out = part + ((int64_t)chunk * 4 + d) * (int64_t)G * q.PP;
#pragma unroll
    for (int m = 0; m < 5; ++m)
#pragma unroll
        for (int n = 0; n < 5; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = r0 + 80 * wr + 16 * m + 4 * g + r, col = c0 + 80 * wc + 16 * n + i16;
                if (row < G && col < q.NB) out[(int64_t)row * q.PP + col] = acc[m][n][r];
            }
    if (do_bias) {
        // the NP threads of an item's chunk are NP consecutive lanes
#pragma unroll
        for (int ps = 0; ps < NPASS; ++ps)
#pragma unroll
            for (int e = 0; e < E; ++e)
#pragma unroll
                for (int o = 1; o < NP; o <<= 1) bsum[ps][e] += __shfl_xor(bsum[ps][e], o);
#pragma unroll
        for (int ps = 0; ps < NPASS; ++ps) {
            if (isrc[ps] != 0 || tid % NP != 0) continue;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int rr = irow[ps] + e;
                if (rr < rlim) out[(int64_t)(r0 + rr) * q.PP + q.NB] = bsum[ps][e];
            }
        }
    }
}

// --- dW, bf16: direct-to-LDS staging and transposed LDS reads ------------------
// The same blocks, chunks, partial layout and XCD placement as k_dw_big, for
// bf16 storage. Each step's 32 cells of dZ rows [r0, r0 + 320) and of the
// column operand [c0, c0 + 160) are copied by direct global-to-LDS loads
// (no registers, no VALU work per element) in the cell-major layout they have
// in memory, two steps ahead into a ring of three buffers. The MFMA operands,
// which hold eight consecutive cells of one row, come from the LDS transpose
// read (ds_read_b64_tr_b16: within each sixteen lanes, lane 4 j + i/4 reads
// four consecutive values at its address and lane i receives value i % 4 of
// the reads of lanes i/4, 4 + i/4, 8 + i/4, 12 + i/4), two reads per
// operand. The 16-byte chunks of a staged row are permuted (chunk j of cell k
// at j ^ s(k)) so that the sixteen rows one transpose read touches fall on
// distinct banks. Invalid cells get their dZ row zeroed once staged, and
// predecessors outside the cell's rectangle or masked their part of the
// column operand; the bias gradient is one more MFMA per gate-row tile with a
// column of ones.
namespace {
constexpr int TR_KC = 32;                      // cells per step
constexpr int TR_AG = BW_RB / 8, TR_BG = BW_CB / 8;  // 16-byte chunks per staged row: dZ, columns
constexpr int TR_AI = TR_KC * TR_AG / 64;      // wave load instructions per step: dZ
constexpr int TR_BI = TR_KC * TR_BG / 64;      //   columns
constexpr int TR_SLOTS = 4;                    // load instructions per wave and step (the last one of the
                                               // workgroup loads the flags, into a spare slot)
constexpr int TR_NBUF = 3;
static_assert(TR_AI + TR_BI + 1 <= 8 * TR_SLOTS && TR_AI + TR_BI + 1 > 8 * (TR_SLOTS - 1), "slot count");
static_assert(TR_AG % 8 == 0 && TR_BG % 4 == 0, "chunk permutation groups");

__device__ __forceinline__ int tr_sa(int k) { return 2 * (((k >> 1) & 1) | ((k >> 2) & 2)); }  // within 8 chunks
__device__ __forceinline__ int tr_sb(int k) { return 2 * ((k >> 3) & 1); }                  // within 4 chunks

typedef short tr_s4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 tr_read(const bf16_t* p) {
    const tr_s4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) tr_s4*)(p));
    uint2 r;
    __builtin_memcpy(&r, &v, 8);
    return r;
}
__device__ __forceinline__ bf16x8 tr_pair(uint2 lo, uint2 hi) { return as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)); }
// LDS-only barrier: no fence, so pending direct-to-LDS loads into other
// buffers are not waited for
__device__ __forceinline__ void tr_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
}  // namespace

__global__ void __launch_bounds__(BW_THREADS)
k_dw_tr(int64_t n_cells, int canvas_w, int C, int H, BigDw q, const bf16_t* __restrict__ dZ,
        const bf16_t* __restrict__ X, const bf16_t* __restrict__ Y, const uint8_t* __restrict__ flags,
        float* __restrict__ part) {
    __shared__ __attribute__((aligned(16))) bf16_t sA[TR_NBUF][TR_KC * BW_RB];
    __shared__ __attribute__((aligned(16))) bf16_t sB[TR_NBUF][TR_KC * BW_CB];
    __shared__ __attribute__((aligned(16))) uint32_t sF[TR_NBUF][64];
    __shared__ __attribute__((aligned(16))) uint32_t sink[256];

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int wr = wave >> 1, wc = wave & 1;
    const int M = q.rblocks * q.cblocks, L = blockIdx.x;
    int gi, mem;
    if ((4 * q.chunks) % 8 == 0) {
        const int slot = L >> 3;
        gi = (slot / M) * 8 + (L & 7);
        mem = slot % M;
    } else {
        gi = L / M;
        mem = L % M;
    }
    const int rb = mem % q.rblocks, cb = mem / q.rblocks, d = gi & 3, chunk = gi >> 2;
    const int G = q.G, N = 20 * H;
    const int r0 = rb * BW_RB, c0 = cb * BW_CB;
    const int64_t k_begin = (int64_t)chunk * q.chunk_cells;
    const int64_t k_end = min(n_cells, k_begin + q.chunk_cells);
    const int lstep = (d & 1) ? 1 : -1;
    const int64_t tstep = (d & 2) ? canvas_w : -(int64_t)canvas_w;
    const uint32_t lbit = (d & 1) ? 4 : 2, tbit = (d & 2) ? 16 : 8;
    const int64_t nsteps = (k_end - k_begin + TR_KC - 1) / TR_KC;
    const int64_t kb_last = k_begin + max(nsteps - 1, (int64_t)0) * TR_KC;  // the last step's first cell

    // The lane's part of every step's loads, slot by slot: the source row
    // base, the bytes per cell of that source, the cell shift (the left or top
    // predecessor for the column operand's Y parts), the cell within the step,
    // the byte offset within the source row and the LDS destination of the
    // wave instruction. Slots 0 .. TR_AI - 1 load dZ, the next TR_BI the
    // column operand (X, left Y, top Y by lane), then one loads the flags of
    // the step's cells and the spare one repeats it into a sink.
    const char* kbase[TR_SLOTS];
    int kstride[TR_SLOTS], kshift[TR_SLOTS], kcell[TR_SLOTS], koff[TR_SLOTS];
    char* kdst[TR_SLOTS];
#pragma unroll
    for (int j = 0; j < TR_SLOTS; ++j) {
        const int sl = wave * TR_SLOTS + j;
        kshift[j] = 0;
        if (sl < TR_AI) {
            const int P = sl * 64 + lane, k = P / TR_AG, pos = P - k * TR_AG, ch = pos ^ tr_sa(k);
            kbase[j] = reinterpret_cast<const char*>(dZ);
            kstride[j] = 2 * N;
            kcell[j] = k;
            koff[j] = 2 * (d * G + min(r0 + 8 * ch, G - 8));  // rows past the direction's end: any valid row
            kdst[j] = reinterpret_cast<char*>(&sA[0][sl * 512]);
        } else if (sl < TR_AI + TR_BI) {
            const int P = (sl - TR_AI) * 64 + lane, k = P / TR_BG, pos = P - k * TR_BG, ch = pos ^ tr_sb(k);
            const int col = c0 + 8 * ch;
            kcell[j] = k;
            kdst[j] = reinterpret_cast<char*>(&sB[0][(sl - TR_AI) * 512]);
            if (col < C || col >= C + 2 * H) {  // X; columns past the end: any valid chunk
                kbase[j] = reinterpret_cast<const char*>(X);
                kstride[j] = 2 * C;
                koff[j] = col < C ? 2 * col : 0;
            } else {
                const bool left = col < C + H;
                kbase[j] = reinterpret_cast<const char*>(Y);
                kstride[j] = 8 * H;
                kshift[j] = left ? lstep : (int)tstep;
                koff[j] = 2 * (d * H + col - C - (left ? 0 : H));
            }
        } else {
            kbase[j] = reinterpret_cast<const char*>(flags);
            kstride[j] = 1;
            kcell[j] = sl == TR_AI + TR_BI ? 4 * min(lane, 7) : 0;  // flags of cells 4 l .. 4 l + 3
            koff[j] = 0;
            kdst[j] = sl == TR_AI + TR_BI ? reinterpret_cast<char*>(&sF[0][0]) : reinterpret_cast<char*>(&sink[0]);
        }
    }
    constexpr int ABUF = TR_KC * BW_RB * 2, BBUF = TR_KC * BW_CB * 2, FBUF = 64 * 4;  // bytes per buffer
    // loads of the step at cell kb into buffer b; cells past the chunk's end
    // re-read its last cell (their flags read as invalid below); predecessors
    // off the canvas read its first or last cell (masked by the flags)
    auto issue = [&](int64_t kb, int b) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < TR_SLOTS; ++j) {
            const int sl = wave * TR_SLOTS + j;
            if (sl < TR_AI + TR_BI) {
                const int64_t cell = min(kb + kcell[j], k_end - 1);
                const int64_t src = min(max(cell + kshift[j], (int64_t)0), n_cells - 1);
                __builtin_amdgcn_global_load_lds(kbase[j] + src * kstride[j] + koff[j],
                                                 kdst[j] + b * (sl < TR_AI ? ABUF : BBUF), 16, 0, 0);
            } else {
                // the flags array is padded past the last cell, so the four
                // bytes at any cell of a step are readable; steps past the
                // chunk's end re-read the last step's
                __builtin_amdgcn_global_load_lds(kbase[j] + min(kb, kb_last) + kcell[j],
                                                 kdst[j] + (sl == TR_AI + TR_BI ? b * FBUF : 0), 4, 0, 0);
            }
        }
    };

    floatx4 acc[5][5], accb[5];
#pragma unroll
    for (int m = 0; m < 5; ++m) {
        accb[m] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int n = 0; n < 5; ++n) acc[m][n] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    // bias: waves of column block 0 and wave column 0, B = a column of ones
    const bool do_bias = cb == 0 && wc == 0;
    const bf16x8 ones = as_bf16x8(i16 == 0 ? make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u)
                                           : make_uint4(0u, 0u, 0u, 0u));
    // transposed-read addresses (elements within a buffer) of the lane: row
    // (cell) 8 g + 4 h + (i16 >> 2), chunk of its sixteen rows or columns,
    // half (i16 & 1) of the chunk
    int aoff[2][5], boff[2][5];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int k = 8 * g + 4 * h + (i16 >> 2);
#pragma unroll
        for (int m = 0; m < 5; ++m) {
            const int ca = (80 * wr + 16 * m) / 8 + ((i16 & 3) >> 1);
            aoff[h][m] = k * BW_RB + 8 * (ca ^ tr_sa(k)) + 4 * (i16 & 1);
            const int cbk = (80 * wc + 16 * m) / 8 + ((i16 & 3) >> 1);
            boff[h][m] = k * BW_CB + 8 * (cbk ^ tr_sb(k)) + 4 * (i16 & 1);
        }
    }
    // the vmcnt immediate: one step's loads of a wave stay in flight
    constexpr int VM_ONE_STEP = 0x0f70 | TR_SLOTS;

    if (nsteps > 0) {
        issue(k_begin, 0);
        issue(k_begin + TR_KC, 1);
    }
    for (int64_t st = 0; st < nsteps; ++st) {
        const int b = (int)(st % TR_NBUF);
        const int64_t kb = k_begin + st * TR_KC;
        __builtin_amdgcn_s_waitcnt(VM_ONE_STEP);  // this wave's loads of step st have landed
        tr_barrier();
        // validity: zero the dZ rows of invalid cells (and of cells past the
        // chunk's end), and the predecessor columns a valid cell must not see
        {
            const int k = tid >> 4, sub = tid & 15;
            const uint32_t f = kb + k < k_end ? (sF[b][k >> 2] >> (8 * (k & 3))) & 0xffu : 0u;
            const uint4 z = make_uint4(0u, 0u, 0u, 0u);
            if (!(f & 1)) {
#pragma unroll
                for (int c = sub; c < TR_AG; c += 16) *reinterpret_cast<uint4*>(&sA[b][k * BW_RB + 8 * c]) = z;
            } else if (!(f & lbit) || !(f & tbit)) {
#pragma unroll
                for (int c = sub; c < TR_BG; c += 16) {
                    const int col = c0 + 8 * (c ^ tr_sb(k));
                    const bool hl = col >= C && col < C + H, ht = col >= C + H && col < C + 2 * H;
                    if ((hl && !(f & lbit)) || (ht && !(f & tbit)))
                        *reinterpret_cast<uint4*>(&sB[b][k * BW_CB + 8 * c]) = z;
                }
            }
        }
        tr_barrier();
        issue(kb + 2 * TR_KC, (int)((st + 2) % TR_NBUF));  // past the end: re-reads the last cell, never used
        const bf16_t* A = sA[b];
        const bf16_t* Bm = sB[b];
        bf16x8 bop[5];
#pragma unroll
        for (int n = 0; n < 5; ++n) bop[n] = tr_pair(tr_read(Bm + boff[0][n]), tr_read(Bm + boff[1][n]));
#pragma unroll
        for (int m = 0; m < 5; ++m) {
            const bf16x8 aop = tr_pair(tr_read(A + aoff[0][m]), tr_read(A + aoff[1][m]));
#pragma unroll
            for (int n = 0; n < 5; ++n) acc[m][n] = mfma_bf16(aop, bop[n], acc[m][n]);
            if (do_bias) accb[m] = mfma_bf16(aop, ones, accb[m]);
        }
    }
    __builtin_amdgcn_s_waitcnt(0x0f70);  // the loads issued past the last step

    // partial [chunk][d][G][PP]: columns then the bias; lane (g, i16) holds
    // rows 4 g + r of tile (m, n)
    float* out = part + ((int64_t)chunk * 4 + d) * (int64_t)G * q.PP;
#pragma unroll
    for (int m = 0; m < 5; ++m) {
#pragma unroll
        for (int n = 0; n < 5; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = r0 + 80 * wr + 16 * m + 4 * g + r, col = c0 + 80 * wc + 16 * n + i16;
                if (row < G && col < q.NB) out[(int64_t)row * q.PP + col] = acc[m][n][r];
            }
        if (do_bias && i16 == 0) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = r0 + 80 * wr + 16 * m + 4 * g + r;
                if (row < G) out[(int64_t)row * q.PP + q.NB] = accb[m][r];
            }
        }
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
// the flags, padded past the last cell: the bf16 input-gradient kernel loads
// the flags of a whole block of DX_CELLS cells from the block's first cell
// (last block: up to n_cells - 1 + DX_CELLS), the bf16 weight-gradient
// kernel those of TR_KC cells from any step's first cell
static_assert(DX_CELLS >= TR_KC, "flag padding covers both kernels");
size_t big_flags_bytes(const LayerGeom& g) { return (size_t)(g.n_cells > 0 ? g.n_cells : 1) + DX_CELLS; }
size_t big_wxt_bytes(const LayerGeom& g) {
    return (size_t)g.c_in * 20 * g.hidden * (g.dtype == 0 ? 4 : 2);
}
size_t big_partial_bytes(const LayerGeom& g) {
    const BigDw q = big_dw(g);
    return (size_t)q.chunks * 4 * q.G * q.PP * sizeof(float);
}

hipError_t launch_bwd_big_dx(const LayerGeom& g, const void* d_dz, const void* d_wx, const uint8_t* d_mask,
                             const int32_t* d_rid, void* d_dx, uint8_t* d_flags, void* d_wxt, hipStream_t s) {
    if (g.n_cells == 0) return hipSuccess;
    const int N = 20 * g.hidden;
    int fb = (int)std::min<int64_t>((g.n_cells + 255) / 256, 4096);
    hipLaunchKernelGGL(k_cell_flags, dim3(fb), dim3(256), 0, s, g.canvas_h, g.canvas_w, d_mask, d_rid, d_flags);
    const int64_t nw = (int64_t)N * g.c_in;
    const int tb = (int)std::min<int64_t>((nw + 255) / 256, 4096);
    // 64-cell waves while they fill the CUs four times over, else workgroups
    // of 16 cells with the reduction split over their waves
    const int64_t cgroups = (g.c_in + 63) / 64, waves64 = (g.n_cells + 63) / 64 * cgroups;
    const bool split = waves64 < 4 * 256;
    const dim3 gx((unsigned)(split ? (g.n_cells + 15) / 16 : ((g.n_cells + 63) / 64 + 3) / 4), (unsigned)cgroups);
    auto dx_big = [&](auto tag, const auto* dz, const auto* wxt, auto* dx) {
        using T = decltype(tag);
        if (split)
            hipLaunchKernelGGL((k_dx_big<T, true>), gx, dim3(256), 0, s, g.n_cells, g.c_in, N, dz, wxt, d_flags, dx);
        else
            hipLaunchKernelGGL((k_dx_big<T, false>), gx, dim3(256), 0, s, g.n_cells, g.c_in, N, dz, wxt, d_flags,
                               dx);
    };
    if (g.dtype == 0) {
        using T = float;
        hipLaunchKernelGGL(k_transpose<T>, dim3(tb), dim3(256), 0, s, N, g.c_in, static_cast<const T*>(d_wx),
                           static_cast<T*>(d_wxt));
        dx_big(T{}, static_cast<const T*>(d_dz), static_cast<const T*>(d_wxt), static_cast<T*>(d_dx));
    } else {
        using T = bf16_t;
        hipLaunchKernelGGL(k_transpose<T>, dim3(tb), dim3(256), 0, s, N, g.c_in, static_cast<const T*>(d_wx),
                           static_cast<T*>(d_wxt));
        const T* dz = static_cast<const T*>(d_dz);
        const T* wxt = static_cast<const T*>(d_wxt);
        T* dx = static_cast<T*>(d_dx);
        bool done = false;
        switch ((g.c_in + 15) / 16) {  // channel tiles (c_in is a multiple of 8, at most 256)
#define MDL_DX_TR(mt) \
    case mt: done = launch_dx_tr<mt>(g, dz, wxt, d_flags, dx, s); break;
            MDL_DX_TR(1) MDL_DX_TR(2) MDL_DX_TR(3) MDL_DX_TR(4) MDL_DX_TR(5) MDL_DX_TR(6) MDL_DX_TR(7) MDL_DX_TR(8)
            MDL_DX_TR(9) MDL_DX_TR(10) MDL_DX_TR(11) MDL_DX_TR(12) MDL_DX_TR(13) MDL_DX_TR(14) MDL_DX_TR(15)
            MDL_DX_TR(16)
#undef MDL_DX_TR
            default: return hipErrorInvalidValue;
        }
        if (!done)
            dx_big(T{}, dz, wxt, dx);
    }
    return hipGetLastError();
}

hipError_t launch_bwd_big_dw(const LayerGeom& g, const void* d_dz, const void* d_x, const void* d_y,
                             const uint8_t* d_flags, float* d_part, float* d_dwx, float* d_du, float* d_db,
                             hipStream_t s) {
    if (g.n_cells == 0) return hipSuccess;
    const BigDw q = big_dw(g);
    const dim3 gw((unsigned)(q.rblocks * q.cblocks * 4 * q.chunks));
    const int64_t total = (int64_t)4 * q.G * q.PP;
    const int rbk = (int)std::min<int64_t>((total + 255) / 256, 4096);
    if (g.dtype == 0) {
        using T = float;
        constexpr int PD = 1;
        hipLaunchKernelGGL((k_dw_big<T, PD>), gw, dim3(BW_THREADS), 0, s, g.n_cells, g.canvas_w, g.c_in, g.hidden, q,
                           static_cast<const T*>(d_dz), static_cast<const T*>(d_x), static_cast<const T*>(d_y),
                           d_flags, d_part);
    } else {
        hipLaunchKernelGGL(k_dw_tr, gw, dim3(BW_THREADS), 0, s, g.n_cells, g.canvas_w, g.c_in, g.hidden, q,
                           static_cast<const bf16_t*>(d_dz), static_cast<const bf16_t*>(d_x),
                           static_cast<const bf16_t*>(d_y), d_flags, d_part);
    }
    hipLaunchKernelGGL(k_dw_big_reduce, dim3(rbk), dim3(256), 0, s, g.c_in, g.hidden, q, d_part, d_dwx, d_du, d_db);
    return hipGetLastError();
}

}  // namespace mdl
