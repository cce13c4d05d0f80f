// Input and weight gradients from dZ in one pass over the canvas, staged
// through LDS strip by strip.
//
// A strip is TC consecutive cells of one canvas row. For each strip the
// workgroup loads, with independent coalesced loads, dZ [TC][20H], X
// [TC][C_in], the layer output Y of the strip's row (one cell of halo on each
// side) and of the rows above and below, and the rectangle ids and mask bytes
// of the same halo block, from which a validity byte per cell follows (cell
// valid; left/right/up/down neighbour in the same rectangle and unmasked).
// Cells outside every rectangle or masked, and predecessors outside the
// cell's rectangle or masked, are zeroed in LDS once staged, so the MFMA
// loops below read plain operands. Then, from LDS:
//   dW_d[r][col] += sum_cells dZ[cell][d*5H + r] * B_d[cell][col],
//     B_d = [X | h_L,d | h_T,d]  (the layer output shifted one cell in
//     direction d's frame: the shifted recurrent operand of Appendix A)
//   db_d[r] += sum_cells dZ[cell][d*5H + r]
//   dX[cell] = sum_d dZ_d[cell] Wx_d
// Wave w of the workgroup owns direction d = w / WPD and a slice of the gate
// rows; the dW tiles (MFMA) and bias sums (VALU) stay in its registers across
// all strips of the workgroup, and are written once as the workgroup's
// partial. A fixed-order reduction over workgroups gives deterministic weight
// gradients.
//
// The loads of the next strip are issued into registers before the current
// strip is computed, so their latency is hidden behind the MFMA work; the
// workgroup's barriers order LDS only and leave them in flight.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

namespace {

template <int H, int C>
struct StripCfg {
    static constexpr int G = 5 * H, N = 20 * H;
    static constexpr int RT = (G + 15) / 16;          // gate-row tiles per direction
    static constexpr int NB = C + 2 * H;              // dW columns (the bias is summed apart)
    static constexpr int CT = (NB + 15) / 16;         // dW column tiles
    static constexpr int PP = CT * 16 + 4;            // partial row pitch; column CT*16 holds the bias
    static constexpr bool ALIGNED = C % 16 == 0 && H % 16 == 0;  // column tiles never straddle X / h_L / h_T
    static constexpr int CXT = (C + 15) / 16;         // dX channel tiles
    static constexpr int WPD = H >= 32 ? 2 : 1;       // waves per direction
    static constexpr int RTW = (RT + WPD - 1) / WPD;  // gate-row tiles per wave
    // cells per strip: 16 where the registers need it (H >= 32) or where two
    // workgroups then fit on a CU (H = 16), else 32
    static constexpr int TC = H >= 16 ? 16 : 32;
    static constexpr int THREADS = 256 * WPD;
    static constexpr int ZP = N + 4;                  // LDS pitch of dZ rows (4 mod 16: the cells read by one MFMA hit distinct banks)
    static constexpr int YP = 4 * H + 4;              // LDS pitch of Y rows
    static constexpr int XP = CXT * 16 + 4;           // LDS pitch of X rows and dX partials
    static constexpr int SY = 3 * (TC + 2) * YP, SDX = 4 * TC * XP;
    static constexpr int HW = TC + 2;                 // halo block width
    // The next strip's loads are prefetched into registers where the dW tiles
    // leave room (H <= 16). With 32-cell strips at H = 16 that takes over 256
    // registers per lane (one workgroup per CU); the 16-cell strips of H = 16
    // (dW steps unrolled by two with 8 input channels) and the other shapes
    // run two workgroups per CU.
    static constexpr bool PREFETCH = H <= 16;
    // workgroups launched: one round of resident workgroups (H = 32 holds
    // one per CU: its registers, and LDS in the direct-to-LDS kernel)
    static constexpr int WGS = (H == 16 && TC == 32) || H >= 32 ? 256 : 512;
    // register budget of the H = 32 shapes: dW steps unrolled by two, dX
    // operands read five blocks at a time
    static constexpr int DW_UNROLL = H >= 32 || (H == 16 && C < 16) ? 2 : TC / 4;
    static constexpr int DXB = H >= 32 ? 5 : (G + 15) / 16;
};

// 4 consecutive elements of storage type T as fp32.
template <typename T>
struct V4;
template <>
struct V4<float> {
    using R = float4;
    static __device__ __forceinline__ R load(const float* p) { return *reinterpret_cast<const float4*>(p); }
    // non-temporal load, for data read once (keeps the re-read Y rows cached)
    static __device__ __forceinline__ R ldnt(const float* p) {
        const floatx4 v = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(p));
        return make_float4(v[0], v[1], v[2], v[3]);
    }
    static __device__ __forceinline__ float4 f(R v) { return v; }
    static __device__ __forceinline__ void store(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
};
template <>
struct V4<bf16_t> {
    using R = uint2;
    static __device__ __forceinline__ R load(const bf16_t* p) { return *reinterpret_cast<const uint2*>(p); }
    static __device__ __forceinline__ R ldnt(const bf16_t* p) {
        const uint64_t v = __builtin_nontemporal_load(reinterpret_cast<const uint64_t*>(p));
        return make_uint2((uint32_t)v, (uint32_t)(v >> 32));
    }
    static __device__ __forceinline__ float4 f(R v) {
        return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u), __uint_as_float(v.y << 16),
                           __uint_as_float(v.y & 0xffff0000u));
    }
    static __device__ __forceinline__ void store(bf16_t* p, float4 v) {
        *reinterpret_cast<uint2*>(p) = make_uint2(f2bf2(v.x, v.y), f2bf2(v.z, v.w));
    }
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
k_bwd_strip(int canvas_h, int canvas_w, int segs, int ngroups, int list_pitch, const int32_t* lists,
            const T* __restrict__ dZ, const T* __restrict__ X, const T* __restrict__ Y, const T* __restrict__ Wx,
            const uint8_t* __restrict__ mask, const int32_t* __restrict__ rid, T* __restrict__ dX,
            float* __restrict__ part) {
    using Cf = StripCfg<H, C>;
    using L4 = V4<T>;
    constexpr int TC = Cf::TC, RTW = Cf::RTW, WPD = Cf::WPD, CT = Cf::CT, CXT = Cf::CXT, HW = Cf::HW;
    constexpr int N = Cf::N, G = Cf::G, ZP = Cf::ZP, YP = Cf::YP, XP = Cf::XP, NTH = Cf::THREADS;
    __shared__ __attribute__((aligned(16))) float sz[TC * ZP + 16];
    __shared__ __attribute__((aligned(16))) float sx[TC][XP];
    // Y rows above, same (with one cell of halo each side), below; later the
    // per-direction dX partials
    __shared__ __attribute__((aligned(16))) float sy_raw[Cf::SY > Cf::SDX ? Cf::SY : Cf::SDX];
    __shared__ int32_t srid[3][HW];
    __shared__ uint32_t smask[3][HW];
    auto sy = reinterpret_cast<float(*)[HW][YP]>(sy_raw);
    auto sdx = reinterpret_cast<float(*)[TC][XP]>(sy_raw);

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, i16 = lane & 15;
    const int d = wave / WPD, rslice = wave % WPD;
    const int rt0 = rslice * RTW;

    // The dZ row padding and the 16 floats after the last row are read
    // (times zero weights) where 5H is not a multiple of 16; they stay zero.
    for (int e = tid; e < TC * (ZP - N) + 16; e += NTH) {
        const int c = e / (ZP - N);
        sz[c < TC ? c * ZP + N + (e - c * (ZP - N)) : TC * ZP + (e - TC * (ZP - N))] = 0.0f;
    }

    floatx4 acc[RTW][CT];
#pragma unroll
    for (int a = 0; a < RTW; ++a)
#pragma unroll
        for (int b = 0; b < CT; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};
    // bias sums: the dW A operands summed per lane (its cell slots), the four
    // slots added across lanes at the end
    float dbp[RTW];
#pragma unroll
    for (int a = 0; a < RTW; ++a) dbp[a] = 0.0f;

    // dX: wave (d, rslice) owns channel tiles ct = rslice, rslice + WPD, ...;
    // M = channels, N = cells, K = the direction's gate rows in blocks of 16:
    // in MFMA j of block m, K slot g is gate row 16 m + 4 g + j, so that a
    // lane reads its four rows of a block as one 16-byte LDS load. The A
    // operand Wx_d^T stays in registers.
    constexpr int CXW = (CXT + WPD - 1) / WPD, KBL = (G + 15) / 16;
    float wa[CXW][KBL][4];
#pragma unroll
    for (int cc = 0; cc < CXW; ++cc) {
        const int ch = (rslice + cc * WPD) * 16 + i16;
#pragma unroll
        for (int m = 0; m < KBL; ++m)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * m + 4 * g + j;
                wa[cc][m][j] = (ch < C && r < G) ? to_f<T>(Wx[((int64_t)d * G + r) * C + ch]) : 0.0f;
            }
    }

    // --- loads of one strip into registers. Every lane issues the same
    // number of loads from valid addresses (slots past the end repeat the last
    // element, cells past the row's end repeat its last cell, halo cells
    // outside the canvas re-read the nearest cell and are marked invalid when
    // staged), so the waits for them are exact.
    constexpr int NZ = TC * N / 4, PZ = (NZ + NTH - 1) / NTH;
    constexpr int NYR = HW * H, NY = 3 * NYR, PY = (NY + NTH - 1) / NTH;
    constexpr int NX = TC * C / 4, PX = (NX + NTH - 1) / NTH;
    constexpr int NHALO = 3 * HW, PH = (NHALO + NTH - 1) / NTH;
    typename L4::R vz[PZ], vy[PY], vx[PX];
    int32_t vr[PH];
    uint32_t vm[PH];
    auto strip_pos = [&](int strip, int& cy, int& cx0, int& len, int64_t& p0) {
        cy = strip / segs;
        cx0 = (strip - cy * segs) * TC;
        len = min(TC, canvas_w - cx0);
        p0 = (int64_t)cy * canvas_w + cx0;
    };
    // part bits: 1 dZ, 2 Y, 4 X, 8 ids and mask bytes
    auto issue = [&](int strip, int parts) {
        int cy, cx0, len;
        int64_t p0;
        strip_pos(strip, cy, cx0, len, p0);
#pragma unroll
        for (int k = 0; k < PZ * (parts & 1); ++k) {
            const int e = min(tid + k * NTH, NZ - 1);
            const int c = (4 * e) / N, n = 4 * e - c * N;
            vz[k] = L4::ldnt(dZ + (p0 + min(c, len - 1)) * N + n);
        }
#pragma unroll
        for (int k = 0; k < PY * ((parts >> 1) & 1); ++k) {
            const int e = min(tid + k * NTH, NY - 1);
            const int row = e / NYR, rem = e - row * NYR;
            const int c = rem / H, k4 = rem - c * H;
            const int yy = min(max(cy + row - 1, 0), canvas_h - 1), xx = min(max(cx0 + c - 1, 0), canvas_w - 1);
            vy[k] = L4::load(Y + ((int64_t)yy * canvas_w + xx) * (4 * H) + 4 * k4);
        }
#pragma unroll
        for (int k = 0; k < PX * ((parts >> 2) & 1); ++k) {
            const int e = min(tid + k * NTH, NX - 1);
            const int c = e / (C / 4), k4 = e - c * (C / 4);
            vx[k] = L4::load(X + (p0 + min(c, len - 1)) * C + 4 * k4);
        }
#pragma unroll
        for (int k = 0; k < PH * ((parts >> 3) & 1); ++k) {
            const int e = min(tid + k * NTH, NHALO - 1);
            const int row = e / HW, c = e - row * HW;
            const int yy = min(max(cy + row - 1, 0), canvas_h - 1), xx = min(max(cx0 + c - 1, 0), canvas_w - 1);
            const int64_t p = (int64_t)yy * canvas_w + xx;
            vr[k] = rid[p];
            vm[k] = mask[p];
        }
    };
    // registers -> LDS; slots past the end store the last element again
    auto commit = [&](int strip, int parts) {
        int cy, cx0, len;
        int64_t p0;
        strip_pos(strip, cy, cx0, len, p0);
#pragma unroll
        for (int k = 0; k < PZ * (parts & 1); ++k) {
            const int e = min(tid + k * NTH, NZ - 1);
            const int c = (4 * e) / N, n = 4 * e - c * N;
            st_f4(&sz[c * ZP + n], L4::f(vz[k]));
        }
#pragma unroll
        for (int k = 0; k < PY * ((parts >> 1) & 1); ++k) {
            const int e = min(tid + k * NTH, NY - 1);
            const int row = e / NYR, rem = e - row * NYR;
            const int c = rem / H, k4 = rem - c * H;
            st_f4(&sy[row][c][4 * k4], L4::f(vy[k]));
        }
#pragma unroll
        for (int k = 0; k < PX * ((parts >> 2) & 1); ++k) {
            const int e = min(tid + k * NTH, NX - 1);
            const int c = e / (C / 4), k4 = e - c * (C / 4);
            st_f4(&sx[c][4 * k4], L4::f(vx[k]));
        }
#pragma unroll
        for (int k = 0; k < PH * ((parts >> 3) & 1); ++k) {
            const int e = min(tid + k * NTH, NHALO - 1);
            const int row = e / HW, c = e - row * HW;
            const int yy = cy + row - 1, xx = cx0 + c - 1;
            const bool inside = yy >= 0 && yy < canvas_h && xx >= 0 && xx < canvas_w;
            srid[row][c] = inside ? vr[k] : -2;  // -2 matches no rectangle id
            smask[row][c] = inside ? vm[k] : 0u;
        }
    };

    // With the prefetch the next strip's loads occupy registers during the
    // compute; shapes whose dW tiles fill the register file load each strip
    // just before staging it, one tensor at a time.
    constexpr bool PREFETCH = Cf::PREFETCH;
    // The strips with a valid cell of this workgroup's group, as in the
    // direct-to-LDS kernel below (the others were skipped, their dX rows
    // zeroed with the strip flags). An entry is loaded two strips ahead, before
    // the next strip's loads, so that it has landed when those are waited for.
    const int wg = (int)blockIdx.x, grp = wg % ngroups, gi = wg / ngroups, gn = (int)gridDim.x / ngroups;
    const int32_t* list = lists + (int64_t)grp * list_pitch;
    auto ld = [&](int64_t k) { return __hip_atomic_load(list + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); };
    auto uni = [](int v) { return __builtin_amdgcn_readfirstlane(v); };
    const int n_live = uni(ld(0));
    const int n_my = n_live > gi ? (n_live - gi + gn - 1) / gn : 0;
    auto entry_raw = [&](int k) { return ld(1 + gi + (int64_t)(k - 1) * gn); };  // k = 1 .. n_my
    int strip = n_my > 0 ? uni(entry_raw(1)) : -1;
    int next_raw = n_my > 1 ? entry_raw(2) : -1;
    if constexpr (PREFETCH) {
        if (strip >= 0) issue(strip, 15);
    }
    for (int kpos = 1; strip >= 0; ++kpos) {
        int cy, cx0, len;
        int64_t p0;
        strip_pos(strip, cy, cx0, len, p0);
        if constexpr (PREFETCH) {
            commit(strip, 15);
        } else {
#pragma unroll
            for (int part = 1; part < 16; part <<= 1) {
                issue(strip, part);
                commit(strip, part);
            }
        }
        lds_barrier();
        // Validity, folded into the staged data: the dZ and X rows of an
        // invalid cell (outside every rectangle, masked, or past the row's
        // end) and every predecessor output that is not in the cell's
        // rectangle or is masked become zero. Each predecessor segment (row,
        // halo cell, direction) has one consumer cell.
        // Lanes 0..TC-1 of every wave find the invalid cells (same ballot in every wave).
        bool cv = false;
        if (lane < TC) {
            const int r = srid[1][lane + 1];
            cv = lane < len && smask[1][lane + 1] && r >= 0;
        }
        const uint64_t valid = __ballot(cv);
        const uint64_t bad = ~valid & ((TC == 64) ? ~0ull : ((1ull << TC) - 1));
        for (uint64_t bm = bad; bm; bm &= bm - 1) {  // uniform loop over the invalid cells
            const int c = __builtin_ctzll(bm);
            for (int e = tid; e < N / 4; e += NTH) st_f4(&sz[c * ZP + 4 * e], make_float4(0.f, 0.f, 0.f, 0.f));
            if (tid < C / 4) st_f4(&sx[c][4 * tid], make_float4(0.f, 0.f, 0.f, 0.f));
        }
        for (int e = tid; e < 8 * TC; e += NTH) {
            // e = (direction, left or top, consumer cell)
            const int c = e % TC, lt = (e / TC) & 1, dd = e / (2 * TC);
            const int row = lt ? ((dd & 2) ? 2 : 0) : 1;
            const int k = lt ? c + 1 : ((dd & 1) ? c + 2 : c);
            const int r = srid[1][c + 1];
            if (!(srid[row][k] == r && smask[row][k])) {
#pragma unroll
                for (int j = 0; j < H; j += 4) st_f4(&sy[row][k][dd * H + j], make_float4(0.f, 0.f, 0.f, 0.f));
            }
        }
        // the next strip's loads (the last strip re-reads itself) stay in flight
        const int next = uni(next_raw);
        next_raw = kpos + 2 <= n_my ? entry_raw(kpos + 2) : -1;
        if constexpr (PREFETCH) issue(next >= 0 ? next : strip, 15);
        lds_barrier();

        // --- dW: K = cells of the strip, 4 per MFMA step; in step ks, K slot g
        // is cell 16 (ks / 4) + 4 g + ks % 4 (the four slots of a step hit
        // distinct LDS banks)
#pragma unroll Cf::DW_UNROLL
        for (int ks = 0; ks < TC / 4; ++ks) {
            const int c = 16 * (ks >> 2) + 4 * g + (ks & 3);
            const int lc = (d & 1) ? c + 2 : c;  // left predecessor in the halo-shifted same row
            const int trow = (d & 2) ? 2 : 0;    // row of the top predecessor
            float av[RTW], bv[CT];
#pragma unroll
            for (int a = 0; a < RTW; ++a) {
                const int r = (rt0 + a) * 16 + i16;
                const float z = sz[c * ZP + d * G + r];  // in bounds for r < RT * 16
                av[a] = r < G ? z : 0.0f;
            }
#pragma unroll
            for (int b = 0; b < CT; ++b) {
                float x;
                if constexpr (Cf::ALIGNED) {
                    // tile b lies in one of X, h_L, h_T
                    if (b < C / 16) x = sx[c][b * 16 + i16];
                    else if (b < (C + H) / 16) x = sy[1][lc][d * H + (b - C / 16) * 16 + i16];
                    else x = sy[trow][c + 1][d * H + (b - (C + H) / 16) * 16 + i16];
                } else {
                    const int col = b * 16 + i16;
                    x = 0.0f;
                    if (col < C) x = sx[c][col];
                    else if (col < C + H) x = sy[1][lc][d * H + col - C];
                    else if (col < C + 2 * H) x = sy[trow][c + 1][d * H + col - C - H];
                }
                bv[b] = x;
            }
#pragma unroll
            for (int a = 0; a < RTW; ++a) {
                dbp[a] += av[a];
#pragma unroll
                for (int b = 0; b < CT; ++b) acc[a][b] = mfma_f32(av[a], bv[b], acc[a][b]);
            }
        }

        // --- dX partial of direction d
        floatx4 axs[CXW][TC / 16];
#pragma unroll
        for (int cc = 0; cc < CXW; ++cc) {
#pragma unroll
            for (int nt = 0; nt < TC / 16; ++nt) {
                floatx4 ax = floatx4{0.f, 0.f, 0.f, 0.f};
                const int cell = nt * 16 + i16;
                if ((rslice + cc * WPD) < CXT) {
                    // operands in groups of DXB blocks: one LDS round trip per group
                    constexpr int DXB = Cf::DXB;
#pragma unroll
                    for (int m0 = 0; m0 < KBL; m0 += DXB) {
                        float4 bz[DXB];
#pragma unroll
                        for (int m = 0; m < DXB; ++m)
                            if (m0 + m < KBL)
                                bz[m] = *reinterpret_cast<const float4*>(&sz[cell * ZP + d * G + 16 * (m0 + m) + 4 * g]);
#pragma unroll
                        for (int m = 0; m < DXB; ++m) {
                            if (m0 + m < KBL) {
                                ax = mfma_f32(wa[cc][m0 + m][0], bz[m].x, ax);
                                ax = mfma_f32(wa[cc][m0 + m][1], bz[m].y, ax);
                                ax = mfma_f32(wa[cc][m0 + m][2], bz[m].z, ax);
                                ax = mfma_f32(wa[cc][m0 + m][3], bz[m].w, ax);
                            }
                        }
                    }
                }
                axs[cc][nt] = ax;
            }
        }
        lds_barrier();  // every wave is done reading the staged Y rows
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
        lds_barrier();
        // sum the four directions in a fixed order (0 at invalid cells, whose
        // dZ rows are zero). Every lane stores 4 channels of one cell in every
        // pass (cells past the row's end and slots past the last repeat the
        // row's last cell).
        {
            constexpr int NXS = TC * C / 4, PXS = (NXS + NTH - 1) / NTH;
#pragma unroll
            for (int k = 0; k < PXS; ++k) {
                const int e = min(tid + k * NTH, NXS - 1);
                const int c = min(e / (C / 4), len - 1), k4 = 4 * (e - (e / (C / 4)) * (C / 4));
                const float4 a0 = *reinterpret_cast<const float4*>(&sdx[0][c][k4]);
                const float4 a1 = *reinterpret_cast<const float4*>(&sdx[1][c][k4]);
                const float4 a2 = *reinterpret_cast<const float4*>(&sdx[2][c][k4]);
                const float4 a3 = *reinterpret_cast<const float4*>(&sdx[3][c][k4]);
                L4::store(dX + (p0 + c) * C + k4,
                          make_float4(((a0.x + a1.x) + a2.x) + a3.x, ((a0.y + a1.y) + a2.y) + a3.y,
                                      ((a0.z + a1.z) + a2.z) + a3.z, ((a0.w + a1.w) + a2.w) + a3.w));
            }
        }
        lds_barrier();
        strip = next;
    }

    // partial of this workgroup: [wg][4][RT*16][PP], bias in column CT*16
    float* out = part + ((int64_t)blockIdx.x * 4 + d) * (Cf::RT * 16) * Cf::PP;
#pragma unroll
    for (int a = 0; a < RTW; ++a) {
        if (rt0 + a >= Cf::RT) continue;
#pragma unroll
        for (int b = 0; b < CT; ++b)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                out[(int64_t)((rt0 + a) * 16 + 4 * g + r) * Cf::PP + b * 16 + i16] = acc[a][b][r];
    }
#pragma unroll
    for (int a = 0; a < RTW; ++a) {
        // lanes i16, i16 + 16, i16 + 32, i16 + 48 hold the four cell slots of row (rt0 + a) * 16 + i16
        float sb = dbp[a];
        sb += __shfl_xor(sb, 16);
        sb += __shfl_xor(sb, 32);
        if (g == 0 && rt0 + a < Cf::RT) out[(int64_t)((rt0 + a) * 16 + i16) * Cf::PP + CT * 16] = sb;
    }
}

// ---------------------------------------------------------------------------
// fp32 storage at H = 32: the same computation, with every strip's dZ, X and
// Y block copied by direct global-to-LDS loads (no registers) into one of two
// buffer sets, the next strip's copy in flight while the current one is
// computed. The accumulators of the dW tiles fill the register file at this
// width, so staging through registers leaves no room to load ahead.
//
// LDS layouts (floats): dZ [TC][20H] with its 16-byte chunks permuted within
// each aligned group of sixteen by the cell index (chunk j of cell c sits at
// j ^ (c & 15)), so that the dX operand reads of sixteen cells hit distinct
// banks; Y [3][TC + 2][4H] (rows above, same, below; one halo cell each
// side); X [TC][C_in]; the validity ids (rectangle id of a valid cell, -1
// for an invalid one, computed once per call) of the halo, [3][TC + 2]. A
// wave's load instruction fills 1 KB of LDS (256 bytes for the ids), lane l
// slot l, so each lane fetches the element its slot holds.
// ---------------------------------------------------------------------------
template <int H, int C>
struct DmaCfg {
    static constexpr int TC = 16, HW = TC + 2, N = 20 * H, G = 5 * H;
    static constexpr int NW = 8, THREADS = 64 * NW;
    static constexpr int ZCH = TC * N / 4, YCH = 3 * HW * H, XCH = TC * C / 4;  // 16-byte chunks per strip
    static constexpr int ZI = ZCH / 64, YI = YCH / 64, XI = XCH / 64;           // wave load instructions
    static_assert(ZCH % 64 == 0 && YCH % 64 == 0 && XCH % 64 == 0, "whole 1 KB load instructions");
    static_assert((N / 4) % 16 == 0, "dZ rows hold whole chunk groups of sixteen");
    static_assert(H == 32 && C % 16 == 0, "laid out for H = 32");
};

__device__ __forceinline__ int zswz(int cell, int f) {  // LDS float index of dZ element f of a strip cell
    return (((f >> 2) ^ (cell & 15)) << 2) | (f & 3);
}

template <int H, int C>
__global__ void __launch_bounds__((DmaCfg<H, C>::THREADS))
k_bwd_strip_dma(int canvas_h, int canvas_w, int segs, int ngroups, int list_pitch, const int32_t* lists,
                const float* __restrict__ dZ, const float* __restrict__ X, const float* __restrict__ Y,
                const float* __restrict__ Wx, const int32_t* __restrict__ vid, float* __restrict__ dX,
                float* __restrict__ part) {
    using Cf = StripCfg<H, C>;
    using Dc = DmaCfg<H, C>;
    constexpr int TC = Dc::TC, HW = Dc::HW, N = Dc::N, G = Dc::G, NW = Dc::NW, NTH = Dc::THREADS;
    constexpr int RTW = Cf::RTW, WPD = Cf::WPD, CT = Cf::CT, CXT = Cf::CXT, XP = Cf::XP;
    static_assert(TC == Cf::TC && NTH == Cf::THREADS, "same strips and waves as the staged kernel");
    __shared__ __attribute__((aligned(16))) float zA[TC * N], zB[TC * N];
    __shared__ __attribute__((aligned(16))) float yA[3 * HW * 4 * H], yB[3 * HW * 4 * H];
    __shared__ __attribute__((aligned(16))) float xA[TC * C], xB[TC * C];
    __shared__ __attribute__((aligned(16))) int32_t vA[64], vB[64];
    // the four directions' dX partials of a strip, summed at the next strip's
    // first barrier (so a strip needs two barriers)
    __shared__ __attribute__((aligned(16))) float sdx[4][TC][XP];
    static_assert(3 * HW <= 64, "the halo's ids fill one 256-byte load instruction");

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
    float dbp[RTW];
#pragma unroll
    for (int a = 0; a < RTW; ++a) dbp[a] = 0.0f;
    // dX A operand Wx_d^T in registers, as in the staged kernel
    constexpr int CXW = (CXT + WPD - 1) / WPD, KBL = G / 16;
    float wa[CXW][KBL][4];
#pragma unroll
    for (int cc = 0; cc < CXW; ++cc) {
        const int ch = (rslice + cc * WPD) * 16 + i16;
#pragma unroll
        for (int m = 0; m < KBL; ++m)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                wa[cc][m][j] = ch < C ? Wx[((int64_t)d * G + 16 * m + 4 * g + j) * C + ch] : 0.0f;
    }
    // with the operand loads complete here, the waits the compiler places in
    // the strip loop need not cover them (which would make the dX products
    // wait for the next strip's copies as well)
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)

    auto strip_pos = [&](int strip, int& cy, int& cx0, int& len, int64_t& p0) {
        cy = strip / segs;
        cx0 = (strip - cy * segs) * TC;
        len = min(TC, canvas_w - cx0);
        p0 = (int64_t)cy * canvas_w + cx0;
    };
    // direct loads of a strip into one buffer set; every lane reads a valid
    // address (cells past the row's end repeat its last cell, halo cells
    // outside the canvas the nearest one; both are marked invalid once staged)
    auto copy_in = [&](int strip, float* zb, float* yb, float* xb, int32_t* vb) __attribute__((always_inline)) {
        int cy, cx0, len;
        int64_t p0;
        strip_pos(strip, cy, cx0, len, p0);
        for (int q = wave; q < Dc::ZI; q += NW) {
            const int s = q * 64 + lane, cell = s / (N / 4), pos = s - cell * (N / 4);
            const float* src = dZ + (p0 + min(cell, len - 1)) * N + 4 * (pos ^ (cell & 15));
            __builtin_amdgcn_global_load_lds(src, zb + q * 256, 16, 0, 0);
        }
        for (int q = wave; q < Dc::YI; q += NW) {
            const int s = q * 64 + lane, row = s / (HW * H), rem = s - row * (HW * H);
            const int c = rem / H, k = rem - c * H;
            const int yy = min(max(cy + row - 1, 0), canvas_h - 1), xx = min(max(cx0 + c - 1, 0), canvas_w - 1);
            __builtin_amdgcn_global_load_lds(Y + ((int64_t)yy * canvas_w + xx) * (4 * H) + 4 * k, yb + q * 256, 16,
                                             0, 0);
        }
        for (int q = wave; q < Dc::XI; q += NW) {
            const int s = q * 64 + lane, cell = s / (C / 4), k = s - cell * (C / 4);
            __builtin_amdgcn_global_load_lds(X + (p0 + min(cell, len - 1)) * C + 4 * k, xb + q * 256, 16, 0, 0);
        }
        if (wave == NW - 1) {
            const int e = min(lane, 3 * HW - 1), row = e / HW, c = e - row * HW;
            const int yy = min(max(cy + row - 1, 0), canvas_h - 1), xx = min(max(cx0 + c - 1, 0), canvas_w - 1);
            __builtin_amdgcn_global_load_lds(vid + (int64_t)yy * canvas_w + xx, vb, 4, 0, 0);
        }
    };

    // dX of a strip: the sum of its four direction partials, in a fixed order
    auto dx_sum = [&](int strip) __attribute__((always_inline)) {
        int cy, cx0, len;
        int64_t p0;
        strip_pos(strip, cy, cx0, len, p0);
        constexpr int NXS = TC * C / 4, PXS = (NXS + NTH - 1) / NTH;
#pragma unroll
        for (int k = 0; k < PXS; ++k) {
            const int e = min(tid + k * NTH, NXS - 1);
            const int c = min(e / (C / 4), len - 1), k4 = 4 * (e - (e / (C / 4)) * (C / 4));
            const float4 a0 = *reinterpret_cast<const float4*>(&sdx[0][c][k4]);
            const float4 a1 = *reinterpret_cast<const float4*>(&sdx[1][c][k4]);
            const float4 a2 = *reinterpret_cast<const float4*>(&sdx[2][c][k4]);
            const float4 a3 = *reinterpret_cast<const float4*>(&sdx[3][c][k4]);
            *reinterpret_cast<float4*>(dX + (p0 + c) * C + k4) =
                make_float4(((a0.x + a1.x) + a2.x) + a3.x, ((a0.y + a1.y) + a2.y) + a3.y,
                            ((a0.z + a1.z) + a2.z) + a3.z, ((a0.w + a1.w) + a2.w) + a3.w);
        }
    };

    // The strips with a valid cell of this workgroup's group (the strips
    // whose column segment is the group's modulo ngroups; workgroups are
    // dealt to the XCDs in turn, so a group's strips, which share halo rows
    // from one row to the next, stay in one L2), after their count (the
    // others hold no valid cell: their dX rows were zeroed with the ids).
    // The group's workgroups take every (gridDim.x / ngroups)-th of them.
    // Entries are read one strip ahead with vector loads, and made uniform
    // only after the next strip's wait (a read right after the load would
    // wait for the copies issued before it).
    const int wg = (int)blockIdx.x, grp = wg % ngroups, gi = wg / ngroups, gn = (int)gridDim.x / ngroups;
    const int32_t* list = lists + (int64_t)grp * list_pitch;
    auto ld = [&](int64_t k) { return __hip_atomic_load(list + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); };
    auto uni = [](int v) { return __builtin_amdgcn_readfirstlane(v); };
    const int n_live = uni(ld(0));
    const int n_my = n_live > gi ? (n_live - gi + gn - 1) / gn : 0;
    auto entry_raw = [&](int k) { return ld(1 + gi + (int64_t)(k - 1) * gn); };  // k = 1 .. n_my

    // strip: the strip to compute (its copies in zb, yb, xb, vb); next_raw:
    // the loaded entry of the strip whose copies start here into the other
    // buffers (-1: none), returned uniform in next; prev: the strip before,
    // whose dX partials are summed here; ahead: the list position read here
    // (the strip after next), its raw entry returned in after_next
    auto process = [&](int strip, int next_raw, int& next, int prev, int ahead, int& after_next, float* zb,
                       float* yb, float* xb, int32_t* vb, float* zn, float* yn, float* xn,
                       int32_t* vn) __attribute__((always_inline)) {
        int cy, cx0, len;
        int64_t p0;
        strip_pos(strip, cy, cx0, len, p0);
        __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's copies into zb, yb, xb, vb have landed
        lds_barrier();  // also: every wave's dX partials of the previous strip are in sdx
        if (prev >= 0) dx_sum(prev);  // before the next barrier, after which this strip's partials overwrite sdx
        // validity folded into the staged data (as in the staged kernel): a
        // cell is valid with a nonnegative id, a predecessor counts when it is
        // on the canvas and has the cell's id
        auto inside = [&](int row, int k) {
            const int yy = cy + row - 1, xx = cx0 + k - 1;
            return yy >= 0 && yy < canvas_h && xx >= 0 && xx < canvas_w;
        };
        bool cv = false;
        if (lane < TC) cv = lane < len && vb[HW + lane + 1] >= 0;
        const uint64_t good = __ballot(cv);  // the same in every wave
        const uint64_t bad = ~good & ((1ull << TC) - 1);
        for (uint64_t bm = bad; bm; bm &= bm - 1) {
            const int c = __builtin_ctzll(bm);
            for (int e = tid; e < N / 4; e += NTH) st_f4(&zb[c * N + 4 * e], make_float4(0.f, 0.f, 0.f, 0.f));
            if (tid < C / 4) st_f4(&xb[c * C + 4 * tid], make_float4(0.f, 0.f, 0.f, 0.f));
        }
        for (int e = tid; e < 8 * TC; e += NTH) {
            const int c = e % TC, lt = (e / TC) & 1, dd = e / (2 * TC);
            const int row = lt ? ((dd & 2) ? 2 : 0) : 1;
            const int k = lt ? c + 1 : ((dd & 1) ? c + 2 : c);
            if (!(inside(row, k) && vb[row * HW + k] == vb[HW + c + 1])) {
#pragma unroll
                for (int j = 0; j < H; j += 4)
                    st_f4(&yb[(row * HW + k) * (4 * H) + dd * H + j], make_float4(0.f, 0.f, 0.f, 0.f));
            }
        }
        lds_barrier();
        next = uni(next_raw);
        if (next >= 0) copy_in(next, zn, yn, xn, vn);  // the other buffers: free since the last barrier
        after_next = ahead <= n_my ? entry_raw(ahead) : -1;  // waited for with the next strip's copies

        // dW (K = the strip's cells, four per MFMA step, slot g = cell 16 (ks / 4) + 4 g + ks % 4);
        // a strip without a valid cell (separator rows, row slack) adds
        // nothing and its dX is zero
#pragma unroll 2
        for (int ks = 0; ks < (good ? TC / 4 : 0); ++ks) {
            const int c = 16 * (ks >> 2) + 4 * g + (ks & 3);
            const int lc = (d & 1) ? c + 2 : c;
            const int trow = (d & 2) ? 2 : 0;
            float av[RTW], bv[CT];
#pragma unroll
            for (int a = 0; a < RTW; ++a) av[a] = zb[c * N + zswz(c, d * G + (rt0 + a) * 16 + i16)];
#pragma unroll
            for (int b = 0; b < CT; ++b) {
                if (b < C / 16) bv[b] = xb[c * C + b * 16 + i16];
                else if (b < (C + H) / 16) bv[b] = yb[(HW + lc) * (4 * H) + d * H + (b - C / 16) * 16 + i16];
                else bv[b] = yb[(trow * HW + c + 1) * (4 * H) + d * H + (b - (C + H) / 16) * 16 + i16];
            }
#pragma unroll
            for (int a = 0; a < RTW; ++a) {
                dbp[a] += av[a];
#pragma unroll
                for (int b = 0; b < CT; ++b) acc[a][b] = mfma_f32(av[a], bv[b], acc[a][b]);
            }
        }
        // dX partial of direction d
        floatx4 axs[CXW];
#pragma unroll
        for (int cc = 0; cc < CXW; ++cc) {
            floatx4 ax = floatx4{0.f, 0.f, 0.f, 0.f};
            if (good && rslice + cc * WPD < CXT) {
                constexpr int DXB = 5;
#pragma unroll
                for (int m0 = 0; m0 < KBL; m0 += DXB) {
                    float4 bz[DXB];
#pragma unroll
                    for (int m = 0; m < DXB; ++m)
                        if (m0 + m < KBL)
                            bz[m] = *reinterpret_cast<const float4*>(
                                &zb[i16 * N + zswz(i16, d * G + 16 * (m0 + m) + 4 * g)]);
#pragma unroll
                    for (int m = 0; m < DXB; ++m) {
                        if (m0 + m < KBL) {
                            ax = mfma_f32(wa[cc][m0 + m][0], bz[m].x, ax);
                            ax = mfma_f32(wa[cc][m0 + m][1], bz[m].y, ax);
                            ax = mfma_f32(wa[cc][m0 + m][2], bz[m].z, ax);
                            ax = mfma_f32(wa[cc][m0 + m][3], bz[m].w, ax);
                        }
                    }
                }
            }
            axs[cc] = ax;
        }
        // every wave read the previous strip's partials before the second
        // barrier above
#pragma unroll
        for (int cc = 0; cc < CXW; ++cc) {
            const int ct = rslice + cc * WPD;
            if (ct < CXT) {
#pragma unroll
                for (int r = 0; r < 4; ++r) sdx[d][i16][ct * 16 + 4 * g + r] = axs[cc][r];
            }
        }
    };

    // list position k + 1 holds the k-th strip
    int strip = n_my > 0 ? uni(entry_raw(1)) : -1, next_raw = n_my > 1 ? entry_raw(2) : -1, prev = -1, k = 0;
    if (strip >= 0) copy_in(strip, zA, yA, xA, vA);
    while (strip >= 0) {
        int next = -1, an = -1;
        process(strip, next_raw, next, prev, k + 3, an, zA, yA, xA, vA, zB, yB, xB, vB);
        prev = strip;
        strip = next;
        next_raw = an;
        ++k;
        if (strip < 0) break;
        process(strip, next_raw, next, prev, k + 3, an, zB, yB, xB, vB, zA, yA, xA, vA);
        prev = strip;
        strip = next;
        next_raw = an;
        ++k;
    }
    if (prev >= 0) {
        lds_barrier();
        dx_sum(prev);
    }

    float* out = part + ((int64_t)blockIdx.x * 4 + d) * (Cf::RT * 16) * Cf::PP;
#pragma unroll
    for (int a = 0; a < RTW; ++a) {
        if (rt0 + a >= Cf::RT) continue;
#pragma unroll
        for (int b = 0; b < CT; ++b)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                out[(int64_t)((rt0 + a) * 16 + 4 * g + r) * Cf::PP + b * 16 + i16] = acc[a][b][r];
    }
#pragma unroll
    for (int a = 0; a < RTW; ++a) {
        float sb = dbp[a];
        sb += __shfl_xor(sb, 16);
        sb += __shfl_xor(sb, 32);
        if (g == 0 && rt0 + a < Cf::RT) out[(int64_t)((rt0 + a) * 16 + i16) * Cf::PP + CT * 16] = sb;
    }
}

// Fixed-order sum over workgroup partials. A block takes 64 consecutive
// outputs; its four thread groups sum every fourth workgroup each (loads
// batched), and the four sums are added in a fixed order.
__global__ void __launch_bounds__(256)
k_strip_reduce(int C, int H, int RT, int PP, int CT, int nwg, const float* __restrict__ part,
               float* __restrict__ dwx, float* __restrict__ du, float* __restrict__ db) {
    __shared__ float ps[4][64];
    const int G = 5 * H, NB = C + 2 * H + 1;  // columns: X, h_L, h_T, bias
    const int total = 4 * G * NB;
    const int oi = blockIdx.x * 64 + (threadIdx.x & 63), grp = threadIdx.x >> 6;
    const int64_t stride = (int64_t)4 * (RT * 16) * PP;
    float s = 0.0f;
    int d = 0, r = 0, col = 0;
    if (oi < total) {
        d = oi / (G * NB);
        const int rem = oi - d * G * NB;
        r = rem / NB;
        col = rem - r * NB;
        const int pc = col < NB - 1 ? col : CT * 16;
        const float* src = part + (int64_t)d * (RT * 16) * PP + (int64_t)r * PP + pc;
        int w = grp;
        for (; w + 28 < nwg; w += 32) {
            float v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = src[(int64_t)(w + 4 * k) * stride];
#pragma unroll
            for (int k = 0; k < 8; ++k) s += v[k];
        }
        for (; w < nwg; w += 4) s += src[(int64_t)w * stride];
    }
    ps[grp][threadIdx.x & 63] = s;
    __syncthreads();
    if (grp == 0 && oi < total) {
        const int t = threadIdx.x;
        const float v = ((ps[0][t] + ps[1][t]) + ps[2][t]) + ps[3][t];
        if (col < C) dwx[((int64_t)d * G + r) * C + col] = v;
        else if (col < C + 2 * H) du[((int64_t)d * G + r) * (2 * H) + (col - C)] = v;
        else db[(int64_t)d * G + r] = v;
    }
}

// Instantiated (storage, H, c_in) shapes; other shapes use the two-kernel path.
#define MDL_STRIP_SHAPES(X) \
    X(float, 4, 4) X(float, 4, 8) X(float, 8, 8) X(float, 16, 8) X(float, 16, 16) X(float, 32, 16) \
    X(float, 32, 32) X(bf16_t, 32, 16) X(bf16_t, 32, 32)

static int strip_tc(const LayerGeom& g) {
    int tc = 0;
#define MDL_STRIP_TC(T, H, C) \
    if (!tc && (g.dtype == 1) == std::is_same<T, bf16_t>::value && g.hidden == H && g.c_in == C) tc = StripCfg<H, C>::TC;
    MDL_STRIP_SHAPES(MDL_STRIP_TC)
#undef MDL_STRIP_TC
    return tc > 0 ? tc : 32;
}

bool strip_supported(const LayerGeom& g) {
#define MDL_STRIP_MATCH(T, H, C) \
    if ((g.dtype == 1) == std::is_same<T, bf16_t>::value && g.hidden == H && g.c_in == C) return true;
    MDL_STRIP_SHAPES(MDL_STRIP_MATCH)
#undef MDL_STRIP_MATCH
    return false;
}

static int strip_wgs(const LayerGeom& g) {
    const int tc = strip_tc(g);
    const int64_t strips = (int64_t)g.canvas_h * ((g.canvas_w + tc - 1) / tc);
    int wgs = 0;
#define MDL_STRIP_WGS(T, H, C) \
    if (!wgs && (g.dtype == 1) == std::is_same<T, bf16_t>::value && g.hidden == H && g.c_in == C) wgs = StripCfg<H, C>::WGS;
    MDL_STRIP_SHAPES(MDL_STRIP_WGS)
#undef MDL_STRIP_WGS
    return (int)std::max<int64_t>(1, std::min<int64_t>(wgs, strips));
}

// strip groups of the direct-to-LDS kernel: one per XCD (workgroups are dealt
// to the eight XCDs in turn) when the workgroups and column segments split
// evenly, else one
constexpr int STRIP_GROUPS_MAX = 8;
static int strip_groups(int nwg, int segs) { return (nwg % 8 == 0 && segs >= 8) ? 8 : 1; }
// int32 entries per group list: its count, then at most every strip of the
// largest group (ceil(segs / ng) segments of every row)
static int64_t strip_list_pitch(int canvas_h, int segs, int ng) { return (int64_t)canvas_h * ((segs + ng - 1) / ng) + 1; }

static int strip_pp(const LayerGeom& g) { return (g.c_in + 2 * g.hidden + 15) / 16 * 16 + 4; }

size_t strip_partial_bytes(const LayerGeom& g) {
    const int RT = (5 * g.hidden + 15) / 16;
    return (size_t)strip_wgs(g) * 4 * RT * 16 * strip_pp(g) * sizeof(float);
}

// Validity id of every canvas cell (its rectangle id where the cell is inside
// a rectangle and unmasked, else -1; written where vid is given), a thread per
// (strip of TC cells, cell), plus a byte
// per strip that says whether it holds a valid cell; the dX rows of the
// strips without one are zeroed here (the strip kernel skips them).
template <int TC, typename T>
__global__ void k_valid_ids_strips(int canvas_h, int canvas_w, int segs, int C, const uint8_t* __restrict__ mask,
                                   const int32_t* __restrict__ rid, int32_t* __restrict__ vid,
                                   uint8_t* __restrict__ live, T* __restrict__ dX) {
    static_assert(64 % TC == 0, "strips within a wave");
    const int64_t n_strips = (int64_t)canvas_h * segs;
    const int64_t total = (n_strips * TC + 63) / 64 * 64;  // whole waves: every lane takes part in the ballot
    const int lane = threadIdx.x & 63;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t strip = i / TC;
        const int j = (int)(i - strip * TC);
        const int cy = (int)(strip / segs), x = (int)(strip - (int64_t)cy * segs) * TC + j;
        const bool in = strip < n_strips && x < canvas_w;
        const int64_t p = (int64_t)cy * canvas_w + x;
        int32_t v = -1;
        if (in) {
            v = (mask[p] && rid[p] >= 0) ? rid[p] : -1;
            if (vid) vid[p] = v;
        }
        const uint64_t b = __ballot(v >= 0);
        const bool any = ((b >> (lane & ~(TC - 1))) & ((1ull << TC) - 1)) != 0;
        if (in && j == 0) live[strip] = any ? 1 : 0;
        if (strip < n_strips && !any) {  // the strip's dX rows, contiguous: lane j takes every TC-th 16 bytes
            const int len = min(TC, canvas_w - (x - j));
            uint4* row = reinterpret_cast<uint4*>(dX + (p - j) * C);
            const int n16 = len * C * (int)sizeof(T) / 16;
            for (int e = j; e < n16; e += TC) row[e] = make_uint4(0u, 0u, 0u, 0u);
        }
    }
}

// Per group of strips (column segment modulo ngroups; row-major within a
// group), the list of its strips with a valid cell in that order: a count per
// chunk of STRIP_CHUNKS equal chunks of the group's strips (one wave each),
// then each chunk writes its strips after the counts of the chunks before it;
// entry 0 of a group's list is its total.
constexpr int STRIP_CHUNKS = 32;
struct StripGroup {  // the group's k-th strip: row k / per_row, segment grp + ngroups (k % per_row)
    int64_t total;
    int per_row;
    __device__ StripGroup(int canvas_h, int segs, int ngroups, int grp) {
        per_row = (segs - grp + ngroups - 1) / ngroups;
        total = (int64_t)canvas_h * per_row;
    }
    __device__ int64_t strip(int64_t k, int segs, int ngroups, int grp) const {
        const int64_t r = k / per_row;
        return r * segs + grp + (k - r * per_row) * ngroups;
    }
};
__global__ void k_strip_counts(int canvas_h, int segs, int ngroups, const uint8_t* __restrict__ live,
                               int32_t* __restrict__ counts) {
    const int grp = blockIdx.x / STRIP_CHUNKS, c = blockIdx.x % STRIP_CHUNKS, lane = threadIdx.x & 63;
    const StripGroup sg(canvas_h, segs, ngroups, grp);
    const int64_t per = (sg.total + STRIP_CHUNKS - 1) / STRIP_CHUNKS, b0 = c * per, b1 = min(sg.total, b0 + per);
    int n = 0;
    for (int64_t k = b0 + lane; k < b1; k += 64) n += live[sg.strip(k, segs, ngroups, grp)] ? 1 : 0;
    for (int o = 32; o > 0; o >>= 1) n += __shfl_xor(n, o);
    if (lane == 0) counts[blockIdx.x] = n;
}
__global__ void k_strip_compact(int canvas_h, int segs, int ngroups, int list_pitch, const uint8_t* __restrict__ live,
                                const int32_t* __restrict__ counts, int32_t* __restrict__ lists) {
    const int grp = blockIdx.x / STRIP_CHUNKS, c = blockIdx.x % STRIP_CHUNKS, lane = threadIdx.x & 63;
    const StripGroup sg(canvas_h, segs, ngroups, grp);
    const int64_t per = (sg.total + STRIP_CHUNKS - 1) / STRIP_CHUNKS, b0 = c * per, b1 = min(sg.total, b0 + per);
    const int32_t* cnt = counts + grp * STRIP_CHUNKS;
    int32_t* list = lists + (int64_t)grp * list_pitch;
    int off = lane < c ? cnt[lane] : 0;  // STRIP_CHUNKS <= 64
    for (int o = 32; o > 0; o >>= 1) off += __shfl_xor(off, o);
    if (c == STRIP_CHUNKS - 1 && lane == 0) list[0] = off + cnt[c];
    for (int64_t k0 = b0; k0 < b1; k0 += 64) {
        const int64_t k = k0 + lane;
        const int64_t st = k < b1 ? sg.strip(k, segs, ngroups, grp) : 0;
        const bool lv = k < b1 && live[st];
        const uint64_t b = __ballot(lv);
        if (lv) list[1 + off + __popcll(b & ((1ull << lane) - 1))] = (int32_t)st;
        off += __popcll(b);
    }
}
static_assert(STRIP_CHUNKS <= 64, "one wave sums the chunk counts");

// fp32 storage at H = 32 takes the direct-to-LDS kernel, the other shapes
// the register-staged one.
template <typename T, int H, int C>
static void launch_strip_shape(const LayerGeom& g, int nwg, int n_strips, int segs, const void* d_dz, const void* d_x,
                               const void* d_y, const void* d_wx, const uint8_t* d_mask, const int32_t* d_rid,
                               int32_t* d_vid, void* d_dx, float* d_part, hipStream_t s) {
    constexpr bool DMA = std::is_same<T, float>::value && H == 32;
    constexpr int TC = StripCfg<H, C>::TC;
    // the strip lists: validity (ids for the direct-to-LDS kernel), a flag per
    // strip and the dX rows of the strips without a valid cell, then the lists
    const int ng = strip_groups(nwg, segs);
    uint8_t* live = reinterpret_cast<uint8_t*>(d_vid + g.n_cells);
    int32_t* counts = reinterpret_cast<int32_t*>(live + (n_strips + 3) / 4 * 4);
    int32_t* lists = counts + STRIP_GROUPS_MAX * STRIP_CHUNKS;
    const int pitch = (int)strip_list_pitch(g.canvas_h, segs, ng);
    const int vb = (int)std::min<int64_t>(((int64_t)n_strips * TC + 255) / 256, 4096);
    hipLaunchKernelGGL((k_valid_ids_strips<TC, T>), dim3(vb), dim3(256), 0, s, g.canvas_h, g.canvas_w, segs, C,
                       d_mask, d_rid, DMA ? d_vid : nullptr, live, static_cast<T*>(d_dx));
    hipLaunchKernelGGL(k_strip_counts, dim3(ng * STRIP_CHUNKS), dim3(64), 0, s, g.canvas_h, segs, ng, live, counts);
    hipLaunchKernelGGL(k_strip_compact, dim3(ng * STRIP_CHUNKS), dim3(64), 0, s, g.canvas_h, segs, ng, pitch, live,
                       counts, lists);
    if constexpr (DMA) {
        hipLaunchKernelGGL((k_bwd_strip_dma<H, C>), dim3(nwg), dim3(DmaCfg<H, C>::THREADS), 0, s, g.canvas_h,
                           g.canvas_w, segs, ng, pitch, lists, static_cast<const float*>(d_dz),
                           static_cast<const float*>(d_x), static_cast<const float*>(d_y),
                           static_cast<const float*>(d_wx), d_vid, static_cast<float*>(d_dx), d_part);
    } else {
        hipLaunchKernelGGL((k_bwd_strip<T, H, C>), dim3(nwg), dim3(StripCfg<H, C>::THREADS), 0, s, g.canvas_h,
                           g.canvas_w, segs, ng, pitch, lists, static_cast<const T*>(d_dz), static_cast<const T*>(d_x),
                           static_cast<const T*>(d_y), static_cast<const T*>(d_wx), d_mask, d_rid,
                           static_cast<T*>(d_dx), d_part);
    }
}

// validity ids (int32 per cell), then the lists of strips with a valid cell:
// a byte per strip (padded to 4), the chunk counts, and per group its count
// and strips
size_t strip_vid_bytes(const LayerGeom& g) {
    const int tc = strip_tc(g);
    const int segs = (g.canvas_w + tc - 1) / tc;
    const int64_t n_strips = (int64_t)g.canvas_h * segs;
    const int ng = strip_groups(strip_wgs(g), segs);
    return (size_t)(g.n_cells > 0 ? g.n_cells : 1) * 4 + (size_t)(n_strips + 3) / 4 * 4 +
           (size_t)STRIP_GROUPS_MAX * STRIP_CHUNKS * 4 + (size_t)ng * strip_list_pitch(g.canvas_h, segs, ng) * 4;
}

hipError_t launch_bwd_strip(const LayerGeom& g, const void* d_dz, const void* d_x, const void* d_y, const void* d_wx,
                            const uint8_t* d_mask, const int32_t* d_rid, int32_t* d_vid, void* d_dx, float* d_part,
                            float* d_dwx, float* d_du, float* d_db, hipStream_t s) {
    const int tc = strip_tc(g);
    const int segs = (g.canvas_w + tc - 1) / tc;
    const int n_strips = g.canvas_h * segs;
    const int nwg = strip_wgs(g);
    const int RT = (5 * g.hidden + 15) / 16, CT = (g.c_in + 2 * g.hidden + 15) / 16;
    bool ok = false;
#define MDL_STRIP_LAUNCH(T, H, C)                                                                                  \
    if (!ok && (g.dtype == 1) == std::is_same<T, bf16_t>::value && g.hidden == H && g.c_in == C) {                 \
        launch_strip_shape<T, H, C>(g, nwg, n_strips, segs, d_dz, d_x, d_y, d_wx, d_mask, d_rid, d_vid, d_dx,      \
                                    d_part, s);                                                                    \
        ok = true;                                                                                                 \
    }
    MDL_STRIP_SHAPES(MDL_STRIP_LAUNCH)
#undef MDL_STRIP_LAUNCH
    if (!ok) return hipErrorInvalidValue;
    const int total = 4 * 5 * g.hidden * (g.c_in + 2 * g.hidden + 1);
    hipLaunchKernelGGL(k_strip_reduce, dim3((total + 63) / 64), dim3(256), 0, s, g.c_in, g.hidden, RT, strip_pp(g),
                       CT, nwg, d_part, d_dwx, d_du, d_db);
    return hipGetLastError();
}

}  // namespace mdl
