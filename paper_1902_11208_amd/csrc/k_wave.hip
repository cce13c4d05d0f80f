// Anti-diagonal wavefront recurrence of the four-direction 2D MDLSTM
// (Section III cell; Section IV-A: after input skewing every cell of an
// anti-diagonal depends only on the previous anti-diagonal, so a whole
// diagonal is computed at once; Section V: state from predecessors outside
// the cell's rectangle or with mask 0 is blocked).
//
// One workgroup runs one unit = (rectangle, scan direction) and walks its
// h + w - 1 local anti-diagonals in order (forward) or in reverse (backward).
// Cells of a diagonal are indexed by their local row y, so a cell's left
// predecessor is row y on the previous diagonal and its top predecessor is
// row y - 1.
//
// Per step, the recurrent contraction is a small dense product done on MFMA:
//   forward   pre[r][cell] += sum_k U[r][k]   hcat[cell][k],  hcat = [h_L ; h_T]
//   backward  g[k][cell]    = sum_r U[r][k]   da[cell][r]
// The workgroup has one wave per block of 16 hidden units (jb). Wave jb keeps,
// for its 16 hidden units, U's rows of all five gates (forward) or U's columns
// for both predecessors (backward) in registers for the whole unit. Output
// tile row 4q + r and column n of lane 16q + n map to hidden unit
// j = 16 jb + 4q + r and the cell of local row 16 nt + n, so every lane holds
// all five gates of four hidden units of one cell and does the cell update
// without any exchange. Values that go to the same row on the next diagonal
// (c_L forward; U_L^T da and dc f_L backward) stay in registers; values for
// the neighbouring row and the full hidden vector go through LDS.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

template <typename T>
struct WaveOps;

// fp32: 16x16x4 MFMA, slot q of the reduction holds a contiguous run of
// KRUN values, one per K step.
template <>
struct WaveOps<float> {
    using Op = float;
    static constexpr int PER_STEP = 1;
    static __device__ __forceinline__ Op lds_op(const float* p) { return *p; }
    static __device__ __forceinline__ floatx4 mma(Op a, Op b, floatx4 c) { return mfma_f32(a, b, c); }
};

// bf16: 16x16x32 MFMA, eight consecutive values per K step.
template <>
struct WaveOps<bf16_t> {
    using Op = bf16x8;
    static constexpr int PER_STEP = 8;
    static __device__ __forceinline__ Op lds_op(const bf16_t* p) {
        return as_bf16x8(*reinterpret_cast<const uint4*>(p));
    }
    static __device__ __forceinline__ floatx4 mma(Op a, Op b, floatx4 c) { return mfma_bf16(a, b, c); }
};

template <typename T>
__device__ __forceinline__ void lds_st4(T* p, floatx4 v);
template <>
__device__ __forceinline__ void lds_st4<float>(float* p, floatx4 v) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
template <>
__device__ __forceinline__ void lds_st4<bf16_t>(bf16_t* p, floatx4 v) {
    uint2 o;
    o.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
    o.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
    *reinterpret_cast<uint2*>(p) = o;
}

__device__ __forceinline__ floatx4 lds_ld4f(const float* p) {
    float4 v = *reinterpret_cast<const float4*>(p);
    return floatx4{v.x, v.y, v.z, v.w};
}

// Load a K-slot of operand values from a row of U (global memory) with
// element stride `es` between consecutive k (1: along a row; 2H: down a column).
template <typename T, int NSTEP>
__device__ __forceinline__ void load_u_slot(const T* __restrict__ base, int es, bool ok,
                                            typename WaveOps<T>::Op (&v)[NSTEP]) {
    if constexpr (std::is_same<T, float>::value) {
#pragma unroll
        for (int ks = 0; ks < NSTEP; ++ks) v[ks] = ok ? base[(int64_t)ks * es] : 0.0f;
    } else {
#pragma unroll
        for (int ks = 0; ks < NSTEP; ++ks) {
            uint32_t w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                uint32_t lo = ok ? base[(int64_t)(8 * ks + 2 * e) * es] : 0;
                uint32_t hi = ok ? base[(int64_t)(8 * ks + 2 * e + 1) * es] : 0;
                w[e] = lo | (hi << 16);
            }
            v[ks] = as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
        }
    }
}

struct WaveArgs {
    const int32_t* units;  // unit = rect*4 + direction, in launch order
    const int32_t* rects;  // [n_rects][4]
    const uint8_t* mask;   // [n_cells]
    const void* u;         // [4][5H][2H]
    void* z;               // [n_cells][20H]: pre-activations in, activated gates out (fwd); dZ out (bwd)
    float* c;              // [n_cells][4H] cell state
    void* y;               // [n_cells][4H] output (fwd)
    const void* dy;        // [n_cells][4H] upstream gradient (bwd)
    int canvas_w;
};

// ---------------------------------------------------------------------------
// Forward.
// ---------------------------------------------------------------------------
template <int H, int NT, typename T>
__global__ void __launch_bounds__(64 * ((H + 15) / 16))
k_wave_fwd(WaveArgs a) {
    using Ops = WaveOps<T>;
    using Op = typename Ops::Op;
    constexpr int G = 5 * H;             // gate rows per direction
    constexpr int KRUN = H / 2;          // hcat values per reduction slot
    constexpr int NSTEP = KRUN / Ops::PER_STEP;
    constexpr int ROWS = NT * 16 + 1;    // +1: row 0 is the zero row above local row 0
    constexpr int HP = H + 16 / (int)sizeof(T);  // padded LDS row pitch (elements)
    static_assert(KRUN % Ops::PER_STEP == 0, "hidden size not supported for this storage type");
    __shared__ __attribute__((aligned(16))) T hbuf[2][ROWS][HP];
    __shared__ __attribute__((aligned(16))) float cbuf[2][ROWS][H];

    const int lane = threadIdx.x & 63, jb = threadIdx.x >> 6;
    const int q = lane >> 4, n16 = lane & 15;
    const int j0 = 16 * jb + 4 * q;  // this lane's four hidden units (output rows)
    const bool jok = j0 < H;
    const int unit = a.units[blockIdx.x];
    const int d = unit & 3;
    const RectD R = reinterpret_cast<const RectD*>(a.rects)[unit >> 2];
    const T* __restrict__ U = static_cast<const T*>(a.u) + (int64_t)d * G * 2 * H;
    T* __restrict__ Z = static_cast<T*>(a.z);
    T* __restrict__ Y = static_cast<T*>(a.y);
    float* __restrict__ Cs = a.c;

    for (int i = threadIdx.x; i < 2 * ROWS * HP; i += blockDim.x) (&hbuf[0][0][0])[i] = T(0);
    for (int i = threadIdx.x; i < 2 * ROWS * H; i += blockDim.x) (&cbuf[0][0][0])[i] = 0.0f;

    // A operand: U rows (gate t, hidden unit 16 jb + n16), reduction slot q
    // holding hcat indices k = q*KRUN .. q*KRUN + KRUN - 1.
    Op A[5][NSTEP];
    {
        const int jr = 16 * jb + n16;
#pragma unroll
        for (int t = 0; t < 5; ++t)
            load_u_slot<T, NSTEP>(U + (int64_t)(t * H + (jr < H ? jr : 0)) * 2 * H + q * KRUN, 1, jr < H, A[t]);
    }
    floatx4 cprev[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) cprev[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
    __syncthreads();

    const int steps = R.h + R.w - 1;
    for (int s = 0; s < steps; ++s) {
        const int cur = s & 1, prv = cur ^ 1;
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (16 * nt > yhi || 16 * nt + 15 < ylo) continue;  // uniform over the workgroup
            const int yy = 16 * nt + n16, xx = s - yy;
            const bool act = yy < R.h && xx >= 0 && xx < R.w;
            const int64_t p = act ? canvas_index(R, d, yy, xx, a.canvas_w) : 0;
            const bool live = act && jok;
            floatx4 zv[5];
            uint8_t m = 0;
            if (live) {
                m = a.mask[p];
#pragma unroll
                for (int t = 0; t < 5; ++t) zv[t] = St<T>::ld4(Z + p * (4 * G) + d * G + t * H + j0);
            }
            // B operand: slot q < 2 reads h_L (row yy of the previous diagonal),
            // q >= 2 reads h_T (row yy - 1); LDS row index is local row + 1.
            const T* brow = (q < 2) ? &hbuf[prv][yy + 1][q * KRUN] : &hbuf[prv][yy][(q - 2) * KRUN];
            floatx4 acc[5];
#pragma unroll
            for (int t = 0; t < 5; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < NSTEP; ++ks) {
                const Op b = Ops::lds_op(brow + ks * Ops::PER_STEP);
#pragma unroll
                for (int t = 0; t < 5; ++t) acc[t] = Ops::mma(A[t][ks], b, acc[t]);
            }
            floatx4 cn = floatx4{0.f, 0.f, 0.f, 0.f}, hn = cn;
            if (live) {
                const floatx4 cL = cprev[nt];
                const floatx4 cT = lds_ld4f(&cbuf[prv][yy][j0]);
                floatx4 gi, gfl, gft, go, gg;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    gi[r] = sigm(acc[0][r] + zv[0][r]);
                    gfl[r] = sigm(acc[1][r] + zv[1][r]);
                    gft[r] = sigm(acc[2][r] + zv[2][r]);
                    go[r] = sigm(acc[3][r] + zv[3][r]);
                    gg[r] = tanh_acc(acc[4][r] + zv[4][r]);
                    float c = gi[r] * gg[r] + gfl[r] * cL[r] + gft[r] * cT[r];
                    cn[r] = c;
                    hn[r] = go[r] * tanh_acc(c);
                }
                if (m) {
                    T* zp = Z + p * (4 * G) + d * G + j0;
                    St<T>::st4(zp + 0 * H, gi);
                    St<T>::st4(zp + 1 * H, gfl);
                    St<T>::st4(zp + 2 * H, gft);
                    St<T>::st4(zp + 3 * H, go);
                    St<T>::st4(zp + 4 * H, gg);
                    St<T>::st4(Y + p * (4 * H) + d * H + j0, hn);
                } else {
                    cn = floatx4{0.f, 0.f, 0.f, 0.f};
                    hn = cn;
                }
                St<float>::st4(Cs + p * (4 * H) + d * H + j0, cn);
            }
            cprev[nt] = cn;
            if (jok) {
                lds_st4<T>(&hbuf[cur][yy + 1][j0], hn);
                *reinterpret_cast<float4*>(&cbuf[cur][yy + 1][j0]) = make_float4(cn[0], cn[1], cn[2], cn[3]);
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Backward (reverse anti-diagonals). For a cell with successors S (right,
// same row, next diagonal) and E (below, row + 1, next diagonal):
//   dh = dY + (U^T da_S)[0:H] + (U^T da_E)[H:2H]
//   dc = dh o (1 - tanh^2 c) + dc_S f_L(S) + dc_E f_T(E)
//   da = (dc g i(1-i), dc c_L f_L(1-f_L), dc c_T f_T(1-f_T), dh tanh(c) o(1-o), dc i (1-g^2))
// Phase A does the cell update and writes da (over the saved gates, and to
// LDS); phase B contracts da with U^T for the predecessors.
// ---------------------------------------------------------------------------
template <int H, int NT, typename T>
__global__ void __launch_bounds__(64 * ((H + 15) / 16))
k_wave_bwd(WaveArgs a) {
    using Ops = WaveOps<T>;
    using Op = typename Ops::Op;
    constexpr int G = 5 * H;
    constexpr int KRUN = G / 4;          // da values per reduction slot
    constexpr int NSTEP = KRUN / Ops::PER_STEP;
    constexpr int GP = G + 16 / (int)sizeof(T);
    static_assert(KRUN % Ops::PER_STEP == 0, "hidden size not supported for this storage type");
    __shared__ __attribute__((aligned(16))) T dabuf[NT * 16][GP];
    __shared__ __attribute__((aligned(16))) float gtbuf[NT * 16 + 1][H];
    __shared__ __attribute__((aligned(16))) float dctbuf[NT * 16 + 1][H];

    const int lane = threadIdx.x & 63, jb = threadIdx.x >> 6;
    const int q = lane >> 4, n16 = lane & 15;
    const int j0 = 16 * jb + 4 * q;
    const bool jok = j0 < H;
    const int unit = a.units[blockIdx.x];
    const int d = unit & 3;
    const RectD R = reinterpret_cast<const RectD*>(a.rects)[unit >> 2];
    const T* __restrict__ U = static_cast<const T*>(a.u) + (int64_t)d * G * 2 * H;
    T* __restrict__ Z = static_cast<T*>(a.z);
    const T* __restrict__ DY = static_cast<const T*>(a.dy);
    const float* __restrict__ Cs = a.c;

    for (int i = threadIdx.x; i < NT * 16 * GP; i += blockDim.x) (&dabuf[0][0])[i] = T(0);
    for (int i = threadIdx.x; i < (NT * 16 + 1) * H; i += blockDim.x) {
        (&gtbuf[0][0])[i] = 0.0f;
        (&dctbuf[0][0])[i] = 0.0f;
    }

    // A operands: U^T rows k (column k of U) for the left part (k = 16 jb + n16)
    // and the top part (k = H + 16 jb + n16); slot q holds gate rows
    // r = q*KRUN .. q*KRUN + KRUN - 1.
    Op AL[NSTEP], AT[NSTEP];
    {
        const int kr = 16 * jb + n16;
        const bool ok = kr < H;
        const int kc = ok ? kr : 0;
        load_u_slot<T, NSTEP>(U + (int64_t)(q * KRUN) * 2 * H + kc, 2 * H, ok, AL);
        load_u_slot<T, NSTEP>(U + (int64_t)(q * KRUN) * 2 * H + H + kc, 2 * H, ok, AT);
    }
    floatx4 gl[NT], dcl[NT], dct_new[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        gl[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
        dcl[nt] = gl[nt];
        dct_new[nt] = gl[nt];
    }
    __syncthreads();

    const int steps = R.h + R.w - 1;
    for (int s = steps - 1; s >= 0; --s) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
        // Phase A: cell updates of diagonal s.
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (16 * nt > yhi || 16 * nt + 15 < ylo) continue;
            const int yy = 16 * nt + n16, xx = s - yy;
            const bool act = yy < R.h && xx >= 0 && xx < R.w;
            floatx4 da[5];
#pragma unroll
            for (int t = 0; t < 5; ++t) da[t] = floatx4{0.f, 0.f, 0.f, 0.f};
            floatx4 ndl = da[0], ndt = da[0];
            if (act && jok) {
                const int64_t p = canvas_index(R, d, yy, xx, a.canvas_w);
                if (a.mask[p]) {
                    const T* zp = Z + p * (4 * G) + d * G + j0;
                    const floatx4 gi = St<T>::ld4(zp), gfl = St<T>::ld4(zp + H), gft = St<T>::ld4(zp + 2 * H),
                                  go = St<T>::ld4(zp + 3 * H), gg = St<T>::ld4(zp + 4 * H);
                    const floatx4 dyv = St<T>::ld4(DY + p * (4 * H) + d * H + j0);
                    const floatx4 cv = St<float>::ld4(Cs + p * (4 * H) + d * H + j0);
                    floatx4 cL = floatx4{0.f, 0.f, 0.f, 0.f}, cT = cL;
                    if (xx > 0) cL = St<float>::ld4(Cs + canvas_index(R, d, yy, xx - 1, a.canvas_w) * (4 * H) + d * H + j0);
                    if (yy > 0) cT = St<float>::ld4(Cs + canvas_index(R, d, yy - 1, xx, a.canvas_w) * (4 * H) + d * H + j0);
                    const floatx4 gt = lds_ld4f(&gtbuf[yy + 1][j0]);
                    const floatx4 dcE = lds_ld4f(&dctbuf[yy + 1][j0]);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        float dh = dyv[r] + gl[nt][r] + gt[r];
                        float tc = tanh_acc(cv[r]);
                        float dc = dcl[nt][r] + dcE[r] + dh * go[r] * (1.0f - tc * tc);
                        da[0][r] = dc * gg[r] * gi[r] * (1.0f - gi[r]);
                        da[1][r] = dc * cL[r] * gfl[r] * (1.0f - gfl[r]);
                        da[2][r] = dc * cT[r] * gft[r] * (1.0f - gft[r]);
                        da[3][r] = dh * tc * go[r] * (1.0f - go[r]);
                        da[4][r] = dc * gi[r] * (1.0f - gg[r] * gg[r]);
                        ndl[r] = dc * gfl[r];
                        ndt[r] = dc * gft[r];
                    }
                    T* dz = Z + p * (4 * G) + d * G + j0;
#pragma unroll
                    for (int t = 0; t < 5; ++t) St<T>::st4(dz + t * H, da[t]);
                }
            }
            if (jok) {
#pragma unroll
                for (int t = 0; t < 5; ++t) lds_st4<T>(&dabuf[yy][t * H + j0], da[t]);
            }
            dcl[nt] = ndl;
            dct_new[nt] = ndt;
        }
        __syncthreads();
        // Phase B: contributions U^T da for the left and top predecessors.
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (16 * nt > yhi || 16 * nt + 15 < ylo) continue;
            const int yy = 16 * nt + n16;
            const T* brow = &dabuf[yy][q * KRUN];
            floatx4 accL = floatx4{0.f, 0.f, 0.f, 0.f}, accT = accL;
#pragma unroll
            for (int ks = 0; ks < NSTEP; ++ks) {
                const Op b = Ops::lds_op(brow + ks * Ops::PER_STEP);
                accL = Ops::mma(AL[ks], b, accL);
                accT = Ops::mma(AT[ks], b, accT);
            }
            gl[nt] = accL;
            if (jok) {
                *reinterpret_cast<float4*>(&gtbuf[yy][j0]) = make_float4(accT[0], accT[1], accT[2], accT[3]);
                floatx4 v = dct_new[nt];
                *reinterpret_cast<float4*>(&dctbuf[yy][j0]) = make_float4(v[0], v[1], v[2], v[3]);
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Dispatch over (hidden size, N tiles, storage type).
// ---------------------------------------------------------------------------
template <int H, int NT, typename T>
static void launch_pair(bool fwd, int n_units, const WaveArgs& a, hipStream_t s) {
    const dim3 grid(n_units), block(64 * ((H + 15) / 16));
    if (fwd) hipLaunchKernelGGL((k_wave_fwd<H, NT, T>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((k_wave_bwd<H, NT, T>), grid, block, 0, s, a);
}

template <int H, typename T>
static hipError_t launch_nt(bool fwd, int nt, int n_units, const WaveArgs& a, hipStream_t s) {
    switch (nt) {
        case 1: launch_pair<H, 1, T>(fwd, n_units, a, s); break;
        case 2: launch_pair<H, 2, T>(fwd, n_units, a, s); break;
        case 3: launch_pair<H, 3, T>(fwd, n_units, a, s); break;
        case 4: launch_pair<H, 4, T>(fwd, n_units, a, s); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

static hipError_t launch_wave(bool fwd, const LayerGeom& g, int nt, int n_units, const WaveArgs& a, hipStream_t s) {
    if (n_units == 0) return hipSuccess;
    if (g.dtype == 0) {
        switch (g.hidden) {
            case 4: return launch_nt<4, float>(fwd, nt, n_units, a, s);
            case 8: return launch_nt<8, float>(fwd, nt, n_units, a, s);
            case 16: return launch_nt<16, float>(fwd, nt, n_units, a, s);
            case 32: return launch_nt<32, float>(fwd, nt, n_units, a, s);
            case 64: return launch_nt<64, float>(fwd, nt, n_units, a, s);
            default: return hipErrorInvalidValue;
        }
    }
    switch (g.hidden) {
        case 32: return launch_nt<32, bf16_t>(fwd, nt, n_units, a, s);
        case 64: return launch_nt<64, bf16_t>(fwd, nt, n_units, a, s);
        case 128: return launch_nt<128, bf16_t>(fwd, nt, n_units, a, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_wavefront_fwd(const LayerGeom& g, int nt, int n_units, const int32_t* d_units,
                                const int32_t* d_rects, const uint8_t* d_mask, const void* d_u, void* d_z,
                                float* d_c, void* d_y, hipStream_t s) {
    WaveArgs a{d_units, d_rects, d_mask, d_u, d_z, d_c, d_y, nullptr, g.canvas_w};
    return launch_wave(true, g, nt, n_units, a, s);
}

hipError_t launch_wavefront_bwd(const LayerGeom& g, int nt, int n_units, const int32_t* d_units,
                                const int32_t* d_rects, const uint8_t* d_mask, const void* d_u, const void* d_dy,
                                void* d_z, const float* d_c, hipStream_t s) {
    WaveArgs a{d_units, d_rects, d_mask, d_u, d_z, const_cast<float*>(d_c), nullptr, d_dy, g.canvas_w};
    return launch_wave(false, g, nt, n_units, a, s);
}

}  // namespace mdl
