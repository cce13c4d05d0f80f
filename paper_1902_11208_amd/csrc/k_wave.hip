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

// Raw 4-element loads kept in registers until use (prefetched one step ahead).
template <typename T>
struct Raw;
template <>
struct Raw<float> {
    using V = float4;
    static __device__ __forceinline__ V load(const float* p) { return *reinterpret_cast<const float4*>(p); }
    static __device__ __forceinline__ floatx4 f(V v) { return floatx4{v.x, v.y, v.z, v.w}; }
    static __device__ __forceinline__ V zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
};
template <>
struct Raw<bf16_t> {
    using V = uint2;
    static __device__ __forceinline__ V load(const bf16_t* p) { return *reinterpret_cast<const uint2*>(p); }
    static __device__ __forceinline__ floatx4 f(V v) {
        return floatx4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u), __uint_as_float(v.y << 16),
                       __uint_as_float(v.y & 0xffff0000u)};
    }
    static __device__ __forceinline__ V zero() { return make_uint2(0, 0); }
};

// Whether a unit keeps the next step's global loads in a second register set.
// Large tiles (H = 128, or many N tiles at H = 64) would spill instead.
template <int H, int NT, typename T>
struct Prefetch {
    static constexpr bool on = (H <= 32 && NT <= 2) || (H == 64 && NT == 1);
};

// ---------------------------------------------------------------------------
// Forward.
// ---------------------------------------------------------------------------
template <int NT, typename T>
struct FwdPre {
    typename Raw<T>::V z[NT][5];
    int64_t p[NT];
    uint32_t m[NT];
    bool live[NT];
};

template <int H, int NT, typename T>
__global__ void __launch_bounds__(64 * ((H + 15) / 16))
k_wave_fwd(WaveArgs a) {
    using Ops = WaveOps<T>;
    using Op = typename Ops::Op;
    using R4 = Raw<T>;
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
    const int steps = R.h + R.w - 1;

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

    // Global loads of step s (pre-activations and mask); they depend only on
    // the position, never on the recurrence, so they can be issued early.
    auto fetch = [&](int s, FwdPre<NT, T>& b) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            b.live[nt] = false;
            if (s >= steps || 16 * nt > yhi || 16 * nt + 15 < ylo) continue;
            const int yy = 16 * nt + n16, xx = s - yy;
            const bool live = jok && yy < R.h && xx >= 0 && xx < R.w;
            b.live[nt] = live;
            if (live) {
                const int64_t p = canvas_index(R, d, yy, xx, a.canvas_w);
                b.p[nt] = p;
                b.m[nt] = a.mask[p];
                const T* zp = Z + p * (4 * G) + d * G + j0;
#pragma unroll
                for (int t = 0; t < 5; ++t) b.z[nt][t] = R4::load(zp + t * H);
            }
        }
    };

    auto compute = [&](int s, const FwdPre<NT, T>& b) {
        const int cur = s & 1, prv = cur ^ 1;
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (16 * nt > yhi || 16 * nt + 15 < ylo) continue;  // uniform over the workgroup
            const int yy = 16 * nt + n16;
            // B operand: slot q < 2 reads h_L (row yy of the previous diagonal),
            // q >= 2 reads h_T (row yy - 1); LDS row index is local row + 1.
            const T* brow = (q < 2) ? &hbuf[prv][yy + 1][q * KRUN] : &hbuf[prv][yy][(q - 2) * KRUN];
            floatx4 acc[5];
#pragma unroll
            for (int t = 0; t < 5; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < NSTEP; ++ks) {
                const Op bop = Ops::lds_op(brow + ks * Ops::PER_STEP);
#pragma unroll
                for (int t = 0; t < 5; ++t) acc[t] = Ops::mma(A[t][ks], bop, acc[t]);
            }
            floatx4 cn = floatx4{0.f, 0.f, 0.f, 0.f}, hn = cn;
            if (b.live[nt]) {
                const floatx4 cL = cprev[nt];
                const floatx4 cT = lds_ld4f(&cbuf[prv][yy][j0]);
                floatx4 gi, gfl, gft, go, gg;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    gi[r] = sigm_fast(acc[0][r] + R4::f(b.z[nt][0])[r]);
                    gfl[r] = sigm_fast(acc[1][r] + R4::f(b.z[nt][1])[r]);
                    gft[r] = sigm_fast(acc[2][r] + R4::f(b.z[nt][2])[r]);
                    go[r] = sigm_fast(acc[3][r] + R4::f(b.z[nt][3])[r]);
                    gg[r] = tanh_fast(acc[4][r] + R4::f(b.z[nt][4])[r]);
                    const float c = gi[r] * gg[r] + gfl[r] * cL[r] + gft[r] * cT[r];
                    cn[r] = c;
                    hn[r] = go[r] * tanh_fast(c);
                }
                const int64_t p = b.p[nt];
                if (b.m[nt]) {
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
    };

    __syncthreads();
    FwdPre<NT, T> b0, b1;
    if constexpr (Prefetch<H, NT, T>::on) {
        // two register sets in turn: step s computes from one while the loads
        // of step s + 1 land in the other
        fetch(0, b0);
        int s = 0;
        for (; s + 1 < steps; s += 2) {
            fetch(s + 1, b1);
            compute(s, b0);
            fetch(s + 2, b0);
            compute(s + 1, b1);
        }
        if (s < steps) compute(s, b0);
    } else {
        for (int s = 0; s < steps; ++s) {
            fetch(s, b0);
            compute(s, b0);
        }
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
template <int NT, typename T>
struct BwdPre {
    typename Raw<T>::V g[NT][5], dy[NT];
    float4 c[NT], cl[NT], ct[NT];
    int64_t p[NT];
    uint32_t m[NT];
    bool live[NT];
};

template <int H, int NT, typename T>
__global__ void __launch_bounds__(64 * ((H + 15) / 16))
k_wave_bwd(WaveArgs a) {
    using Ops = WaveOps<T>;
    using Op = typename Ops::Op;
    using R4 = Raw<T>;
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
    const int steps = R.h + R.w - 1;

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

    auto fetch = [&](int s, BwdPre<NT, T>& b) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            b.live[nt] = false;
            if (s < 0 || 16 * nt > yhi || 16 * nt + 15 < ylo) continue;
            const int yy = 16 * nt + n16, xx = s - yy;
            const bool live = jok && yy < R.h && xx >= 0 && xx < R.w;
            b.live[nt] = live;
            if (live) {
                const int64_t p = canvas_index(R, d, yy, xx, a.canvas_w);
                b.p[nt] = p;
                b.m[nt] = a.mask[p];
                const T* zp = Z + p * (4 * G) + d * G + j0;
#pragma unroll
                for (int t = 0; t < 5; ++t) b.g[nt][t] = R4::load(zp + t * H);
                b.dy[nt] = R4::load(DY + p * (4 * H) + d * H + j0);
                b.c[nt] = Raw<float>::load(Cs + p * (4 * H) + d * H + j0);
                b.cl[nt] = xx > 0 ? Raw<float>::load(Cs + canvas_index(R, d, yy, xx - 1, a.canvas_w) * (4 * H) + d * H + j0)
                                  : Raw<float>::zero();
                b.ct[nt] = yy > 0 ? Raw<float>::load(Cs + canvas_index(R, d, yy - 1, xx, a.canvas_w) * (4 * H) + d * H + j0)
                                  : Raw<float>::zero();
            }
        }
    };

    auto compute = [&](int s, const BwdPre<NT, T>& b) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
        // Phase A: cell updates of diagonal s.
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (16 * nt > yhi || 16 * nt + 15 < ylo) continue;
            const int yy = 16 * nt + n16;
            floatx4 da[5];
#pragma unroll
            for (int t = 0; t < 5; ++t) da[t] = floatx4{0.f, 0.f, 0.f, 0.f};
            floatx4 ndl = da[0], ndt = da[0];
            if (b.live[nt] && b.m[nt]) {
                const floatx4 gi = R4::f(b.g[nt][0]), gfl = R4::f(b.g[nt][1]), gft = R4::f(b.g[nt][2]),
                              go = R4::f(b.g[nt][3]), gg = R4::f(b.g[nt][4]);
                const floatx4 dyv = R4::f(b.dy[nt]);
                const floatx4 cv = Raw<float>::f(b.c[nt]), cL = Raw<float>::f(b.cl[nt]), cT = Raw<float>::f(b.ct[nt]);
                const floatx4 gt = lds_ld4f(&gtbuf[yy + 1][j0]);
                const floatx4 dcE = lds_ld4f(&dctbuf[yy + 1][j0]);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float dh = dyv[r] + gl[nt][r] + gt[r];
                    const float tc = tanh_fast(cv[r]);
                    const float dc = dcl[nt][r] + dcE[r] + dh * go[r] * (1.0f - tc * tc);
                    da[0][r] = dc * gg[r] * gi[r] * (1.0f - gi[r]);
                    da[1][r] = dc * cL[r] * gfl[r] * (1.0f - gfl[r]);
                    da[2][r] = dc * cT[r] * gft[r] * (1.0f - gft[r]);
                    da[3][r] = dh * tc * go[r] * (1.0f - go[r]);
                    da[4][r] = dc * gi[r] * (1.0f - gg[r] * gg[r]);
                    ndl[r] = dc * gfl[r];
                    ndt[r] = dc * gft[r];
                }
                T* dz = Z + b.p[nt] * (4 * G) + d * G + j0;
#pragma unroll
                for (int t = 0; t < 5; ++t) St<T>::st4(dz + t * H, da[t]);
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
                const Op bop = Ops::lds_op(brow + ks * Ops::PER_STEP);
                accL = Ops::mma(AL[ks], bop, accL);
                accT = Ops::mma(AT[ks], bop, accT);
            }
            gl[nt] = accL;
            if (jok) {
                *reinterpret_cast<float4*>(&gtbuf[yy][j0]) = make_float4(accT[0], accT[1], accT[2], accT[3]);
                const floatx4 v = dct_new[nt];
                *reinterpret_cast<float4*>(&dctbuf[yy][j0]) = make_float4(v[0], v[1], v[2], v[3]);
            }
        }
        __syncthreads();
    };

    __syncthreads();
    BwdPre<NT, T> b0, b1;
    if constexpr (Prefetch<H, NT, T>::on) {
        fetch(steps - 1, b0);
        int s = steps - 1;
        for (; s - 1 >= 0; s -= 2) {
            fetch(s - 1, b1);
            compute(s, b0);
            fetch(s - 2, b0);
            compute(s - 1, b1);
        }
        if (s >= 0) compute(s, b0);
    } else {
        for (int s = steps - 1; s >= 0; --s) {
            fetch(s, b0);
            compute(s, b0);
        }
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
