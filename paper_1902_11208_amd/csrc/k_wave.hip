// Anti-diagonal wavefront recurrence of the four-direction 2D MDLSTM
// (Section III cell; Section IV-A: after input skewing every cell of an
// anti-diagonal depends only on the previous anti-diagonal; Section V: state
// from predecessors outside the cell's rectangle or with mask 0 is blocked).
//
// One workgroup runs one unit = (rectangle, scan direction) and walks its
// h + w - 1 local anti-diagonals. Cells of a diagonal are indexed by local
// row y: the left predecessor is row y of the previous diagonal, the top
// predecessor row y - 1.
//
// The unit's hidden units are split over NW waves in quads of four. Forward,
// per step and 16-cell tile:
//  * each wave computes, on MFMA, the pre-activations of the four sigmoid
//    gates (i, f_L, f_T, o) of its quads from [h_L ; h_T]; the A operand rows
//    are ordered (quad member, gate) so that lane 16q + n ends up holding all
//    four gates of hidden unit 4*quad + q of cell n;
//  * the cell-candidate pre-activations are split over the waves by
//    reduction range and summed through LDS in a fixed order;
//  * then every lane updates c and h of its (cell, hidden unit) pairs.
// Backward, per step: every lane does the gate-gradient update of its pairs
// (phase A), then the waves contract da with U^T on MFMA, split by output
// tile and reduction range, partials summed through LDS in a fixed order
// (phase B). The U operands stay in VGPRs for the whole unit.
#include <algorithm>
#include <climits>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace mdl {

namespace {

template <typename T>
struct Ops;
template <>
struct Ops<float> {  // 16x16x4 f32 MFMA: one reduction value per slot and step
    using Op = float;
    static constexpr int PER = 1;
    static __device__ __forceinline__ Op lds(const float* p) { return *p; }
    static __device__ __forceinline__ floatx4 mma(Op a, Op b, floatx4 c) { return mfma_f32(a, b, c); }
};
template <>
struct Ops<bf16_t> {  // 16x16x32 bf16 MFMA: eight consecutive values per slot and step
    using Op = bf16x8;
    static constexpr int PER = 8;
    static __device__ __forceinline__ Op lds(const bf16_t* p) { return as_bf16x8(*reinterpret_cast<const uint4*>(p)); }
    static __device__ __forceinline__ floatx4 mma(Op a, Op b, floatx4 c) { return mfma_bf16(a, b, c); }
};

template <typename T>
__device__ __forceinline__ float ld1f(const T* p) { return St<T>::ld1(p); }

// N consecutive operands from LDS; fp32 runs of a multiple of four (two)
// values as 16-byte (8-byte) reads, which the row pitches and run offsets of
// the callers keep aligned. With row pitches of 4 mod 32 banks, the lanes of
// a 16-byte read that the LDS serves together fall on distinct bank quads.
template <typename T, int N>
__device__ __forceinline__ void lds_run(const T* p, typename Ops<T>::Op (&v)[N]) {
    if constexpr (std::is_same<T, float>::value && N % 4 == 0) {
#pragma unroll
        for (int k = 0; k < N / 4; ++k) {
            const float4 f = *reinterpret_cast<const float4*>(p + 4 * k);
            v[4 * k] = f.x;
            v[4 * k + 1] = f.y;
            v[4 * k + 2] = f.z;
            v[4 * k + 3] = f.w;
        }
    } else if constexpr (std::is_same<T, float>::value && N % 2 == 0) {
#pragma unroll
        for (int k = 0; k < N / 2; ++k) {
            const float2 f = *reinterpret_cast<const float2*>(p + 2 * k);
            v[2 * k] = f.x;
            v[2 * k + 1] = f.y;
        }
    } else {
#pragma unroll
        for (int ks = 0; ks < N; ++ks) v[ks] = Ops<T>::lds(p + ks * Ops<T>::PER);
    }
}

template <typename T>
__device__ __forceinline__ T from_f(float v);
template <>
__device__ __forceinline__ float from_f<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16_t from_f<bf16_t>(float v) { return f2bf(v); }

// A-operand values of one reduction slot from global memory: element stride
// `es` between consecutive k.
template <typename T, int NSTEP>
__device__ __forceinline__ void load_slot(const T* __restrict__ base, int64_t es, bool ok,
                                          typename Ops<T>::Op (&v)[NSTEP]) {
    if constexpr (std::is_same<T, float>::value) {
#pragma unroll
        for (int ks = 0; ks < NSTEP; ++ks) v[ks] = ok ? base[ks * es] : 0.0f;
    } else {
#pragma unroll
        for (int ks = 0; ks < NSTEP; ++ks) {
            uint32_t w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t lo = ok ? base[(8 * ks + 2 * e) * es] : 0;
                const uint32_t hi = ok ? base[(8 * ks + 2 * e + 1) * es] : 0;
                w[e] = lo | (hi << 16);
            }
            v[ks] = as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
        }
    }
}

template <int H, typename T>
struct Geo {
    // Waves per unit: fp32, one hidden-unit quad per wave up to eight waves.
    // The waves of a workgroup share the four SIMDs of a CU, and a wave alone
    // on its SIMD leaves MFMA and VALU issue slots idle, so more waves with
    // less work each shorten every step (beyond eight the VGPR budget spills).
    static constexpr int NW = std::is_same<T, float>::value ? (H <= 4 ? 1 : (H <= 32 ? H / 4 : 8))
                                                             : (H <= 8 ? 2 : (H <= 32 ? 4 : 8));
    static constexpr int WQ = (H / 4) / NW;                                     // hidden-unit quads per wave
    static constexpr int G = 5 * H;
    static constexpr int PER = Ops<T>::PER;
    // forward
    static constexpr int KRUN = H / 2;                  // hcat values per reduction slot
    static constexpr int NSTEP = KRUN / PER;
    static constexpr int GT = (H + 15) / 16;            // cell-candidate tiles
    static constexpr int SPL = NW / GT;                 // waves sharing one candidate tile
    static constexpr int GSTEP = NSTEP / SPL;           // candidate K steps per wave
    // backward
    static constexpr int KRUNB = G / 4;                 // da values per reduction slot
    static constexpr int NSTEPB = KRUNB / PER;
    static constexpr int MT = (2 * H + 15) / 16;        // output tiles of U^T da
    static constexpr int TPW = MT >= NW ? MT / NW : 1;  // output tiles per wave
    static constexpr int SPLB = MT >= NW ? 1 : NW / MT;  // waves sharing one output tile
    static constexpr int BSTEP = NSTEPB / SPLB;
    static_assert(KRUN % PER == 0 && NSTEP % SPL == 0 && GT * SPL == NW, "forward split");
    static_assert(KRUNB % PER == 0 && NSTEPB % SPLB == 0, "backward split");
    static_assert(MT >= NW ? MT % NW == 0 : NW % MT == 0, "backward tiles");
};

// Per-step outputs of one cell, staged in LDS as 16-byte chunks and written
// back by the whole workgroup with contiguous 16-byte stores: forward, the
// 5H activated gates then the H outputs (storage type) then the H cell states
// (fp32); backward, the 5H gate gradients.
template <int H, typename T>
struct OutQ {
    static constexpr int QZ = 5 * H * (int)sizeof(T) / 16;
    static constexpr int QY = H * (int)sizeof(T) / 16;
    static constexpr int QC = H * 4 / 16;
    static constexpr int QF = QZ + QY + QC;  // forward chunks per cell
    static_assert(QZ * 16 == 5 * H * (int)sizeof(T) && QY * 16 == H * (int)sizeof(T), "chunking");
};

// Waves of a unit (forward and backward) in groups of NW, one group per
// 16-row tile, when the workgroup stays within 1024 threads and the registers
// allow (fp32 up to H = 32): the tiles of a diagonal then run side by side on
// their own waves instead of one after another on the same ones.
template <int H, int NT, typename T>
struct TileGroups {
    static constexpr int NG =
        (std::is_same<T, float>::value && H <= 32 && NT >= 2 && 64 * Geo<H, T>::NW * NT <= 1024) ? NT : 1;
};

// LDS bytes of the forward kernel without and with staging of its inputs
// (two diagonals of pre-activations) and outputs (one diagonal).
template <int H, int NT, typename T>
constexpr size_t fwd_lds_base() {
    using Gm = Geo<H, T>;
    return (size_t)2 * (NT * 16 + 1) * (H + 16 / sizeof(T)) * sizeof(T) + (size_t)2 * (NT * 16 + 1) * (H + 2) * 4 +
           (size_t)Gm::SPL * NT * 16 * (H + 2) * 4 + (size_t)NT * 16 * 8;
}
template <int H, int NT, typename T>
constexpr bool fwd_stage() {
    using Q = OutQ<H, T>;
    return fwd_lds_base<H, NT, T>() + (size_t)NT * 16 * 16 * ((Q::QF + 1) + 2 * (Q::QZ + 1)) <= 128 * 1024;
}

// LDS bytes of the backward kernel without and with staging of its inputs
// (two diagonals of gates, upstream gradients and cell states).
template <int H, int NT, typename T>
constexpr size_t bwd_lds_base() {
    using Gm = Geo<H, T>;
    return (size_t)NT * 16 * (Gm::G + 16 / sizeof(T)) * sizeof(T) +
           (size_t)Gm::SPLB * (NT * 16 + 2) * (2 * H + 2) * 4 + (size_t)(NT * 16 + 2) * (H + 2) * 4;
}
template <int H, int NT, typename T>
constexpr size_t bwd_lds_stage() {
    constexpr size_t nth = 64 * Geo<H, T>::NW * TileGroups<H, NT, T>::NG;
    return 2 * ((NT * 16 * (OutQ<H, T>::QF + 1) + nth - 1) / nth * nth) * 16;
}
template <int H, int NT, typename T>
constexpr bool bwd_stage() {
    return bwd_lds_base<H, NT, T>() + bwd_lds_stage<H, NT, T>() <= 128 * 1024;
}

template <typename T>
struct Prefetch2 {
    template <int NT, int WQ>
    static constexpr bool on() { return NT * WQ <= 2; }
};

struct WaveArgs {
    const int32_t* units;  // unit = rect*4 + direction, in launch order
    const int32_t* rects;  // [n_rects][4]
    const uint8_t* mask;   // [n_cells]
    const void* u;         // [4][5H][2H]
    void* z;               // [n_cells][20H]: pre-activations in, gates out (fwd); dZ out (bwd)
    float* c;              // [n_cells][4H] cell state
    void* y;               // [n_cells][4H] output (fwd)
    const void* dy;        // [n_cells][4H] upstream gradient (bwd)
    int canvas_w;
    int s0, s1;            // forward: local diagonals [s0, s1) of every unit
    unsigned* queue;       // next unit to take (zeroed before the launch), or NULL: unit = block
    int n_units;
    // forward: when rid is set, the output rows [yrow_words x 8 bytes] of the
    // cells outside every rectangle or masked are zeroed before the units run
    const int32_t* rid;    // [n_cells] rectangle id, -1 outside every rectangle
    int64_t n_cells;
    int yrow_words;
};

template <int NT, int WQ, typename T>
struct FPre {
    T z[NT][WQ][5];
    int64_t p[NT];
    uint32_t m[NT];
    bool live[NT];
};

template <int NT, int WQ, typename T>
struct BPre {
    T g[NT][WQ][5], dy[NT][WQ];
    float c[NT][WQ], cl[NT][WQ], ct[NT][WQ];
    int64_t p[NT];
    uint32_t m[NT];
    bool live[NT], hasl[NT], hast[NT];
};

}  // namespace

// ---------------------------------------------------------------------------
// Forward.
// ---------------------------------------------------------------------------
template <int H, int NT, typename T, int PFD>
__device__ __forceinline__ void wave_fwd_unit(const WaveArgs& a, const int unit) {
    using Gm = Geo<H, T>;
    using O = Ops<T>;
    using Op = typename O::Op;
    using Q = OutQ<H, T>;
    constexpr int NW = Gm::NW, WQ = Gm::WQ, G = Gm::G, KRUN = Gm::KRUN, NSTEP = Gm::NSTEP;
    // tile groups: NG groups of NW waves, group tg owning tiles tg, tg + NG, ...
    constexpr int NG = TileGroups<H, NT, T>::NG, TPG = NT / NG;
    constexpr int SPL = Gm::SPL, GSTEP = Gm::GSTEP, NTH = 64 * NW * NG;
    constexpr int ROWS = NT * 16 + 1;             // row 0: zero row above local row 0
    constexpr int HP = H + 16 / (int)sizeof(T);   // padded LDS row pitch (elements)
    // Staged: the pre-activations of the next diagonal are loaded as contiguous
    // 16-byte chunks into registers one step ahead and pass through LDS to
    // the lanes that use them; the outputs leave through LDS the same way.
    // Otherwise every lane loads and stores its own values.
    constexpr bool STAGE = fwd_stage<H, NT, T>();
    constexpr int NC = STAGE ? NT * 16 : 1;
    constexpr int PF = STAGE ? Q::QF + 1 : 1;     // chunk pitches; the extra chunk
    constexpr int PZ = STAGE ? Q::QZ + 1 : 1;     // keeps rows in different LDS banks
    // input slots, rounded up to whole workgroup passes so every lane loads
    constexpr int NSL = STAGE ? (NT * 16 * PZ + NTH - 1) / NTH * NTH : 1;
    constexpr int NITZ = STAGE ? NSL / NTH : 0;
    __shared__ __attribute__((aligned(16))) T hbuf[2][ROWS][HP];
    __shared__ __attribute__((aligned(16))) float cbuf[2][ROWS][H + 2];  // pitch H + 2: rows of a tile in different banks
    __shared__ __attribute__((aligned(16))) float gpart[SPL][NT * 16][H + 2];
    __shared__ __attribute__((aligned(16))) u32x4 ostage[NC][PF];
    __shared__ __attribute__((aligned(16))) u32x4 zst[STAGE ? 2 : 1][NSL];  // by diagonal parity
    // mask bytes by diagonal parity; a slot per thread so that every lane
    // writes (rows below 16 NT are read)
    __shared__ uint32_t mst[STAGE ? 2 : 1][STAGE ? NTH : 1];

    const int lane = threadIdx.x & 63;
    const int tg = NG == 1 ? 0 : (int)(threadIdx.x >> 6) / NW;     // tile group
    const int w = NG == 1 ? (int)(threadIdx.x >> 6) : (int)(threadIdx.x >> 6) % NW;  // wave in the group
    const int q = lane >> 4, n16 = lane & 15;
    const int gt = w / SPL, sp = w % SPL;  // candidate tile and reduction slice of this wave
    const int d = unit & 3;
    const RectD R = reinterpret_cast<const RectD*>(a.rects)[unit >> 2];
    const T* __restrict__ U = static_cast<const T*>(a.u) + (int64_t)d * G * 2 * H;
    T* __restrict__ Z = static_cast<T*>(a.z);
    T* __restrict__ Y = static_cast<T*>(a.y);
    float* __restrict__ Cs = a.c;
    const int steps = R.h + R.w - 1;
    // Diagonals [sb, se) of the unit: all of them in one launch, or one per
    // launch, in which case the state of diagonal sb - 1 is read back from the
    // outputs and cell states the previous launch wrote.
    const int sb = a.s0, se = min(a.s1, steps);
    if (sb >= se) return;

    for (int i = threadIdx.x; i < 2 * ROWS * HP; i += blockDim.x) (&hbuf[0][0][0])[i] = T(0);
    for (int i = threadIdx.x; i < 2 * ROWS * (H + 2); i += blockDim.x) (&cbuf[0][0][0])[i] = 0.0f;
    if (sb > 0) {
        lds_barrier();  // every zero written before the read-back fills the same rows
        const int pb = (sb & 1) ^ 1;  // buffer of diagonal sb - 1
        for (int i = threadIdx.x; i < NT * 16 * H; i += blockDim.x) {
            const int yy = i / H, j = i - yy * H, xx = sb - 1 - yy;
            if (yy < R.h && xx >= 0 && xx < R.w) {
                const int64_t p = canvas_index(R, d, yy, xx, a.canvas_w);
                hbuf[pb][yy + 1][j] = Y[p * (4 * H) + d * H + j];
                cbuf[pb][yy + 1][j] = Cs[p * (4 * H) + d * H + j];
            }
        }
    }

    // A operands. Own tiles: row n16 = 4*jj + gate -> U row gate*H + 4*quad + jj.
    // Candidate tile gt: row n16 -> U row 4H + 16*gt + n16, K steps of slice sp only.
    Op Aown[WQ][NSTEP], Ag[GSTEP];
#pragma unroll
    for (int wq = 0; wq < WQ; ++wq) {
        const int quad = w * WQ + wq;
        const int row = (n16 & 3) * H + 4 * quad + (n16 >> 2);
        load_slot<T, NSTEP>(U + (int64_t)row * 2 * H + q * KRUN, 1, true, Aown[wq]);
    }
    {
        const int j = 16 * gt + n16;
        const bool ok = j < H;
        load_slot<T, GSTEP>(U + (int64_t)(4 * H + (ok ? j : 0)) * 2 * H + q * KRUN + sp * GSTEP * O::PER, 1, ok, Ag);
    }
    float cprev[TPG][WQ];  // c_L: the lane's cell state of the previous diagonal
#pragma unroll
    for (int lt = 0; lt < TPG; ++lt)
#pragma unroll
        for (int wq = 0; wq < WQ; ++wq) {
            const int nt = tg + NG * lt;
            const int yy = 16 * nt + n16, j = 4 * (w * WQ + wq) + q, xx = sb - 1 - yy;
            cprev[lt][wq] = sb > 0 && yy < R.h && xx >= 0 && xx < R.w
                                ? Cs[canvas_index(R, d, yy, xx, a.canvas_w) * (4 * H) + d * H + j]
                                : 0.0f;
        }
    // The U operands are in registers before the step loop starts, so no wait
    // inside the loop is attributed to them.
    __builtin_amdgcn_s_waitcnt(0);

    // Loads of step s: the lane's cells, their mask bytes and the
    // pre-activations (staged: chunks into zr, else the lane's own values).
    // They are issued for every lane from a valid cell of the rectangle (the
    // row clamped into the diagonal's active range) so their number is the
    // same on every path, which lets the compiler wait for exactly these loads
    // one step later; `live` says whether they are used.
    // Staged chunks and mask bytes loaded PFD steps ahead of their diagonal's
    // staging step (set k holds diagonals sb + k, sb + k + PFD, ...).
    static_assert(PFD == 1 || PFD == 2, "prefetch distance");
    u32x4 zr[PFD][NITZ > 0 ? NITZ : 1];
    uint32_t mr[PFD];
    const DiagMap M(R, d, a.canvas_w);
    constexpr int RBZ = 4 * G * (int)sizeof(T);  // bytes per canvas cell of Z
    // Cell (y, s - y) of the unit is canvas index M.c0 + idx with
    // idx = sx*s + y*ky, which fits 32 bits; the lanes keep 64-bit pointers to
    // their chunks at idx = 0 and add idx times the tensor's row bytes.
    const uint8_t* mrow = a.mask + M.c0;
    // The lane's chunk of each staged-input pass: cell row and address (slot S
    // of zst is chunk S % PZ of the row of cell S / PZ; the padding chunk and
    // the slots past the last cell repeat a valid one).
    int zcell[NITZ > 0 ? NITZ : 1];
    const char* zptr[NITZ > 0 ? NITZ : 1];
#pragma unroll
    for (int it = 0; it < NITZ; ++it) {
        const int S = it * NTH + (int)threadIdx.x;
        zcell[it] = min(S / PZ, NT * 16 - 1);
        zptr[it] = reinterpret_cast<const char*>(Z) + M.c0 * RBZ + (d * G) * (int)sizeof(T) +
                   16 * min(S - (S / PZ) * PZ, Q::QZ - 1);
    }
    // Loads of step s: the lanes' mask bytes and the pre-activations (staged:
    // chunks into zr, else the lane's own values). They are issued for every
    // lane from a valid cell of the rectangle (the row clamped into the
    // diagonal's active range) so their number is the same on every path,
    // which lets the compiler wait for exactly these loads one step later;
    // `live` says whether they are used.
    auto fetch = [&](int s, FPre<TPG, WQ, T>& b) {
        const int sc = min(s, steps - 1);
        const int ylo = max(0, sc - R.w + 1), yhi = min(R.h - 1, sc);
        const int sxs = M.sx * sc;
#pragma unroll
        for (int lt = 0; lt < TPG; ++lt) {
            const int nt = tg + NG * lt;
            const int yy = 16 * nt + n16;
            b.live[lt] = s < steps && yy >= ylo && yy <= yhi;
            const int idx = sxs + min(max(yy, ylo), yhi) * M.ky;
            b.m[lt] = mrow[idx];
            if constexpr (!STAGE) {
                const int64_t p = M.c0 + idx;
                b.p[lt] = p;
                const T* zp = Z + p * (4 * G) + d * G;
#pragma unroll
                for (int wq = 0; wq < WQ; ++wq) {
                    const int j = 4 * (w * WQ + wq) + q;
#pragma unroll
                    for (int t = 0; t < 5; ++t) b.z[lt][wq][t] = zp[t * H + j];
                }
            }
        }
    };
    // Staged pre-activation chunks and the mask byte of row threadIdx.x (of
    // the last row above 16 NT, unused there) of diagonal s into register set k.
    auto fetch_z = [&](int s, int k) {
        const int sc = min(s, steps - 1);
        const int ylo = max(0, sc - R.w + 1), yhi = min(R.h - 1, sc);
        const int sxs = M.sx * sc;
        if constexpr (STAGE) {
#pragma unroll
            for (int it = 0; it < NITZ; ++it) {
                const int idx = sxs + min(max(zcell[it], ylo), yhi) * M.ky;
                zr[k][it] = *reinterpret_cast<const u32x4*>(zptr[it] + (int64_t)idx * RBZ);
            }
            // every lane loads (a valid byte), which keeps the number of loads per step fixed
            mr[k] = mrow[sxs + min(max(min((int)threadIdx.x, NT * 16 - 1), ylo), yhi) * M.ky];
        }
    };
    // Register set k -> LDS buffers of diagonal s's parity.
    auto stage_in = [&](int s, int k) {
#pragma unroll
        for (int it = 0; it < NITZ; ++it) zst[s & 1][it * NTH + threadIdx.x] = zr[k][it];
        if constexpr (STAGE) mst[s & 1][threadIdx.x] = mr[k];
    };

    // Write back the outputs staged by diagonal sp. Every lane stores in every
    // pass (rows outside the diagonal repeat its nearest cell, which writes
    // the same bytes twice), so the number of stores is fixed. All LDS reads
    // are issued before the first store: one LDS round trip.
    constexpr int NITF = STAGE ? (NT * 16 * Q::QF + NTH - 1) / NTH : 0;
    // The lane's chunk of each write-back pass: cell row, chunk index in the
    // staged row and bytes per canvas cell of its tensor (gates, outputs or
    // cell states) packed as rowbytes << 8 | chunk, and its address at idx = 0.
    int fcell[NITF > 0 ? NITF : 1], fcr[NITF > 0 ? NITF : 1];
    char* fptr[NITF > 0 ? NITF : 1];
#pragma unroll
    for (int it = 0; it < NITF; ++it) {
        const int i = min(it * NTH + (int)threadIdx.x, NT * 16 * Q::QF - 1);
        const int r = i % Q::QF;
        fcell[it] = i / Q::QF;
        if (r < Q::QZ) {
            fptr[it] = reinterpret_cast<char*>(Z + d * G) + 16 * r + M.c0 * RBZ;
            fcr[it] = RBZ << 8 | r;
        } else if (r < Q::QZ + Q::QY) {
            fptr[it] = reinterpret_cast<char*>(Y + d * H) + 16 * (r - Q::QZ) + M.c0 * (4 * H * (int)sizeof(T));
            fcr[it] = (4 * H * (int)sizeof(T)) << 8 | r;
        } else {
            fptr[it] = reinterpret_cast<char*>(Cs + d * H) + 16 * (r - Q::QZ - Q::QY) + M.c0 * (16 * H);
            fcr[it] = (16 * H) << 8 | r;
        }
    }
    auto flush_read = [&](int sp, u32x4 (&v)[NITF > 0 ? NITF : 1]) {
        const int ylo = max(0, sp - R.w + 1), yhi = min(R.h - 1, sp);
#pragma unroll
        for (int it = 0; it < NITF; ++it) v[it] = ostage[min(max(fcell[it], ylo), yhi)][fcr[it] & 255];
    };
    auto flush_store = [&](int sp, const u32x4 (&v)[NITF > 0 ? NITF : 1]) {
        const int ylo = max(0, sp - R.w + 1), yhi = min(R.h - 1, sp);
        const int sxs = M.sx * sp;
#pragma unroll
        for (int it = 0; it < NITF; ++it) {
            const int cell = min(max(fcell[it], ylo), yhi);
            *reinterpret_cast<u32x4*>(fptr[it] + (int64_t)(sxs + cell * M.ky) * (fcr[it] >> 8)) = v[it];
        }
    };
    auto flush = [&](int sp) {
        if constexpr (STAGE) {
            u32x4 v[NITF > 0 ? NITF : 1];
            flush_read(sp, v);
            flush_store(sp, v);
        }
    };

    // Recurrent contraction of step s on MFMA from [h_L ; h_T] of the previous
    // diagonal: the lane's own sigmoid gates (acc) and this wave's reduction
    // slice of the candidate tile (ag). Staged, tiles outside the diagonal are
    // computed too (their results are not used), which keeps a step's MFMAs
    // in one block with the memory work issued behind them; otherwise they
    // are skipped.
    constexpr bool SKIP = !STAGE;
    auto mma = [&](int s, floatx4 (&acc)[TPG][WQ], floatx4 (&ag)[TPG]) {
        const int prv = (s & 1) ^ 1;
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
#pragma unroll
        for (int lt = 0; lt < TPG; ++lt) {
            const int nt = tg + NG * lt;
            if (SKIP && (16 * nt > yhi || 16 * nt + 15 < ylo)) continue;  // uniform over the workgroup
            const int yy = 16 * nt + n16;
            const T* brow = (q < 2) ? &hbuf[prv][yy + 1][q * KRUN] : &hbuf[prv][yy][(q - 2) * KRUN];
            Op bop[NSTEP], bg[GSTEP];
            lds_run<T, NSTEP>(brow, bop);
            lds_run<T, GSTEP>(brow + sp * GSTEP * O::PER, bg);
            ag[lt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < GSTEP; ++ks) ag[lt] = O::mma(Ag[ks], bg[ks], ag[lt]);
#pragma unroll
            for (int wq = 0; wq < WQ; ++wq) acc[lt][wq] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < NSTEP; ++ks)
#pragma unroll
                for (int wq = 0; wq < WQ; ++wq) acc[lt][wq] = O::mma(Aown[wq][ks], bop[ks], acc[lt][wq]);
        }
    };
    // The candidate slices go to LDS for the cell phase to sum.
    auto partials = [&](int s, const floatx4 (&ag)[TPG]) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
        const int j0 = 16 * gt + 4 * q;
#pragma unroll
        for (int lt = 0; lt < TPG; ++lt) {
            const int nt = tg + NG * lt;
            if (SKIP && (16 * nt > yhi || 16 * nt + 15 < ylo)) continue;
            const int yy = 16 * nt + n16;
            if (j0 < H) {
                *reinterpret_cast<float2*>(&gpart[sp][yy][j0]) = make_float2(ag[lt][0], ag[lt][1]);
                *reinterpret_cast<float2*>(&gpart[sp][yy][j0 + 2]) = make_float2(ag[lt][2], ag[lt][3]);
            }
        }
    };
    // Inputs of the cell updates of step s that are ready before its
    // contraction: the pre-activations and the top neighbours' cell states.
    auto pre_read = [&](int s, const FPre<TPG, WQ, T>& b, float (&zv)[TPG][WQ][5], float (&ct)[TPG][WQ],
                        uint32_t (&mk)[TPG]) {
        const int prv = (s & 1) ^ 1;
#pragma unroll
        for (int lt = 0; lt < TPG; ++lt) {
            const int nt = tg + NG * lt;
            const int yy = 16 * nt + n16;
            if constexpr (STAGE)
                mk[lt] = mst[s & 1][yy];
            else
                mk[lt] = b.m[lt];
#pragma unroll
            for (int wq = 0; wq < WQ; ++wq) {
                const int j = 4 * (w * WQ + wq) + q;
#pragma unroll
                for (int t = 0; t < 5; ++t) {
                    if constexpr (STAGE)
                        zv[lt][wq][t] = ld1f<T>(reinterpret_cast<const T*>(&zst[s & 1][yy * PZ]) + t * H + j);
                    else
                        zv[lt][wq][t] = ld1f<T>(&b.z[lt][wq][t]);
                }
                ct[lt][wq] = cbuf[prv][yy][j];
            }
        }
    };
    // Cell updates: the lane owns (cell 16 nt + n16, hidden unit 4 (w WQ + wq) + q).
    auto update = [&](int s, const FPre<TPG, WQ, T>& b, const floatx4 (&acc)[TPG][WQ], const float (&zv0)[TPG][WQ][5],
                      const float (&ct)[TPG][WQ], const uint32_t (&mk)[TPG]) {
        const int cur = s & 1, prv = cur ^ 1;
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
#pragma unroll
        for (int lt = 0; lt < TPG; ++lt) {
            const int nt = tg + NG * lt;
            if (16 * nt > yhi || 16 * nt + 15 < ylo) continue;
            const int yy = 16 * nt + n16;
#pragma unroll
            for (int wq = 0; wq < WQ; ++wq) {
                const int j = 4 * (w * WQ + wq) + q;
                float cn = 0.0f, hn = 0.0f;
                if (yy >= ylo && yy <= yhi) {
                    const float* zv = zv0[lt][wq];
                    float gs = 0.0f;
#pragma unroll
                    for (int k = 0; k < SPL; ++k) gs += gpart[k][yy][j];
                    const float gi = sigm_fast(acc[lt][wq][0] + zv[0]);
                    const float gfl = sigm_fast(acc[lt][wq][1] + zv[1]);
                    const float gft = sigm_fast(acc[lt][wq][2] + zv[2]);
                    const float go = sigm_fast(acc[lt][wq][3] + zv[3]);
                    const float gg = tanh_fast(gs + zv[4]);
                    cn = gi * gg + gfl * cprev[lt][wq] + gft * ct[lt][wq];
                    hn = go * tanh_fast(cn);
                    if (!mk[lt]) {
                        cn = 0.0f;
                        hn = 0.0f;
                    }
                    if constexpr (STAGE) {
                        T* oz = reinterpret_cast<T*>(&ostage[yy][0]);
                        oz[0 * H + j] = from_f<T>(gi);
                        oz[1 * H + j] = from_f<T>(gfl);
                        oz[2 * H + j] = from_f<T>(gft);
                        oz[3 * H + j] = from_f<T>(go);
                        oz[4 * H + j] = from_f<T>(gg);
                        oz[5 * H + j] = from_f<T>(hn);
                        reinterpret_cast<float*>(&ostage[yy][Q::QZ + Q::QY])[j] = cn;
                    } else {
                        const int64_t p = b.p[lt];
                        if (mk[lt]) {
                            T* zp = Z + p * (4 * G) + d * G + j;
                            zp[0 * H] = from_f<T>(gi);
                            zp[1 * H] = from_f<T>(gfl);
                            zp[2 * H] = from_f<T>(gft);
                            zp[3 * H] = from_f<T>(go);
                            zp[4 * H] = from_f<T>(gg);
                            Y[p * (4 * H) + d * H + j] = from_f<T>(hn);
                        }
                        Cs[p * (4 * H) + d * H + j] = cn;
                    }
                }
                cprev[lt][wq] = cn;
                hbuf[cur][yy + 1][j] = from_f<T>(hn);
                cbuf[cur][yy + 1][j] = cn;
            }
        }
    };
    auto compute = [&](int s, const FPre<TPG, WQ, T>& b) {
        floatx4 acc[TPG][WQ], ag[TPG];
        float zv[TPG][WQ][5], ct[TPG][WQ];
        uint32_t mk[TPG];
        pre_read(s, b, zv, ct, mk);
        mma(s, acc, ag);
        partials(s, ag);
        lds_barrier();
        update(s, b, acc, zv, ct, mk);
        lds_barrier();
    };

    lds_barrier();
    FPre<TPG, WQ, T> b0, b1;
    if constexpr (STAGE) {
        // Step s: the MFMAs first, then the LDS reads that the previous step
        // made ready (the outputs of step s - 1 to write back, the
        // pre-activations and mask bytes staged for step s, the top cell
        // states); behind them the registers loaded for step s + 1 PFD steps
        // ago go to LDS, the loads of step s + 1 + PFD are issued into them
        // (past the last step they re-read valid cells) and step s - 1 is
        // written back; the candidate partials go to LDS once their MFMAs are
        // done; then the cell phase. Two steps of prefetch cover the load
        // latency when the whole chip streams to and from memory.
        auto step = [&](int s, int k, auto with_flush) {
            constexpr bool WF = decltype(with_flush)::value;
            floatx4 acc[TPG][WQ], ag[TPG];
            mma(s, acc, ag);
            u32x4 fv[NITF > 0 ? NITF : 1];
            if constexpr (WF) flush_read(s - 1, fv);
            float zv[TPG][WQ][5], ct[TPG][WQ];
            uint32_t mk[TPG];
            pre_read(s, b0, zv, ct, mk);
            stage_in(s + 1, k);
            fetch_z(s + 1 + PFD, k);
            if constexpr (WF) flush_store(s - 1, fv);
            partials(s, ag);
            lds_barrier();
            update(s, b0, acc, zv, ct, mk);
            lds_barrier();
        };
        constexpr int K1 = PFD - 1;  // register set of diagonals sb + 1, sb + 3, ...
        fetch_z(sb, 0);
        stage_in(sb, 0);
        fetch_z(sb + PFD, 0);
        if constexpr (PFD == 2) fetch_z(sb + 1, 1);
        lds_barrier();
        step(sb, K1, std::false_type{});
        int s = sb + 1;
        for (; s + 1 < se; s += 2) {
            step(s, 0, std::true_type{});
            step(s + 1, K1, std::true_type{});
        }
        if (s < se) step(s, 0, std::true_type{});
        flush(se - 1);
    } else if constexpr (Prefetch2<T>::template on<TPG, WQ>()) {
        fetch(sb, b0);
        int s = sb;
        for (; s + 1 < se; s += 2) {
            fetch(s + 1, b1);
            compute(s, b0);
            fetch(s + 2, b0);
            compute(s + 1, b1);
        }
        if (s < se) compute(s, b0);
    } else {
        for (int s = sb; s < se; ++s) {
            fetch(s, b0);
            compute(s, b0);
        }
    }
}

// ---------------------------------------------------------------------------
// Forward for wide layers (bf16, H = 128: four quads per wave, where the
// staged kernel's LDS buffers do not fit and its registers spill).
//
// Lane 16q + n of wave w owns the four consecutive hidden units
// u0 = 16w + 4q .. u0 + 3 of cell n of a tile. The rows of own MFMA tile k
// are ordered (unit offset jj, gate) -> U row gate*H + 16w + 4jj + k, so the
// lane ends with the four sigmoid gates of unit u0 + k in tile k; the rows of
// the candidate tile are the wave's sixteen units in order, so its register
// k is the candidate of unit u0 + k. No value crosses lanes: the cell update
// follows each tile's MFMAs without a barrier, both neighbours' cell states
// come from LDS, and pre-activations arrive as 8-byte vectors. Tiles of a
// diagonal run one after another (the accumulators of one tile only), their
// pre-activations loaded two tiles ahead. The diagonal's gates, outputs and
// cell states are left in LDS and, after a barrier, written back by the whole
// workgroup as contiguous 16-byte chunks (a lane's own values would be
// 8-byte pieces of sixteen canvas rows per store).
// ---------------------------------------------------------------------------
// Target of the gate-gradient stores of lanes whose cell is outside the
// diagonal in the wide-layer backward: every lane stores on every path, so the
// number of memory operations in flight is the same on all paths and the
// compiler waits for exactly the loads it needs (a skipped store would make it
// wait for everything). 1536 bytes per lane (room for a cell's gate gradients
// of one direction), shared by workgroups eight apart; never read.
constexpr int SINK_LANE = 96;  // 16-byte slots per lane
__device__ __attribute__((aligned(256))) uint4 g_wave_sink[8 * 64 * SINK_LANE];

template <typename T>
__device__ __forceinline__ T* wave_sink() {
    return reinterpret_cast<T*>(&g_wave_sink[((blockIdx.x & 7) * 64 + (threadIdx.x & 63)) * SINK_LANE]);
}

template <int H, typename T>
struct FwdBig {
    static constexpr bool on = sizeof(T) == 2 && Geo<H, T>::NW == 8 && Geo<H, T>::WQ == 4;
};

template <int H, int NT, typename T>
__device__ __forceinline__ void wave_fwd_big(const WaveArgs& a, const int unit) {
    using O = Ops<T>;
    using Op = typename O::Op;
    constexpr int G = 5 * H, KRUN = H / 2, NSTEP = KRUN / O::PER, NTH = 512;
    constexpr int ROWS = NT * 16 + 1;            // row 0: zero row above local row 0
    constexpr int HP = H + 16 / (int)sizeof(T);  // padded LDS row pitches
    constexpr int CP = H + 4;
    constexpr int GP = G + 16 / (int)sizeof(T);
    // 16-byte chunks of a cell's outputs: gates, output, cell state
    constexpr int QZ = G * (int)sizeof(T) / 16, QY = H * (int)sizeof(T) / 16, QC = H * 4 / 16;
    constexpr int QF = QZ + QY + QC, NPS = NT * 16 * QF / NTH;
    static_assert(NT * 16 * QF % NTH == 0, "store passes");
    __shared__ __attribute__((aligned(16))) T hbuf[2][ROWS][HP];
    // Cell states of the previous diagonal, overwritten row by row by the
    // current one: the tiles run from the bottom up, so a tile never
    // overwrites a row that a later tile of the diagonal still reads (a
    // lane's hidden units are its wave's columns, read before written).
    __shared__ __attribute__((aligned(16))) float cbuf[ROWS][CP];
    __shared__ __attribute__((aligned(16))) T gst[NT * 16][GP];  // activated gates of the diagonal

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int q = lane >> 4, n16 = lane & 15;
    const int u0 = 16 * w + 4 * q;
    const int d = unit & 3;
    const RectD R = reinterpret_cast<const RectD*>(a.rects)[unit >> 2];
    const T* __restrict__ U = static_cast<const T*>(a.u) + (int64_t)d * G * 2 * H;
    T* __restrict__ Z = static_cast<T*>(a.z);
    T* __restrict__ Y = static_cast<T*>(a.y);
    float* __restrict__ Cs = a.c;
    const int steps = R.h + R.w - 1;
    const int sb = a.s0, se = min(a.s1, steps);
    if (sb >= se) return;

    for (int i = threadIdx.x; i < 2 * ROWS * HP; i += blockDim.x) (&hbuf[0][0][0])[i] = T(0);
    for (int i = threadIdx.x; i < ROWS * CP; i += blockDim.x) (&cbuf[0][0])[i] = 0.0f;
    if (sb > 0) {  // state of diagonal sb - 1 from the previous launch's outputs
        lds_barrier();  // every zero written before the read-back fills the same rows
        const int pb = (sb & 1) ^ 1;
        for (int i = threadIdx.x; i < NT * 16 * H; i += blockDim.x) {
            const int yy = i / H, j = i - yy * H, xx = sb - 1 - yy;
            if (yy < R.h && xx >= 0 && xx < R.w) {
                const int64_t p = canvas_index(R, d, yy, xx, a.canvas_w);
                hbuf[pb][yy + 1][j] = Y[p * (4 * H) + d * H + j];
                cbuf[yy + 1][j] = Cs[p * (4 * H) + d * H + j];
            }
        }
    }

    Op Aown[4][NSTEP], Ag[NSTEP];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int row = (n16 & 3) * H + 16 * w + 4 * (n16 >> 2) + k;
        load_slot<T, NSTEP>(U + (int64_t)row * 2 * H + q * KRUN, 1, true, Aown[k]);
    }
    load_slot<T, NSTEP>(U + (int64_t)(4 * H + 16 * w + n16) * 2 * H + q * KRUN, 1, true, Ag);
    __builtin_amdgcn_s_waitcnt(0);

    const DiagMap M(R, d, a.canvas_w);
    const uint8_t* mrow = a.mask + M.c0;
    const T* const zb = Z + M.c0 * (4 * G) + d * G + u0;  // the lane's pre-activations at idx = 0

    // Outputs of diagonal s, staged in LDS, written back as contiguous 16-byte
    // chunks (pass ps, thread t: chunk (ps * 512 + t) % QF of cell row slot
    // (ps * 512 + t) / QF); every thread stores in every pass (rows outside
    // the diagonal repeat its nearest cell, which writes the same bytes twice).
    char* const zd = reinterpret_cast<char*>(Z + d * G) + M.c0 * (4 * G * (int)sizeof(T));
    char* const yd = reinterpret_cast<char*>(Y + d * H) + M.c0 * (4 * H * (int)sizeof(T));
    char* const cd = reinterpret_cast<char*>(Cs + d * H) + M.c0 * (16 * H);
    auto write_back = [&](int s) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
        const int cur = s & 1, sxs = M.sx * s;
        constexpr int GR = 4;  // passes per LDS round trip (registers)
        static_assert(NPS % GR == 0, "pass groups");
#pragma unroll
        for (int p0 = 0; p0 < NPS; p0 += GR) {
            u32x4 v[GR];
#pragma unroll
            for (int k = 0; k < GR; ++k) {
                const int i = (p0 + k) * NTH + (int)threadIdx.x, r = i % QF;
                const int cell = min(max(i / QF, ylo), yhi);
                const u32x4* src = r < QZ        ? reinterpret_cast<const u32x4*>(&gst[cell][0]) + r
                                   : r < QZ + QY ? reinterpret_cast<const u32x4*>(&hbuf[cur][cell + 1][0]) + (r - QZ)
                                                 : reinterpret_cast<const u32x4*>(&cbuf[cell + 1][0]) + (r - QZ - QY);
                v[k] = *src;
            }
#pragma unroll
            for (int k = 0; k < GR; ++k) {
                const int i = (p0 + k) * NTH + (int)threadIdx.x, r = i % QF;
                const int64_t idx = sxs + min(max(i / QF, ylo), yhi) * M.ky;
                char* dst = r < QZ        ? zd + idx * (4 * G * (int)sizeof(T)) + 16 * r
                            : r < QZ + QY ? yd + idx * (4 * H * (int)sizeof(T)) + 16 * (r - QZ)
                                          : cd + idx * (16 * H) + 16 * (r - QZ - QY);
                *reinterpret_cast<u32x4*>(dst) = v[k];
            }
        }
    };

    // Pre-activations (5 gates x 4 units) and mask byte of the lane's cell of
    // tile nt of diagonal s; past the last diagonal, or for rows outside the
    // diagonal, a valid cell of the rectangle is read instead (fixed number of
    // loads on every path).
    auto load = [&](int s, int nt, uint2 (&zr)[5], uint32_t& m) {
        const int sc = min(s, se - 1);
        const int ylo = max(0, sc - R.w + 1), yhi = min(R.h - 1, sc);
        const int idx = M.sx * sc + min(max(16 * nt + n16, ylo), yhi) * M.ky;
        const T* zp = zb + (int64_t)idx * (4 * G);
#pragma unroll
        for (int t = 0; t < 5; ++t) zr[t] = *reinterpret_cast<const uint2*>(zp + t * H);
        m = mrow[idx];
    };
    // Next tile of the walk: the next active tile up the diagonal, else the
    // bottom active tile of the next one.
    auto advance = [&](int& s, int& nt) {
        const int ylo = max(0, s - R.w + 1);
        if (16 * nt > ylo) {
            --nt;
        } else {
            ++s;
            nt = min(R.h - 1, s) >> 4;
        }
    };
    auto tile = [&](int s, int nt, const uint2 (&zr)[5], uint32_t m) {
        const int cur = s & 1, prv = cur ^ 1;
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
        const int yy = 16 * nt + n16;
        const T* brow = (q < 2) ? &hbuf[prv][yy + 1][q * KRUN] : &hbuf[prv][yy][(q - 2) * KRUN];
        floatx4 acc[4], ag = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[k] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NSTEP; ++ks) {
            const Op b = O::lds(brow + ks * O::PER);
            ag = O::mma(Ag[ks], b, ag);
#pragma unroll
            for (int k = 0; k < 4; ++k) acc[k] = O::mma(Aown[k][ks], b, acc[k]);
        }
        const float4 cl = *reinterpret_cast<const float4*>(&cbuf[yy + 1][u0]);
        const float4 ct = *reinterpret_cast<const float4*>(&cbuf[yy][u0]);
        const float clv[4] = {cl.x, cl.y, cl.z, cl.w}, ctv[4] = {ct.x, ct.y, ct.z, ct.w};
        const bool live = yy >= ylo && yy <= yhi && m != 0;
        float gv[5][4], hv[4], cv[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            float zv[5];
#pragma unroll
            for (int t = 0; t < 5; ++t) {
                const uint32_t wd = (k < 2) ? zr[t].x : zr[t].y;
                zv[t] = __uint_as_float((k & 1) ? (wd & 0xffff0000u) : (wd << 16));
            }
            gv[0][k] = sigm_fast(acc[k][0] + zv[0]);
            gv[1][k] = sigm_fast(acc[k][1] + zv[1]);
            gv[2][k] = sigm_fast(acc[k][2] + zv[2]);
            gv[3][k] = sigm_fast(acc[k][3] + zv[3]);
            gv[4][k] = tanh_fast(ag[k] + zv[4]);
            const float cn = gv[0][k] * gv[4][k] + gv[1][k] * clv[k] + gv[2][k] * ctv[k];
            const float hn = gv[3][k] * tanh_fast(cn);
            cv[k] = live ? cn : 0.0f;
            hv[k] = live ? hn : 0.0f;
        }
        auto pack = [](const float (&v)[4]) {
            return make_uint2(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]));
        };
        *reinterpret_cast<uint2*>(&hbuf[cur][yy + 1][u0]) = pack(hv);
        *reinterpret_cast<float4*>(&cbuf[yy + 1][u0]) = make_float4(cv[0], cv[1], cv[2], cv[3]);
#pragma unroll
        for (int t = 0; t < 5; ++t) *reinterpret_cast<uint2*>(&gst[yy][t * H + u0]) = pack(gv[t]);
        if (16 * nt <= ylo) {  // top tile of the diagonal: publish it, write it back
            lds_barrier();
            write_back(s);
            lds_barrier();
        }
    };

    lds_barrier();
    uint2 z0[5], z1[5];
    uint32_t m0, m1;
    int s = sb, nt = min(R.h - 1, sb) >> 4;
    int ls = s, lnt = nt;
    load(ls, lnt, z0, m0);
    advance(ls, lnt);
    load(ls, lnt, z1, m1);
    advance(ls, lnt);
    for (;;) {
        tile(s, nt, z0, m0);
        load(ls, lnt, z0, m0);
        advance(ls, lnt);
        advance(s, nt);
        if (s >= se) break;
        tile(s, nt, z1, m1);
        load(ls, lnt, z1, m1);
        advance(ls, lnt);
        advance(s, nt);
        if (s >= se) break;
    }
}

// ---------------------------------------------------------------------------
// Backward (reverse anti-diagonals). With successors S (right, same row, next
// diagonal) and E (below, row + 1, next diagonal):
//   dh = dY + (U^T da_S)[0:H] + (U^T da_E)[H:2H]
//   dc = dh o (1 - tanh^2 c) + dc_S f_L(S) + dc_E f_T(E)
//   da = (dc g i(1-i), dc c_L f_L(1-f_L), dc c_T f_T(1-f_T), dh tanh(c) o(1-o), dc i (1-g^2))
// ---------------------------------------------------------------------------
template <int H, int NT, typename T>
__device__ __forceinline__ void wave_bwd_unit(const WaveArgs& a, const int unit) {
    using Gm = Geo<H, T>;
    using O = Ops<T>;
    using Op = typename O::Op;
    using Q = OutQ<H, T>;
    // tile groups as in the forward: group tg owns tiles tg, tg + NG, ...
    constexpr int NG = TileGroups<H, NT, T>::NG, TPG = NT / NG;
    constexpr int WQ = Gm::WQ, G = Gm::G, KRUNB = Gm::KRUNB, NTH = 64 * Gm::NW * NG;
    constexpr int TPW = Gm::TPW, SPLB = Gm::SPLB, BSTEP = Gm::BSTEP;
    constexpr int GP = G + 16 / (int)sizeof(T);
    // Staged: the gates, upstream gradients and cell states of a diagonal are
    // loaded as contiguous 16-byte chunks into registers two steps ahead and
    // kept in LDS for two steps (own cells, then left/top predecessors of the
    // next diagonal). Otherwise every lane loads its own values.
    constexpr bool STAGE = bwd_stage<H, NT, T>();
    constexpr int PB = STAGE ? Q::QF + 1 : 1;  // row pitch in chunks; the extra chunk spreads LDS banks
    constexpr int NSL = STAGE ? (NT * 16 * PB + NTH - 1) / NTH * NTH : 1;
    constexpr int NITZ = STAGE ? NSL / NTH : 0;
    constexpr int NITF = (NT * 16 * Q::QZ + NTH - 1) / NTH;  // passes writing back the gate gradients
    constexpr int CC = Q::QZ + Q::QY;                        // first cell-state chunk of a row
    __shared__ __attribute__((aligned(16))) T dabuf[NT * 16][GP];
    // row NT*16 stays zero; row NT*16 + 1 takes the writes of tiles outside
    // the diagonal (and of padding columns), which nobody reads
    __shared__ __attribute__((aligned(16))) float gbuf[SPLB][NT * 16 + 2][2 * H + 2];
    __shared__ __attribute__((aligned(16))) float dct[NT * 16 + 2][H + 2];
    __shared__ __attribute__((aligned(16))) u32x4 ist[STAGE ? 2 : 1][NSL];

    const int lane = threadIdx.x & 63;
    const int tg = NG == 1 ? 0 : (int)(threadIdx.x >> 6) / Gm::NW;
    const int w = NG == 1 ? (int)(threadIdx.x >> 6) : (int)(threadIdx.x >> 6) % Gm::NW;
    const int q = lane >> 4, n16 = lane & 15;
    const int mt0 = (w / SPLB) * TPW, sb = w % SPLB;  // output tiles and reduction slice of this wave
    const int d = unit & 3;
    const RectD R = reinterpret_cast<const RectD*>(a.rects)[unit >> 2];
    const T* __restrict__ U = static_cast<const T*>(a.u) + (int64_t)d * G * 2 * H;
    T* __restrict__ Z = static_cast<T*>(a.z);
    const T* __restrict__ DY = static_cast<const T*>(a.dy);
    const float* __restrict__ Cs = a.c;
    const int steps = R.h + R.w - 1;

    for (int i = threadIdx.x; i < NT * 16 * GP; i += blockDim.x) (&dabuf[0][0])[i] = T(0);
    for (int i = threadIdx.x; i < SPLB * (NT * 16 + 2) * (2 * H + 2); i += blockDim.x) (&gbuf[0][0][0])[i] = 0.0f;
    for (int i = threadIdx.x; i < (NT * 16 + 2) * (H + 2); i += blockDim.x) (&dct[0][0])[i] = 0.0f;

    // A operands: U^T rows k = 16 mt + n16 (column k of U); slot q holds gate
    // rows r = q*KRUNB + ..., slice sb of the K steps.
    Op A[TPW][BSTEP];
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
        const int k = 16 * (mt0 + tt) + n16;
        const bool ok = k < 2 * H;
        load_slot<T, BSTEP>(U + (int64_t)(q * KRUNB + sb * BSTEP * O::PER) * 2 * H + (ok ? k : 0), 2 * H, ok, A[tt]);
    }
    float dcl[TPG][WQ], dcn[TPG][WQ];
#pragma unroll
    for (int lt = 0; lt < TPG; ++lt)
#pragma unroll
        for (int wq = 0; wq < WQ; ++wq) dcl[lt][wq] = dcn[lt][wq] = 0.0f;
    __builtin_amdgcn_s_waitcnt(0);  // U operands in registers before the step loop

    // Cells of diagonal s, their mask bytes and (unstaged) the lane's inputs,
    // issued for every lane from valid cells (see the forward pass);
    // predecessors outside the rectangle read the cell itself and are zeroed
    // on use.
    const DiagMap M(R, d, a.canvas_w);
    auto fetch = [&](int s, BPre<TPG, WQ, T>& b) {
        const int sc = max(s, 0);
        const int ylo = max(0, sc - R.w + 1), yhi = min(R.h - 1, sc);
        const int64_t base = M.base(sc);
#pragma unroll
        for (int lt = 0; lt < TPG; ++lt) {
            const int yy = 16 * (tg + NG * lt) + n16;
            b.live[lt] = s >= 0 && yy >= ylo && yy <= yhi;
            const int yc = min(max(yy, ylo), yhi), xc = sc - yc;
            const int64_t p = M.at(base, yc);
            b.p[lt] = p;
            b.m[lt] = a.mask[p];
            b.hasl[lt] = xc > 0;
            b.hast[lt] = yc > 0;
            if constexpr (!STAGE) {
                const int64_t pl = xc > 0 ? canvas_index(R, d, yc, xc - 1, a.canvas_w) : p;
                const int64_t pt = yc > 0 ? canvas_index(R, d, yc - 1, xc, a.canvas_w) : p;
#pragma unroll
                for (int wq = 0; wq < WQ; ++wq) {
                    const int j = 4 * (w * WQ + wq) + q;
                    const T* zp = Z + p * (4 * G) + d * G + j;
#pragma unroll
                    for (int t = 0; t < 5; ++t) b.g[lt][wq][t] = zp[t * H];
                    b.dy[lt][wq] = DY[p * (4 * H) + d * H + j];
                    b.c[lt][wq] = Cs[p * (4 * H) + d * H + j];
                    b.cl[lt][wq] = Cs[pl * (4 * H) + d * H + j];
                    b.ct[lt][wq] = Cs[pt * (4 * H) + d * H + j];
                }
            }
        }
    };

    // Staged rows of diagonal s (clamped at 0) into zr: slot S is chunk S % PB
    // of the row of cell S / PB, a row being the 5H gates, the H upstream
    // gradients and the H cell states of the cell (padding chunk and slots
    // past the last cell repeat a valid chunk).
    u32x4 zr[NITZ > 0 ? NITZ : 1];
    // The lane's chunk of each staged-input pass: cell row, and the chunk's
    // address at canvas index 0 with the bytes per canvas cell of its tensor.
    int zcell[NITZ > 0 ? NITZ : 1], zrb[NITZ > 0 ? NITZ : 1];
    const char* zsrc[NITZ > 0 ? NITZ : 1];
#pragma unroll
    for (int it = 0; it < NITZ; ++it) {
        const int S = it * NTH + (int)threadIdx.x;
        const int r = min(S % PB, Q::QF - 1);
        zcell[it] = min(S / PB, NT * 16 - 1);
        if (r < Q::QZ) {
            zsrc[it] = reinterpret_cast<const char*>(Z + d * G) + 16 * r;
            zrb[it] = 4 * G * (int)sizeof(T);
        } else if (r < CC) {
            zsrc[it] = reinterpret_cast<const char*>(DY + d * H) + 16 * (r - Q::QZ);
            zrb[it] = 4 * H * (int)sizeof(T);
        } else {
            zsrc[it] = reinterpret_cast<const char*>(Cs + d * H) + 16 * (r - CC);
            zrb[it] = 16 * H;
        }
    }
    auto fetch_rows = [&](int s) {
        if constexpr (STAGE) {
            const int sc = max(s, 0);
            const int ylo = max(0, sc - R.w + 1), yhi = min(R.h - 1, sc);
            const int64_t base = M.base(sc);
#pragma unroll
            for (int it = 0; it < NITZ; ++it) {
                const int yc = min(max(zcell[it], ylo), yhi);
                zr[it] = *reinterpret_cast<const u32x4*>(zsrc[it] + M.at(base, yc) * zrb[it]);
            }
        }
    };
    auto stage_in = [&](int s) {
#pragma unroll
        for (int it = 0; it < NITZ; ++it) ist[s & 1][it * NTH + threadIdx.x] = zr[it];
    };

    // The lane's chunk of each gate-gradient write-back pass (cell row, chunk).
    int dcell[NITF], dchunk[NITF];
#pragma unroll
    for (int it = 0; it < NITF; ++it) {
        const int i = min(it * NTH + (int)threadIdx.x, NT * 16 * Q::QZ - 1);
        dcell[it] = i / Q::QZ;
        dchunk[it] = i - dcell[it] * Q::QZ;
    }
    char* const Zd = reinterpret_cast<char*>(Z + d * G);
    auto compute = [&](int s, const BPre<TPG, WQ, T>& b) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
        // Phase A: gate-gradient update of this lane's (cell, hidden unit) pairs.
#pragma unroll
        for (int lt = 0; lt < TPG; ++lt) {
            const int nt = tg + NG * lt;
            if (16 * nt > yhi || 16 * nt + 15 < ylo) continue;
            const int yy = 16 * nt + n16;
#pragma unroll
            for (int wq = 0; wq < WQ; ++wq) {
                const int j = 4 * (w * WQ + wq) + q;
                float da[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
                float ndl = 0.0f, ndt = 0.0f;
                if (b.live[lt] && b.m[lt]) {
                    float g[5], dyv, cv, cL, cT;
                    if constexpr (STAGE) {
                        const T* row = reinterpret_cast<const T*>(&ist[s & 1][yy * PB]);
#pragma unroll
                        for (int t = 0; t < 5; ++t) g[t] = ld1f<T>(row + t * H + j);
                        dyv = ld1f<T>(row + 5 * H + j);
                        cv = reinterpret_cast<const float*>(&ist[s & 1][yy * PB + CC])[j];
                        const u32x4* prv = &ist[(s - 1) & 1][0];
                        cL = b.hasl[lt] ? reinterpret_cast<const float*>(prv + yy * PB + CC)[j] : 0.0f;
                        cT = b.hast[lt] ? reinterpret_cast<const float*>(prv + max(yy - 1, 0) * PB + CC)[j] : 0.0f;
                    } else {
#pragma unroll
                        for (int t = 0; t < 5; ++t) g[t] = ld1f<T>(&b.g[lt][wq][t]);
                        dyv = ld1f<T>(&b.dy[lt][wq]);
                        cv = b.c[lt][wq];
                        cL = b.hasl[lt] ? b.cl[lt][wq] : 0.0f;
                        cT = b.hast[lt] ? b.ct[lt][wq] : 0.0f;
                    }
                    const float gi = g[0], gfl = g[1], gft = g[2], go = g[3], gg = g[4];
                    float gl = 0.0f, gtv = 0.0f;
#pragma unroll
                    for (int k = 0; k < SPLB; ++k) {
                        gl += gbuf[k][yy][j];
                        gtv += gbuf[k][yy + 1][H + j];
                    }
                    const float dh = dyv + gl + gtv;
                    const float tc = tanh_fast(cv);
                    const float dc = dcl[lt][wq] + dct[yy + 1][j] + dh * go * (1.0f - tc * tc);
                    da[0] = dc * gg * gi * (1.0f - gi);
                    da[1] = dc * cL * gfl * (1.0f - gfl);
                    da[2] = dc * cT * gft * (1.0f - gft);
                    da[3] = dh * tc * go * (1.0f - go);
                    da[4] = dc * gi * (1.0f - gg * gg);
                    ndl = dc * gfl;
                    ndt = dc * gft;
                }
#pragma unroll
                for (int t = 0; t < 5; ++t) dabuf[yy][t * H + j] = from_f<T>(da[t]);
                dcl[lt][wq] = ndl;
                dcn[lt][wq] = ndt;
            }
        }
        lds_barrier();
        // Phase B: U^T da for the left (rows k < H) and top (k >= H)
        // predecessors, on MFMA; issued first so that the memory work below
        // runs behind it. Staged, tiles outside the diagonal are computed too
        // (their results are not used), which keeps the MFMAs in one block.
        floatx4 acc[TPG][TPW];
#pragma unroll
        for (int lt = 0; lt < TPG; ++lt) {
            const int nt = tg + NG * lt;
            if (!STAGE && (16 * nt > yhi || 16 * nt + 15 < ylo)) continue;
            const int yy = 16 * nt + n16;
            const T* brow = &dabuf[yy][q * KRUNB + sb * BSTEP * O::PER];
            Op bop[BSTEP];
            lds_run<T, BSTEP>(brow, bop);
#pragma unroll
            for (int tt = 0; tt < TPW; ++tt) {
                acc[lt][tt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < BSTEP; ++ks) acc[lt][tt] = O::mma(A[tt][ks], bop[ks], acc[lt][tt]);
            }
        }
        // The rows of dabuf are the gate gradients of the diagonal's cells:
        // write them back with contiguous 16-byte stores. Every lane stores in
        // every pass (rows outside the diagonal repeat its nearest cell; cells
        // with mask 0 get zero gradients), so the number of stores is fixed.
        {
            const int64_t base = M.base(s);
            u32x4 v[NITF];
            char* dst[NITF];
#pragma unroll
            for (int it = 0; it < NITF; ++it) {
                const int cell = min(max(dcell[it], ylo), yhi);
                v[it] = reinterpret_cast<const u32x4*>(&dabuf[cell][0])[dchunk[it]];
                dst[it] = Zd + M.at(base, cell) * (4 * G * (int)sizeof(T)) + 16 * dchunk[it];
            }
            // Staged rows of diagonal s - 2 replace those of diagonal s, which
            // no lane reads any more; the rows of diagonal s - 3 start loading.
            if constexpr (STAGE) {
                stage_in(s - 2);
                fetch_rows(s - 3);
            }
            // non-temporal: the gate gradients are read again only by the
            // gradient GEMMs after the whole wavefront
#pragma unroll
            for (int it = 0; it < NITF; ++it) __builtin_nontemporal_store(v[it], reinterpret_cast<u32x4*>(dst[it]));
        }
        // The products and the dc of the top predecessors go to LDS without
        // branches (tiles outside the diagonal and padding columns write to
        // the unread last rows), so the MFMA results are read in the same
        // straight-line block that produced them.
#pragma unroll
        for (int lt = 0; lt < TPG; ++lt) {
            const int nt = tg + NG * lt;
            const bool act = !(16 * nt > yhi || 16 * nt + 15 < ylo);
            const int yy = act ? 16 * nt + n16 : NT * 16 + 1;
#pragma unroll
            for (int tt = 0; tt < TPW; ++tt) {
                const int k0 = 16 * (mt0 + tt) + 4 * q;
                float* gp = (act && k0 < 2 * H) ? &gbuf[sb][yy][k0] : &gbuf[sb][NT * 16 + 1][0];
                *reinterpret_cast<float2*>(gp) = make_float2(acc[lt][tt][0], acc[lt][tt][1]);
                *reinterpret_cast<float2*>(gp + 2) = make_float2(acc[lt][tt][2], acc[lt][tt][3]);
            }
#pragma unroll
            for (int wq = 0; wq < WQ; ++wq) dct[yy][act ? 4 * (w * WQ + wq) + q : 0] = dcn[lt][wq];
        }
        lds_barrier();
    };

    BPre<TPG, WQ, T> b0, b1;
    if constexpr (STAGE) {
        // Before step s: rows of diagonals s and s - 1 in LDS, rows of s - 2
        // loading, cells of s in registers.
        fetch_rows(steps - 1);
        stage_in(steps - 1);
        fetch_rows(steps - 2);
        stage_in(steps - 2);
        fetch_rows(steps - 3);
        fetch(steps - 1, b0);
        lds_barrier();
        auto step = [&](int s, const BPre<TPG, WQ, T>& cur, BPre<TPG, WQ, T>& nxt) {
            fetch(s - 1, nxt);
            compute(s, cur);
        };
        for (int s = steps - 1; s >= 0; s -= 2) {
            step(s, b0, b1);
            if (s - 1 >= 0) step(s - 1, b1, b0);
        }
    } else if constexpr (Prefetch2<T>::template on<TPG, WQ>()) {
        lds_barrier();
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
        lds_barrier();
        for (int s = steps - 1; s >= 0; --s) {
            fetch(s, b0);
            compute(s, b0);
        }
    }
}

// ---------------------------------------------------------------------------
// Backward for wide layers (bf16, H = 128), with the forward's lane mapping:
// lane 16q + n of wave w owns units u0 = 16w + 4q .. u0 + 3 of cell n of a
// tile. The wave computes the two U^T da output tiles of its own units, the
// left-predecessor part (rows u0 + r) and the top-predecessor part
// (rows H + u0 + r), so the left part lands in the lane that needs it on the
// next diagonal (the cell's left predecessor is on the same row) and stays in
// registers; the top part and dc f_T go one row up through LDS, within the
// wave. Only the gate gradients cross waves (all of them are the reduction
// operand), so a diagonal runs as segments [A(t0)] [B(t0) A(t1)] ... [B(t1)]
// with a barrier after each: A = gate-gradient update of a tile, B = its
// U^T da products on MFMA.
// ---------------------------------------------------------------------------
template <int H, typename T>
struct BwdBig {
    static constexpr bool on = sizeof(T) == 2 && Geo<H, T>::NW == 8 && Geo<H, T>::WQ == 4 && 2 * H == 256;
    static_assert(!on || 5 * H * sizeof(T) <= SINK_LANE * 16, "sink row");
};

template <int H, int NT, typename T>
__device__ __forceinline__ void wave_bwd_big(const WaveArgs& a, const int unit) {
    using O = Ops<T>;
    using Op = typename O::Op;
    constexpr int G = 5 * H, KRUNB = G / 4, NSTEPB = KRUNB / O::PER;
    constexpr int GP = G + 16 / (int)sizeof(T);  // padded LDS row pitches
    constexpr int CP = H + 4;
    __shared__ __attribute__((aligned(16))) T dabuf[NT * 16][GP];
    // per cell row: the top-predecessor part of U^T da, and dc f_T (row NT*16 stays zero)
    __shared__ __attribute__((aligned(16))) float gtop[NT * 16 + 1][CP];
    __shared__ __attribute__((aligned(16))) float dct[NT * 16 + 1][CP];

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int q = lane >> 4, n16 = lane & 15;
    const int u0 = 16 * w + 4 * q;
    const int d = unit & 3;
    const RectD R = reinterpret_cast<const RectD*>(a.rects)[unit >> 2];
    const T* __restrict__ U = static_cast<const T*>(a.u) + (int64_t)d * G * 2 * H;
    T* __restrict__ Z = static_cast<T*>(a.z);
    const T* __restrict__ DY = static_cast<const T*>(a.dy);
    const float* __restrict__ Cs = a.c;
    const int steps = R.h + R.w - 1;

    for (int i = threadIdx.x; i < NT * 16 * GP; i += blockDim.x) (&dabuf[0][0])[i] = T(0);
    for (int i = threadIdx.x; i < (NT * 16 + 1) * CP; i += blockDim.x) {
        (&gtop[0][0])[i] = 0.0f;
        (&dct[0][0])[i] = 0.0f;
    }
    // A operands: U^T rows k = u-part + 16w + n16 (column k of U); slot q
    // holds gate rows q*KRUNB + 8 ks + e.
    Op A[2][NSTEPB];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
        load_slot<T, NSTEPB>(U + (int64_t)(q * KRUNB) * 2 * H + tt * H + 16 * w + n16, 2 * H, true, A[tt]);
    floatx4 gl[NT], dcl[NT];  // left-successor parts of dh and dc, per tile row
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) gl[nt] = dcl[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
    __builtin_amdgcn_s_waitcnt(0);

    const DiagMap M(R, d, a.canvas_w);
    const uint8_t* mrow = a.mask + M.c0;
    T* const zb = Z + M.c0 * (4 * G) + d * G + u0;
    const T* const dyb = DY + M.c0 * (4 * H) + d * H + u0;
    const float* const cb = Cs + M.c0 * (4 * H) + d * H + u0;

    struct In {
        uint2 g[5], dy;
        float4 c, cl, ct;
        uint32_t m;
    };
    // Inputs of the lane's cell of tile nt of diagonal s (rows outside the
    // diagonal read its nearest cell; a missing predecessor reads the cell).
    auto load = [&](int s, int nt, In& in) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
        const int yc = min(max(16 * nt + n16, ylo), yhi), xc = s - yc;
        const int idx = M.sx * s + yc * M.ky;
        const int il = xc > 0 ? idx - M.sx : idx;
        const int it = yc > 0 ? idx - M.sx - M.ky : idx;
        const T* zp = zb + (int64_t)idx * (4 * G);
#pragma unroll
        for (int t = 0; t < 5; ++t) in.g[t] = *reinterpret_cast<const uint2*>(zp + t * H);
        in.dy = *reinterpret_cast<const uint2*>(dyb + (int64_t)idx * (4 * H));
        in.c = *reinterpret_cast<const float4*>(cb + (int64_t)idx * (4 * H));
        in.cl = *reinterpret_cast<const float4*>(cb + (int64_t)il * (4 * H));
        in.ct = *reinterpret_cast<const float4*>(cb + (int64_t)it * (4 * H));
        in.m = mrow[idx];
    };
    auto bf = [](const uint2& v, int k) {
        const uint32_t wd = (k < 2) ? v.x : v.y;
        return __uint_as_float((k & 1) ? (wd & 0xffff0000u) : (wd << 16));
    };
    auto pack = [](const float (&v)[4]) {
        return make_uint2(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]));
    };
    // Phase A of tile nt: gate gradients of the lane's four units.
    auto phase_a = [&](int s, int nt, const In& in) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
        const int yy = 16 * nt + n16;
        const bool inr = yy >= ylo && yy <= yhi;
        const bool live = inr && in.m != 0;
        const bool hasl = s - yy > 0, hast = yy > 0;
        const float4 gt4 = *reinterpret_cast<const float4*>(&gtop[yy + 1][u0]);
        const float4 dt4 = *reinterpret_cast<const float4*>(&dct[yy + 1][u0]);
        const float gtv[4] = {gt4.x, gt4.y, gt4.z, gt4.w}, dtv[4] = {dt4.x, dt4.y, dt4.z, dt4.w};
        const float cv4[4] = {in.c.x, in.c.y, in.c.z, in.c.w};
        const float cl4[4] = {in.cl.x, in.cl.y, in.cl.z, in.cl.w};
        const float ct4[4] = {in.ct.x, in.ct.y, in.ct.z, in.ct.w};
        float da[5][4], ndl[4], ndt[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float gi = bf(in.g[0], k), gfl = bf(in.g[1], k), gft = bf(in.g[2], k), go = bf(in.g[3], k),
                        gg = bf(in.g[4], k);
            const float cL = hasl ? cl4[k] : 0.0f, cT = hast ? ct4[k] : 0.0f;
            const float dh = bf(in.dy, k) + gl[nt][k] + gtv[k];
            const float tc = tanh_fast(cv4[k]);
            const float dc = dcl[nt][k] + dtv[k] + dh * go * (1.0f - tc * tc);
            da[0][k] = live ? dc * gg * gi * (1.0f - gi) : 0.0f;
            da[1][k] = live ? dc * cL * gfl * (1.0f - gfl) : 0.0f;
            da[2][k] = live ? dc * cT * gft * (1.0f - gft) : 0.0f;
            da[3][k] = live ? dh * tc * go * (1.0f - go) : 0.0f;
            da[4][k] = live ? dc * gi * (1.0f - gg * gg) : 0.0f;
            ndl[k] = live ? dc * gfl : 0.0f;
            ndt[k] = live ? dc * gft : 0.0f;
        }
        dcl[nt] = floatx4{ndl[0], ndl[1], ndl[2], ndl[3]};
        *reinterpret_cast<float4*>(&dct[yy][u0]) = make_float4(ndt[0], ndt[1], ndt[2], ndt[3]);
#pragma unroll
        for (int t = 0; t < 5; ++t) *reinterpret_cast<uint2*>(&dabuf[yy][t * H + u0]) = pack(da[t]);
        {
            T* const zp = inr ? zb + (int64_t)(M.sx * s + yy * M.ky) * (4 * G) : wave_sink<T>();
#pragma unroll
            for (int t = 0; t < 5; ++t) *reinterpret_cast<uint2*>(zp + t * H) = pack(da[t]);
        }
    };
    // Phase B of tile nt: U^T da of its cells for the wave's units.
    auto phase_b = [&](int nt) {
        const T* brow = &dabuf[16 * nt + n16][q * KRUNB];
        floatx4 al = floatx4{0.f, 0.f, 0.f, 0.f}, at = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < NSTEPB; ++ks) {
            const Op b = O::lds(brow + ks * O::PER);
            al = O::mma(A[0][ks], b, al);
            at = O::mma(A[1][ks], b, at);
        }
        gl[nt] = al;
        *reinterpret_cast<float4*>(&gtop[16 * nt + n16][u0]) = make_float4(at[0], at[1], at[2], at[3]);
    };

    // The inputs of the next tile's phase A are loaded right after the
    // current one (one register set), so they are in flight across the
    // barrier and the next segment's MFMAs.
    In in;
    load(steps - 1, max(0, steps - R.w) >> 4, in);
    lds_barrier();
    for (int s = steps - 1; s >= 0; --s) {
        const int ylo = max(0, s - R.w + 1), yhi = min(R.h - 1, s);
        const int t0 = ylo >> 4, t1 = yhi >> 4;
#pragma unroll
        for (int k = 0; k <= NT; ++k) {
            const bool pa = k < NT && k >= t0 && k <= t1;      // A(k) in this segment
            const bool pb = k >= 1 && k - 1 >= t0 && k - 1 <= t1;  // B(k - 1) in this segment
            if (pb) phase_b(k - 1);
            if (pa) {
                phase_a(s, k, in);
                if (k < t1) load(s, k + 1, in);
                else load(max(s - 1, 0), max(0, s - R.w) >> 4, in);  // first tile of the next diagonal
            }
            if (pa || pb) lds_barrier();
        }
    }
}

// ---------------------------------------------------------------------------
// Kernels. With a queue, a fixed number of workgroups per CU take units in
// launch order (longest first) from a counter until none is left, so a long
// unit shares its CU with fewer others than when every unit has its own
// workgroup from the start; without one, workgroup b runs unit b.
// ---------------------------------------------------------------------------
// Forward loads run one step ahead with one workgroup per unit, two steps
// ahead when several workgroups per CU take units from the queue (the load
// latency grows while every CU streams to and from memory).
// Output rows of the invalid cells (outside every rectangle, or masked) set
// to zero, a wave per 64 cells over the grid: each lane reads one cell's mask
// byte and rect id, then the wave clears the rows of the invalid ones with the
// lanes along the row. Done before any unit starts; the units write the rows
// of the valid cells.
__device__ __forceinline__ void zero_invalid_rows(const WaveArgs& a) {
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
    uint2* const y = static_cast<uint2*>(a.y);
    for (int64_t c0 = ((int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * 64; c0 < a.n_cells;
         c0 += waves * 64) {
        const int64_t p = c0 + lane;
        const bool bad = p < a.n_cells && (a.mask[p] == 0 || a.rid[p] < 0);
        for (uint64_t bm = __ballot(bad); bm; bm &= bm - 1) {
            uint2* row = y + (c0 + __builtin_ctzll(bm)) * a.yrow_words;
            for (int k = lane; k < a.yrow_words; k += 64) row[k] = make_uint2(0u, 0u);
        }
    }
}

template <int H, int NT, typename T, bool FWD, bool QUEUE>
__device__ __forceinline__ void run_units(const WaveArgs& a) {
    if constexpr (FWD) {
        if (a.rid) zero_invalid_rows(a);
    }
    if constexpr (!QUEUE) {
        if constexpr (FWD && FwdBig<H, T>::on) wave_fwd_big<H, NT, T>(a, a.units[blockIdx.x]);
        else if (FWD) wave_fwd_unit<H, NT, T, 1>(a, a.units[blockIdx.x]);
        else if constexpr (BwdBig<H, T>::on) wave_bwd_big<H, NT, T>(a, a.units[blockIdx.x]);
        else wave_bwd_unit<H, NT, T>(a, a.units[blockIdx.x]);
        return;
    }
    __shared__ int slot;
    for (;;) {
        lds_barrier();
        if (threadIdx.x == 0) slot = (int)atomicAdd(a.queue, 1u);
        lds_barrier();
        const int k = slot;
        if (k >= a.n_units) break;
        // forward: two steps of prefetch, except where tile groups at H >= 32
        // leave too few registers (1024 threads) and one step measured faster
        if constexpr (FWD && FwdBig<H, T>::on) wave_fwd_big<H, NT, T>(a, a.units[k]);
        else if (FWD) wave_fwd_unit<H, NT, T, (TileGroups<H, NT, T>::NG > 1 && H >= 32) ? 1 : 2>(a, a.units[k]);
        else if constexpr (BwdBig<H, T>::on) wave_bwd_big<H, NT, T>(a, a.units[k]);
        else wave_bwd_unit<H, NT, T>(a, a.units[k]);
    }
    // Count the workgroup out; the last one leaves both counters at zero for
    // the next launch (every other workgroup's last take precedes its count).
    if (threadIdx.x == 0) {
        __threadfence();
        if (atomicAdd(a.queue + 1, 1u) == gridDim.x - 1) {
            __threadfence();
            atomicExch(a.queue, 0u);
            atomicExch(a.queue + 1, 0u);
        }
    }
}

template <int H, int NT, typename T, bool QUEUE>
__global__ void __launch_bounds__((64 * Geo<H, T>::NW * TileGroups<H, NT, T>::NG))
k_wave_fwd(WaveArgs a) {
    run_units<H, NT, T, true, QUEUE>(a);
}

template <int H, int NT, typename T, bool QUEUE>
__global__ void __launch_bounds__((64 * Geo<H, T>::NW * TileGroups<H, NT, T>::NG))
k_wave_bwd(WaveArgs a) {
    run_units<H, NT, T, false, QUEUE>(a);
}

// ---------------------------------------------------------------------------
// Dispatch over (hidden size, N tiles, storage type).
// ---------------------------------------------------------------------------
// LDS of the backward kernel; shapes beyond the 160 KB of a CU are not built.
template <int H, int NT, typename T>
constexpr bool bwd_fits() {
    if constexpr (BwdBig<H, T>::on)
        return (size_t)NT * 16 * (5 * H + 16 / sizeof(T)) * sizeof(T) + (size_t)2 * (NT * 16 + 1) * (H + 4) * 4 <=
               160 * 1024;
    return bwd_lds_base<H, NT, T>() + (bwd_stage<H, NT, T>() ? bwd_lds_stage<H, NT, T>() : 0) <= 160 * 1024;
}

template <int H, int NT, typename T>
static void launch_unit(bool fwd, int n_groups, const WaveArgs& a, hipStream_t s) {
    const dim3 grid(n_groups), block(64 * Geo<H, T>::NW * TileGroups<H, NT, T>::NG);
    if (a.queue) {
        if (fwd) hipLaunchKernelGGL((k_wave_fwd<H, NT, T, true>), grid, block, 0, s, a);
        else if constexpr (bwd_fits<H, NT, T>()) hipLaunchKernelGGL((k_wave_bwd<H, NT, T, true>), grid, block, 0, s, a);
    } else {
        if (fwd) hipLaunchKernelGGL((k_wave_fwd<H, NT, T, false>), grid, block, 0, s, a);
        else if constexpr (bwd_fits<H, NT, T>()) hipLaunchKernelGGL((k_wave_bwd<H, NT, T, false>), grid, block, 0, s, a);
    }
}

template <int H, typename T>
static hipError_t launch_nt(bool fwd, int nt, int n_units, const WaveArgs& a, hipStream_t s) {
    if (nt == 4 && !bwd_fits<H, 4, T>()) return hipErrorInvalidValue;  // host rejects these rectangles
    switch (nt) {
        case 1: launch_unit<H, 1, T>(fwd, n_units, a, s); break;
        case 2: launch_unit<H, 2, T>(fwd, n_units, a, s); break;
        case 3: launch_unit<H, 3, T>(fwd, n_units, a, s); break;
        case 4: launch_unit<H, 4, T>(fwd, n_units, a, s); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Workgroups per CU when units are taken from a queue: the forward runs
// fastest with a unit per CU at a time, the backward (fewer registers, more
// latency per step) with two.
constexpr int FWD_GROUPS_PER_CU = 1, BWD_GROUPS_PER_CU = 2;

static hipError_t launch_wave(bool fwd, const LayerGeom& g, int nt, int n_units, WaveArgs a, hipStream_t s) {
    if (n_units == 0) return hipSuccess;
    a.n_units = n_units;
    if (a.queue) {
        int dev = 0, cus = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        const int groups = (fwd ? FWD_GROUPS_PER_CU : BWD_GROUPS_PER_CU) * std::max(cus, 1);
        if (n_units > groups) {  // else one workgroup per unit
            n_units = groups;
        } else {
            a.queue = nullptr;
        }
    }
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
                                const int32_t* d_rects, const uint8_t* d_mask, const int32_t* d_rid, const void* d_u,
                                void* d_z, float* d_c, void* d_y, unsigned* d_queue, hipStream_t s) {
    const int yrow_words = 4 * g.hidden * (g.dtype == 1 ? 2 : 4) / 8;
    // the launch's own workgroups zero the invalid rows when there are enough
    // of them to cover the canvas quickly (at least one per CU); else a
    // separate kernel does
    int dev = 0, cus = 256;
    if (d_rid && (hipGetDevice(&dev) != hipSuccess ||
                  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess))
        return hipErrorInvalidDevice;
    if (d_rid && n_units < cus) {
        const hipError_t e = launch_zero_invalid(g, 4 * g.hidden, d_mask, d_rid, d_y, s);
        if (e != hipSuccess) return e;
        d_rid = nullptr;
    }
    WaveArgs a{d_units,  d_rects, d_mask, d_u,   d_z,       d_c,       d_y,       nullptr, g.canvas_w, 0,
               INT_MAX, d_queue, n_units, d_rid, g.n_cells, yrow_words};
    return launch_wave(true, g, nt, n_units, a, s);
}

hipError_t launch_wavefront_bwd(const LayerGeom& g, int nt, int n_units, const int32_t* d_units,
                                const int32_t* d_rects, const uint8_t* d_mask, const void* d_u, const void* d_dy,
                                void* d_z, const float* d_c, unsigned* d_queue, hipStream_t s) {
    WaveArgs a{d_units, d_rects, d_mask,  d_u,     d_z,     const_cast<float*>(d_c), nullptr, d_dy, g.canvas_w, 0,
               INT_MAX, d_queue, n_units, nullptr, 0,       0};
    return launch_wave(false, g, nt, n_units, a, s);
}

// Forward kernel of a shape and its workgroup size, for graph nodes.
template <int H, typename T>
static bool fwd_kernel(int nt, const void** fn, int* threads) {
    constexpr int w64 = 64 * Geo<H, T>::NW;
    switch (nt) {
        case 1: *threads = w64 * TileGroups<H, 1, T>::NG; *fn = reinterpret_cast<const void*>(&k_wave_fwd<H, 1, T, false>); return true;
        case 2: *threads = w64 * TileGroups<H, 2, T>::NG; *fn = reinterpret_cast<const void*>(&k_wave_fwd<H, 2, T, false>); return true;
        case 3: *threads = w64 * TileGroups<H, 3, T>::NG; *fn = reinterpret_cast<const void*>(&k_wave_fwd<H, 3, T, false>); return true;
        case 4: *threads = w64 * TileGroups<H, 4, T>::NG; *fn = reinterpret_cast<const void*>(&k_wave_fwd<H, 4, T, false>); return true;
        default: return false;
    }
}

hipError_t build_wavefront_fwd_graph(const LayerGeom& g, int nt, int n_units, int max_steps, const int32_t* d_units,
                                     const int32_t* d_rects, const uint8_t* d_mask, const void* d_u, void* d_z,
                                     float* d_c, void* d_y, hipGraphExec_t* exec) {
    const void* fn = nullptr;
    int threads = 0;
    bool ok = false;
    if (g.dtype == 0) {
        switch (g.hidden) {
            case 4: ok = fwd_kernel<4, float>(nt, &fn, &threads); break;
            case 8: ok = fwd_kernel<8, float>(nt, &fn, &threads); break;
            case 16: ok = fwd_kernel<16, float>(nt, &fn, &threads); break;
            case 32: ok = fwd_kernel<32, float>(nt, &fn, &threads); break;
            case 64: ok = fwd_kernel<64, float>(nt, &fn, &threads); break;
            default: break;
        }
    } else {
        switch (g.hidden) {
            case 32: ok = fwd_kernel<32, bf16_t>(nt, &fn, &threads); break;
            case 64: ok = fwd_kernel<64, bf16_t>(nt, &fn, &threads); break;
            case 128: ok = fwd_kernel<128, bf16_t>(nt, &fn, &threads); break;
            default: break;
        }
    }
    if (!ok || n_units <= 0 || max_steps <= 0) return hipErrorInvalidValue;
    hipGraph_t graph;
    hipError_t e = hipGraphCreate(&graph, 0);
    if (e != hipSuccess) return e;
    hipGraphNode_t prev = nullptr;
    for (int st = 0; st < max_steps && e == hipSuccess; ++st) {
        WaveArgs a{d_units, d_rects, d_mask, d_u, d_z, d_c, d_y, nullptr, g.canvas_w, st, st + 1, nullptr, n_units,
                   nullptr, 0,       0};
        void* params[] = {&a};
        hipKernelNodeParams p{};
        p.func = const_cast<void*>(fn);
        p.gridDim = dim3(n_units);
        p.blockDim = dim3(threads);
        p.sharedMemBytes = 0;
        p.kernelParams = params;
        p.extra = nullptr;
        hipGraphNode_t node;
        e = hipGraphAddKernelNode(&node, graph, prev ? &prev : nullptr, prev ? 1 : 0, &p);
        prev = node;
    }
    if (e == hipSuccess) e = hipGraphInstantiate(exec, graph, nullptr, nullptr, 0);
    const hipError_t e2 = hipGraphDestroy(graph);
    return e != hipSuccess ? e : e2;
}

}  // namespace mdl
