// Shared device helpers for the MDLSTM kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // 16-byte chunk held in registers
typedef uint16_t bf16_t;  // bfloat16 storage (upper half of an fp32)

// ---------------------------------------------------------------------------
// bfloat16 <-> fp32
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf2f(bf16_t v) { return __uint_as_float(((uint32_t)v) << 16); }

// Two fp32 values to packed bf16 (lo in the low half): round to nearest,
// ties to even, a NaN stays a (quiet) NaN; one hardware conversion
// (v_cvt_pk_bf16_f32) for the pair.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
    const bf16x2 b = __builtin_convertvector(floatx2{lo, hi}, bf16x2);
    uint32_t r;
    __builtin_memcpy(&r, &b, 4);
    return r;
}
__device__ __forceinline__ bf16_t f2bf(float f) { return (bf16_t)(f2bf2(f, 0.0f) & 0xffffu); }

// Storage traits: loads/stores of 4 consecutive elements as fp32.
template <typename T>
struct St;

template <>
struct St<float> {
    static __device__ __forceinline__ floatx4 ld4(const float* p) {
        float4 v = *reinterpret_cast<const float4*>(p);
        return floatx4{v.x, v.y, v.z, v.w};
    }
    static __device__ __forceinline__ void st4(float* p, floatx4 v) {
        *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    }
    static __device__ __forceinline__ float ld1(const float* p) { return *p; }
    static __device__ __forceinline__ void st1(float* p, float v) { *p = v; }
};

template <>
struct St<bf16_t> {
    static __device__ __forceinline__ floatx4 ld4(const bf16_t* p) {
        uint2 v = *reinterpret_cast<const uint2*>(p);
        return floatx4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                       __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u)};
    }
    static __device__ __forceinline__ void st4(bf16_t* p, floatx4 v) {
        uint2 o;
        o.x = f2bf2(v[0], v[1]);
        o.y = f2bf2(v[2], v[3]);
        *reinterpret_cast<uint2*>(p) = o;
    }
    static __device__ __forceinline__ float ld1(const bf16_t* p) { return bf2f(*p); }
    static __device__ __forceinline__ void st1(bf16_t* p, float v) { *p = f2bf(v); }
};

// ---------------------------------------------------------------------------
// Gate nonlinearities (fp32). The recurrence uses the hardware exp2 and
// reciprocal (about 1 ulp each); arguments are scaled by log2(e) first, so
// the relative error grows with |z| by |z| * 2^-24, far below the 1e-5
// tolerance for gate pre-activations of ordinary size.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float sigm(float z) { return 1.0f / (1.0f + expf(-z)); }

__device__ __forceinline__ float sigm_fast(float z) {
    return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

// tanh(z) = sign(z) (1 - e) / (1 + e), e = exp(-2|z|): no cancellation for
// large |z|; absolute error a few ulp of 1 near 0.
__device__ __forceinline__ float tanh_fast(float z) {
    const float e = __builtin_amdgcn_exp2f(-2.8853900817779268f * fabsf(z));
    return copysignf((1.0f - e) * __builtin_amdgcn_rcpf(1.0f + e), z);
}

__device__ __forceinline__ float tanh_acc(float z) {
    float a = fabsf(z);
    float r;
    if (a < 0.125f) {
        // odd Taylor series, error below 2e-10 relative on |z| < 1/8
        float p = z * z;
        r = z * (1.0f + p * (-1.0f / 3.0f + p * (2.0f / 15.0f + p * (-17.0f / 315.0f))));
    } else {
        float e = expf(-2.0f * a);
        r = copysignf((1.0f - e) / (1.0f + e), z);
    }
    return r;
}

// ---------------------------------------------------------------------------
// MFMA 16x16 tiles. For both instructions used here the output tile D[16][16]
// lives in lane l = 16*q + n as D[4*q + r][n], r = 0..3; the A operand row is
// l % 16 and the B operand column is l % 16, with the reduction slot l / 16.
// ---------------------------------------------------------------------------
__device__ __forceinline__ floatx4 mfma_f32(float a, float b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mfma_bf16(bf16x8 a, bf16x8 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
    bf16x8 r;
    __builtin_memcpy(&r, &v, sizeof(r));
    return r;
}

// ---------------------------------------------------------------------------
// Device-side rectangle and unit decoding.
// ---------------------------------------------------------------------------
struct RectD {
    int32_t y0, x0, h, w;
};

// Canvas index of a unit's local cell (y, x) in scan direction d's frame:
// direction bit 0 mirrors x (scan from the right), bit 1 mirrors y (from the bottom).
__device__ __forceinline__ int64_t canvas_index(const RectD& R, int d, int y, int x, int canvas_w) {
    int cy = R.y0 + ((d & 2) ? (R.h - 1 - y) : y);
    int cx = R.x0 + ((d & 1) ? (R.w - 1 - x) : x);
    return (int64_t)cy * canvas_w + cx;
}

// Workgroup barrier that orders LDS accesses only: global memory operations
// of the waves stay in flight across it (__syncthreads also waits for them).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Canvas index of local cell (y, s - y) of diagonal s of a unit in scan
// direction d (as canvas_index), written c0 + sx*s + y*ky: with the
// direction's mirroring folded into per-unit constants, a step's base costs
// one add and a cell one multiply-add.
struct DiagMap {
    int64_t c0;
    int sx, ky;
    __device__ __forceinline__ DiagMap(const RectD& R, int d, int canvas_w) {
        const int cy0 = R.y0 + ((d & 2) ? R.h - 1 : 0), cx0 = R.x0 + ((d & 1) ? R.w - 1 : 0);
        sx = (d & 1) ? -1 : 1;
        ky = ((d & 2) ? -canvas_w : canvas_w) - sx;
        c0 = (int64_t)cy0 * canvas_w + cx0;
    }
    __device__ __forceinline__ int64_t base(int s) const { return c0 + (int64_t)(sx * s); }
    __device__ __forceinline__ int64_t at(int64_t b, int y) const { return b + (int64_t)y * ky; }
};
