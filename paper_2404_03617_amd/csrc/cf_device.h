// cf_device.h -- device-side helpers shared by the gfx950 kernels of the
// ConvFirst library: I/O dtype traits, MFMA wrappers, packed conversions and
// the activation functions.  Internal header; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cf {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// 16 bytes = 8 elements of the I/O dtype, viewed as four 32-bit words.
union Pack8 {
    u32x4 u;
    half8 h;
    bf16x8 b;
    uint32_t w[4];
};

struct F16 {
    static constexpr bool is_bf16 = false;
    static __device__ __forceinline__ float4v mfma(const u32x4 &a, const u32x4 &b, const float4v &c) {
        Pack8 pa, pb;
        pa.u = a;
        pb.u = b;
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(pa.h, pb.h, c, 0, 0, 0);
    }
    // two fp32 -> packed pair, round to nearest even (v_cvt_pk_f16_f32)
    static __device__ __forceinline__ uint32_t pack2(float lo, float hi) {
        half2v v;
        v.x = (_Float16)lo;
        v.y = (_Float16)hi;
        return __builtin_bit_cast(uint32_t, v);
    }
    static __device__ __forceinline__ float lo(uint32_t w) {
        return (float)__builtin_bit_cast(half2v, w).x;
    }
    static __device__ __forceinline__ float hi(uint32_t w) {
        return (float)__builtin_bit_cast(half2v, w).y;
    }
};

struct BF16 {
    static constexpr bool is_bf16 = true;
    static __device__ __forceinline__ float4v mfma(const u32x4 &a, const u32x4 &b, const float4v &c) {
        Pack8 pa, pb;
        pa.u = a;
        pb.u = b;
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa.b, pb.b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ uint32_t pack2(float lo, float hi) {
        bf16x2 v;
        v.x = (__bf16)lo;
        v.y = (__bf16)hi;
        return __builtin_bit_cast(uint32_t, v);
    }
    // bf16 -> fp32 is exact: the bf16 bits are the high half of the fp32 bits
    static __device__ __forceinline__ float lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
    static __device__ __forceinline__ float hi(uint32_t w) {
        return __builtin_bit_cast(float, w & 0xffff0000u);
    }
};

// ---------------------------------------------------------------------------
// GELU in packed fp16, evaluated in the scaled variable w = u / 4 and returning
// GELU(u) / 4 = w * Phi(4 w).
//
// Phi(4w) ~= clamp01(0.5 + w * Q(w*w)) with Q a degree-4 polynomial.  The
// coefficients come from a fit made for this library (iteratively reweighted
// least squares towards the minimax error of u*(P - Phi) on |u| <= 3.5, refined
// by direct search on the error of this exact fp16 evaluation over every
// finite fp16 input; the generator is gelu_fit.py next to this file).  Q's
// leading coefficient is positive, so past the fitted range P grows
// monotonically and the [0, 1] clamp (folded into v_pk_fma_f16) saturates it
// on the correct side; fp16 overflow of w*w gives +-inf, which clamps the same
// way.  Measured over all finite fp16 inputs, in units of u: |error| < 3.4e-3
// for |u| < 10 and exact (saturated) beyond.
// Cost: 7 packed instructions per pair of hidden values.
constexpr float GELU_Q0 = 1.57329215f;
constexpr float GELU_Q1 = -3.77201461f;
constexpr float GELU_Q2 = 6.60125630f;
constexpr float GELU_Q3 = -6.30715993f;
constexpr float GELU_Q4 = 2.47227138f;

__device__ __forceinline__ half2v splat2(float v) { return half2v{(_Float16)v, (_Float16)v}; }

__device__ __forceinline__ half2v gelu_pk_f16_quarter(half2v w) {
    const half2v s = w * w;
    half2v q = __builtin_elementwise_fma(s, splat2(GELU_Q4), splat2(GELU_Q3));
    q = __builtin_elementwise_fma(s, q, splat2(GELU_Q2));
    q = __builtin_elementwise_fma(s, q, splat2(GELU_Q1));
    q = __builtin_elementwise_fma(s, q, splat2(GELU_Q0));
    half2v p = __builtin_elementwise_fma(w, q, splat2(0.5f));
    p = __builtin_elementwise_min(__builtin_elementwise_max(p, splat2(0.0f)), splat2(1.0f));
    return w * p;
}

// Exact-erf GELU in fp32 (bf16 path; the device erff of the ROCm math library).
__device__ __forceinline__ float gelu_f32(float u) { return 0.5f * u * (1.0f + erff(u * 0.70710678118654752f)); }

enum { ACT_GELU = 0, ACT_RELU = 1, ACT_NONE = 2 };

__host__ __device__ constexpr int ceil_div(int a, int b) { return (a + b - 1) / b; }

// n / d for n < 2^31 by multiply-high (Granlund-Montgomery): q = (umulhi(n, m) + n) >> s.
struct FastDiv {
    uint32_t d, m, s;
};

inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t s = 0;
    while ((1ull << s) < d)
        s++;
    const uint64_t m = (((1ull << s) - d) << 32) / d + 1;
    return FastDiv{d, (uint32_t)m, s};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) {
    return (__umulhi(n, f.m) + n) >> f.s;
}

}  // namespace cf
