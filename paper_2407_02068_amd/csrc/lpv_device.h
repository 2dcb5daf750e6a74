// lpv_device.h -- device-side types and helpers shared by the liblpv kernels
// (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lpv {

// Matrix-core operand and accumulator vectors.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Element types by their lpv_dtype code (1 = fp16, 2 = bf16).  Each one knows
// its 32x32x16 MFMA with float32 accumulation and its conversions.
template <int DT> struct Elem;

template <> struct Elem<2> {
    typedef bf16x8 frag;
    __device__ static inline f32x16 mma(frag a, frag b, f32x16 c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static inline float to_f32(uint16_t bits)
    {
        return __uint_as_float((uint32_t)bits << 16);
    }
    // round to nearest even (NaN stays NaN)
    __device__ static inline uint16_t from_f32(float v)
    {
        return __builtin_bit_cast(uint16_t, (__bf16)v);
    }
};

template <> struct Elem<1> {
    typedef f16x8 frag;
    __device__ static inline f32x16 mma(frag a, frag b, f32x16 c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
    }
    __device__ static inline float to_f32(uint16_t bits)
    {
        return (float)__builtin_bit_cast(_Float16, bits);
    }
    __device__ static inline uint16_t from_f32(float v)
    {
        return __builtin_bit_cast(uint16_t, (_Float16)v);
    }
};

template <typename F> __device__ inline F as_frag(uint4 v) { return __builtin_bit_cast(F, v); }

// Two float32 values rounded to nearest even and packed (low = a): one
// v_cvt_pk_bf16_f32 / v_cvt_pk_f16_f32.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
template <int DT> __device__ inline uint32_t pack2(float a, float b)
{
    const f32x2 v = {a, b};
    if constexpr (DT == 2)
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
    else
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2));
}

// GELU with the error function, x Phi(x), Phi(x) = erfc(-x / sqrt 2) / 2, in
// float32 without branches.  erfc(a), a = |x| / sqrt 2 < 4, is 2^f(a) with f
// a degree-7 polynomial fitted to log2 erfc on [0, 4] (coefficients from
// gelu_fit.py beside this package's Python files: erfc to 6e-6 relative in
// float32).  Then x Phi(x) = max(x, 0) - |x| erfc(a) / 2 for either sign of x
// (for x < 0 that term is the whole result, so the negative tail keeps its
// relative accuracy), and |x| / 2 = a / sqrt 2, so the term is a e with
// e = 2^(f(a) - 1/2): one fused multiply-add.  GELU to 5e-6 relative.  From
// a = 4 on (|x| > 5.65, where |x| erfc(a) / 2 < 5e-8 |x|) the result is
// max(x, 0); a NaN input gives NaN.
__device__ inline float gelu_erf(float v)
{
    const float a = fabsf(v) * 0.70710678118654752f;
    float f = -2.055665755e-05f;
    f = fmaf(f, a, 4.903716035e-04f);
    f = fmaf(f, a, -5.252704490e-03f);
    f = fmaf(f, a, 3.400664404e-02f);
    f = fmaf(f, a, -1.525942534e-01f);
    f = fmaf(f, a, -9.169431329e-01f);
    f = fmaf(f, a, -1.628112197e+00f);
    f = fmaf(f, a, 4.628196166e-06f - 0.5f);
    const float e = __builtin_amdgcn_exp2f(f);  // erfc(a) / sqrt 2
    const float r = fmaxf(v, 0.0f);
    return a >= 4.0f ? r : fmaf(-a, e, r);
}

// Wave-level inclusive prefix sum over the 64 lanes.
__device__ inline int wave_inclusive_scan(int v)
{
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int u = __shfl_up(v, d, 64);
        if (lane >= d)
            v += u;
    }
    return v;
}

__device__ inline int wave_sum(int v)
{
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1)
        v += __shfl_xor(v, d, 64);
    return v;
}

// Number of lanes below this one whose predicate is set, and the wave total.
__device__ inline int lanes_below(uint64_t ballot)
{
    const int lane = threadIdx.x & 63;
    const uint64_t below = lane ? (ballot & (~0ull >> (64 - lane))) : 0ull;
    return __popcll(below);
}

}  // namespace lpv
