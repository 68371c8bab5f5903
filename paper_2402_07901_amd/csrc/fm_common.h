// Device helpers shared by the Fastmax HIP kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fm {

typedef uint16_t bf16_t;  // bfloat16 kept as raw bits

__device__ __forceinline__ float bf16_to_f32(bf16_t b)
{
    return __uint_as_float(((uint32_t)b) << 16);
}

// float32 -> bfloat16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

template <typename T> struct io;
template <> struct io<float> {
    static __device__ __forceinline__ float ld(const float *p, size_t i) { return p[i]; }
    static __device__ __forceinline__ void st(float *p, size_t i, float x) { p[i] = x; }
};
template <> struct io<bf16_t> {
    static __device__ __forceinline__ float ld(const bf16_t *p, size_t i) { return bf16_to_f32(p[i]); }
    static __device__ __forceinline__ void st(bf16_t *p, size_t i, float x) { p[i] = f32_to_bf16(x); }
};

// Taylor polynomial of exp truncated at degree p (Sec. 2.2) and its derivative.
template <int P> __device__ __forceinline__ float taylor(float s);
template <> __device__ __forceinline__ float taylor<1>(float s) { return 1.0f + s; }
template <> __device__ __forceinline__ float taylor<2>(float s) { return fmaf(0.5f * s, s, 1.0f + s); }
template <int P> __device__ __forceinline__ float dtaylor(float s);
template <> __device__ __forceinline__ float dtaylor<1>(float) { return 1.0f; }
template <> __device__ __forceinline__ float dtaylor<2>(float s) { return 1.0f + s; }

// Number of moment features for order p: [1, k, (k_m k_l)_{m<=l}].
__host__ __device__ constexpr int n_features(int D, int p)
{
    return 1 + D + (p >= 2 ? D * (D + 1) / 2 : 0);
}

// Index of the symmetric pair (m, l), m <= l, in m-major order, offset past
// the constant and linear features.
__host__ __device__ constexpr int pair_feature(int D, int m, int l)
{
    return 1 + D + m * D - (m * (m - 1)) / 2 + (l - m);
}

// Quadratic-term dropout (Sec. 2.4, dropout paragraph; Fig. 2): keep bits
// on the D(D+1)/2 quadratic features of every key token.  A token's bits
// fill mask_words(D) uint32 words; pair feature t (m-major, m <= l, the
// order of pair_feature) is bit t % 32 of word t / 32.
__host__ __device__ constexpr int mask_words(int D)
{
    return (D * (D + 1) / 2 + 31) / 32;
}

// Sum over the four rows of 16 lanes (lanes r16, r16 + 16, r16 + 32, r16 + 48),
// in every lane, with the permlane swaps (no LDS round trip): swapping the odd
// rows of one copy with the even rows of another puts rows 2j and 2j + 1 side
// by side, then the two halves of the wave likewise.  Every lane of the wave
// must take part.
__device__ __forceinline__ float rows4_sum(float x)
{
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

}  // namespace fm
