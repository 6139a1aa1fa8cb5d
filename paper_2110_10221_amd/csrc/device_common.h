// Device-side helpers shared by the HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rag {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float floatx4;
typedef __attribute__((ext_vector_type(16))) float floatx16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kWave = 64;
constexpr int kTile = 64;     // attention tile edge (rows / cols of a score tile)
constexpr int kHeadDim = 64;  // head dimension the attention kernels are built for

// Status-word bits (mirrors the public enum).
constexpr int kDataNegLength = 1, kDataLongLength = 2, kDataTokenCount = 4, kDataQktCap = 8,
              kDataAvCap = 16, kDataScoreCap = 32;

// Variable-sized batched GEMM: output tile, size limits and status-word bits
// (mirror the public constants).
constexpr int kVgemmTileM = 128, kVgemmTileN = 256, kVgemmMaxBatch = 4096, kVgemmMaxDim = 65536;
constexpr int kVgemmNegSize = 1, kVgemmLargeSize = 2, kVgemmTileCap = 4, kVgemmOperandCap = 8,
              kVgemmBf16Shape = 16;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

// Round to nearest, ties to even (gfx950's v_cvt_pk_bf16_f32, branch-free).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f)); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(uint32_t, v);
}

// Low / high bf16 halves of a packed pair, widened.
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// Reductions within aligned groups of `g` lanes (g a power of two <= 64).
__device__ __forceinline__ float group_max(float v, int g) {
    for (int o = g >> 1; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ __forceinline__ float group_sum(float v, int g) {
    for (int o = g >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }

__device__ __forceinline__ float gelu_tanh(float x) {
    const float c = 0.79788456080286536f;  // sqrt(2/pi)
    return 0.5f * x * (1.0f + tanhf(c * (x + 0.044715f * x * x * x)));
}

template <int ACT>
__device__ __forceinline__ float activate(float x) {
    if constexpr (ACT == 1) return gelu_erf(x);
    else if constexpr (ACT == 2) return gelu_tanh(x);
    else return x;
}

// GELU (erf form) for bf16 outputs with a branch-free erfc: Abramowitz & Stegun,
// Handbook of Mathematical Functions, formula 7.1.26, erfc(z) ~ t*(a1 + t*(a2 +
// t*(a3 + t*(a4 + t*a5)))) * exp(-z^2), t = 1/(1 + p z), z >= 0, |error| <= 1.5e-7
// (far below bf16 resolution).  Since x*erf(x/sqrt2) is even in x,
// x*Phi(x) = max(x, 0) - |x| * erfc(|x|/sqrt2) / 2, which needs no sign branch and
// keeps the relative accuracy of the small negative branch; the 1/2 is folded into
// the coefficients and exp(-x^2/2) is evaluated as a power of two.
__device__ __forceinline__ float gelu_erf_fast(float x) {
    const float ax = fabsf(x);
    const float t = __builtin_amdgcn_rcpf(fmaf(ax, 0.3275911f * 0.70710678118654752f, 1.0f));
    const float e = __builtin_amdgcn_exp2f(x * x * (-0.5f * 1.4426950408889634f));
    const float half_poly =
        t * (0.5f * 0.254829592f +
             t * (0.5f * -0.284496736f + t * (0.5f * 1.421413741f + t * (0.5f * -1.453152027f + t * (0.5f * 1.061405429f)))));
    return fmaf(-ax, half_poly * e, fmaxf(x, 0.f));
}

template <int ACT>
__device__ __forceinline__ float activate_bf16(float x) {
    if constexpr (ACT == 1) return gelu_erf_fast(x);
    else return activate<ACT>(x);
}

__device__ __forceinline__ floatx4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const floatx4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 32x32x16: lane l supplies row (l % 32) of A and column (l % 32) of B with the 8
// k values 8*(l/32) .. 8*(l/32)+7; it receives C column l % 32, rows
// 8*(r/4) + 4*(l/32) + (r%4) for accumulator element r = 0..15.  Measured on
// MI355X, chains of this form sustain about 2.1 PFLOP/s against about 1.2 for
// the 16x16x32 form, so the dense contractions use it.
__device__ __forceinline__ floatx16 mfma32x32x16(const bf16x8& a, const bf16x8& b, const floatx16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& v) {
    return __builtin_bit_cast(bf16x8, v);
}

}  // namespace rag
