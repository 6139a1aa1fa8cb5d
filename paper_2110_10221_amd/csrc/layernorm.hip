// LayerNorm over the d features of each packed token row (the layer's two
// LayerNorm operators).  One wave per row: each lane holds its 16-byte chunks
// of the row in registers, so the row is read once and written once (the
// operator is bound by HBM bandwidth).  Mean and population variance are
// computed in two passes over the registers.
#include "device_common.h"
#include "launch.h"

namespace rag {
namespace {

template <bool BF16>
struct LnIO;

template <>
struct LnIO<true> {
    static constexpr int kPerChunk = 8;  // 8 bf16 = 16 bytes
    static __device__ __forceinline__ void load(const void* base, int64_t off, float* v) {
        const u32x4 c = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(base) + off);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[2 * e] = lo_bf16(c[e]);
            v[2 * e + 1] = hi_bf16(c[e]);
        }
    }
    static __device__ __forceinline__ void store(void* base, int64_t off, const float* v) {
        u32x4 c;
#pragma unroll
        for (int e = 0; e < 4; ++e) c[e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
        *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(base) + off) = c;
    }
};

template <>
struct LnIO<false> {
    static constexpr int kPerChunk = 4;  // 4 fp32 = 16 bytes
    static __device__ __forceinline__ void load(const void* base, int64_t off, float* v) {
        const floatx4 c = *reinterpret_cast<const floatx4*>(static_cast<const float*>(base) + off);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = c[e];
    }
    static __device__ __forceinline__ void store(void* base, int64_t off, const float* v) {
        *reinterpret_cast<floatx4*>(static_cast<float*>(base) + off) = floatx4{v[0], v[1], v[2], v[3]};
    }
};

template <bool BF16, int MAXC>
__global__ __launch_bounds__(256) void k_layernorm(const void* x, int ldx, const void* gamma, const void* beta,
                                                    float eps, void* y, int ldy, int T, int d) {
    using IO = LnIO<BF16>;
    constexpr int E = IO::kPerChunk;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int row = blockIdx.x * 4 + wave;
    if (row >= T) return;
    const int nch = d / E;
    // Every load is issued before the first value is used (one wait for all of
    // them): chunk indexes are clamped into the row and lanes past it ignore what
    // they read.  gamma and beta join them while the registers allow.
    constexpr bool kEarlyGB = MAXC <= 4;
    constexpr int kGB = kEarlyGB ? MAXC : 1;
    float v[MAXC][E], g[kGB][E], bt[kGB][E];
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int ch = min(lane + kWave * c, nch - 1);
        IO::load(x, (int64_t)row * ldx + ch * E, v[c]);
        if constexpr (kEarlyGB) {
            IO::load(gamma, ch * E, g[c]);
            IO::load(beta, ch * E, bt[c]);
        }
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        if (lane + kWave * c < nch) {
#pragma unroll
            for (int e = 0; e < E; ++e) s += v[c][e];
        }
    }
    const float mean = wave_sum(s) / d;
    float q = 0.f;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int ch = lane + kWave * c;
        if (ch < nch) {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float u = v[c][e] - mean;
                q += u * u;
            }
        }
    }
    const float inv = 1.0f / sqrtf(wave_sum(q) / d + eps);
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int ch = lane + kWave * c;
        if (ch < nch) {
            const int cg = kEarlyGB ? c : 0;
            if constexpr (!kEarlyGB) {
                IO::load(gamma, ch * E, g[0]);
                IO::load(beta, ch * E, bt[0]);
            }
            float o[E];
#pragma unroll
            for (int e = 0; e < E; ++e) o[e] = g[cg][e] * ((v[c][e] - mean) * inv) + bt[cg][e];
            IO::store(y, (int64_t)row * ldy + ch * E, o);
        }
    }
}

template <bool BF16>
hipError_t launch_ln(const void* x, int ldx, const void* g, const void* b, float eps, void* y, int ldy, int T, int d,
                     hipStream_t s) {
    constexpr int E = LnIO<BF16>::kPerChunk;
    const int nch = d / E;
    const dim3 grid((T + 3) / 4), block(256);
    if (nch <= kWave) hipLaunchKernelGGL((k_layernorm<BF16, 1>), grid, block, 0, s, x, ldx, g, b, eps, y, ldy, T, d);
    else if (nch <= 2 * kWave) hipLaunchKernelGGL((k_layernorm<BF16, 2>), grid, block, 0, s, x, ldx, g, b, eps, y, ldy, T, d);
    else if (nch <= 4 * kWave) hipLaunchKernelGGL((k_layernorm<BF16, 4>), grid, block, 0, s, x, ldx, g, b, eps, y, ldy, T, d);
    else if (nch <= 8 * kWave) hipLaunchKernelGGL((k_layernorm<BF16, 8>), grid, block, 0, s, x, ldx, g, b, eps, y, ldy, T, d);
    else hipLaunchKernelGGL((k_layernorm<BF16, 16>), grid, block, 0, s, x, ldx, g, b, eps, y, ldy, T, d);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_layernorm(int dtype, const void* x, int ldx, const void* gamma, const void* beta, float eps, void* y,
                            int ldy, int T, int d, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (dtype == 1) return launch_ln<true>(x, ldx, gamma, beta, eps, y, ldy, T, d, s);
    return launch_ln<false>(x, ldx, gamma, beta, eps, y, ldy, T, d, s);
}

}  // namespace rag
