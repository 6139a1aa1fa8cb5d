// Packed-token linear operator y = act(x w^T + bias) + residual over the T real
// tokens (the layer's Proj1 / Proj2 / FF1 / FF2; Section 7.2 runs them as one
// fused loop over the batch and length loops, so they are plain GEMMs with
// M = T and no padding).
//
// bf16: 256x256 output tile per workgroup, K step 64, four waves in a 2x2 grid,
// each wave a 128x128 sub-tile of v_mfma_f32_16x16x32_bf16 accumulators.  Both
// operands are K-contiguous in memory (x is [T, K], w is [N, K]), which is the
// operand layout the MFMA wants, so they are staged through LDS without any
// transposition.  The MFMA computes the transposed tile C[n][m] = sum_k
// w[n][k] x[m][k], so each lane ends with four consecutive output features of
// one token, stored as one 8-byte write with bias / activation / residual fused.
// LDS rows are 128 bytes; the 16-byte chunk index is XOR-swizzled with the row
// so that the fragment reads of 16 consecutive rows hit distinct banks.  Two
// LDS stages: the global loads of step k+1 are in flight while step k computes.
#include "device_common.h"
#include "launch.h"

namespace rag {
namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kGemmThreads = 256;
constexpr int WM = 128, WN = 128;           // wave tile
constexpr int FM = WM / 16, FN = WN / 16;   // 16x16 fragments per wave
constexpr int kRowsPerPass = kGemmThreads / 8;  // 8 chunks of 16 B per 128-B row
constexpr int kPasses = BM / kRowsPerPass;      // 8

__device__ __forceinline__ int swz(int row, int chunk) { return (chunk ^ (row & 7)); }

// Map the linear workgroup id so that each XCD (workgroups are dealt to the 8
// XCDs round-robin) receives a contiguous range of output tiles.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
    const int per = nblocks / 8, rem = nblocks % 8;
    const int xcd = bid % 8, idx = bid / 8;
    return xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
}

template <int ACT, bool HAS_BIAS, bool HAS_RES>
__global__ __launch_bounds__(kGemmThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_gemm_bf16(const uint16_t* __restrict__ x, int ldx, const uint16_t* __restrict__ w,
                 const uint16_t* __restrict__ bias, const uint16_t* residual, int ldr, uint16_t* y, int ldy,
                 int T, int K, int N, int tiles_n) {
    extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
    // stage s: x tile at smem + s*BM*BK, w tile at smem + 2*BM*BK + s*BN*BK

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const int m0 = tm * BM, n0 = tn * BN;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int wm = wave / 2, wn = wave % 2;
    const int l16 = lane % 16, q4 = lane / 16;

    // global -> register staging: thread loads chunk (tid & 7) of rows (tid >> 3) + 32 * p
    const int ld_chunk = tid & 7, ld_row = tid >> 3;
    const uint16_t* xg[kPasses];
    const uint16_t* wg[kPasses];
#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
        const int r = ld_row + kRowsPerPass * p;
        xg[p] = x + (int64_t)min(m0 + r, T - 1) * ldx + ld_chunk * 8;
        wg[p] = w + (int64_t)min(n0 + r, N - 1) * K + ld_chunk * 8;
    }
    u32x4 xr[kPasses], wr[kPasses];
    auto load_global = [&](int k0) {
#pragma unroll
        for (int p = 0; p < kPasses; ++p) {
            xr[p] = *reinterpret_cast<const u32x4*>(xg[p] + k0);
            wr[p] = *reinterpret_cast<const u32x4*>(wg[p] + k0);
        }
    };
    auto store_lds = [&](int buf) {
#pragma unroll
        for (int p = 0; p < kPasses; ++p) {
            const int r = ld_row + kRowsPerPass * p;
            *reinterpret_cast<u32x4*>(smem + buf * BM * BK + r * BK + swz(r, ld_chunk) * 8) = xr[p];
            *reinterpret_cast<u32x4*>(smem + 2 * BM * BK + buf * BN * BK + r * BK + swz(r, ld_chunk) * 8) = wr[p];
        }
    };

    floatx4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int nk = K / BK;
    load_global(0);
    store_lds(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) load_global((kt + 1) * BK);
        const uint16_t* xb = smem + cur * BM * BK;
        const uint16_t* wb = smem + 2 * BM * BK + cur * BN * BK;
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            const int chunk = ks * 4 + q4;
            bf16x8 af[FN], bfr[FM];
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                const int r = wn * WN + i * 16 + l16;
                af[i] = as_bf16x8(*reinterpret_cast<const u32x4*>(wb + r * BK + swz(r, chunk) * 8));
            }
#pragma unroll
            for (int j = 0; j < FM; ++j) {
                const int r = wm * WM + j * 16 + l16;
                bfr[j] = as_bf16x8(*reinterpret_cast<const u32x4*>(xb + r * BK + swz(r, chunk) * 8));
            }
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j) acc[i][j] = mfma16x16x32(af[i], bfr[j], acc[i][j]);
        }
        if (kt + 1 < nk) store_lds(cur ^ 1);
        __syncthreads();
    }

    // epilogue: acc[i][j][r] = y[m][n + r], m = m0 + wm*128 + j*16 + l16,
    // n = n0 + wn*128 + i*16 + 4*q4
#pragma unroll
    for (int i = 0; i < FN; ++i) {
        const int n = n0 + wn * WN + i * 16 + 4 * q4;
        if (n >= N) continue;
        float bv[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (HAS_BIAS) {
            const u32x2 bb = *reinterpret_cast<const u32x2*>(bias + n);
            bv[0] = lo_bf16(bb[0]);
            bv[1] = hi_bf16(bb[0]);
            bv[2] = lo_bf16(bb[1]);
            bv[3] = hi_bf16(bb[1]);
        }
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int m = m0 + wm * WM + j * 16 + l16;
            if (m >= T) continue;
            float o[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) o[r] = activate<ACT>(acc[i][j][r] + bv[r]);
            if constexpr (HAS_RES) {
                const u32x2 rr = *reinterpret_cast<const u32x2*>(residual + (int64_t)m * ldr + n);
                o[0] += lo_bf16(rr[0]);
                o[1] += hi_bf16(rr[0]);
                o[2] += lo_bf16(rr[1]);
                o[3] += hi_bf16(rr[1]);
            }
            const u32x2 out = {pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
            *reinterpret_cast<u32x2*>(y + (int64_t)m * ldy + n) = out;
        }
    }
}

// fp32: 64x64 tiles, K step 16, 4x4 outputs per thread, plain FMA.
template <int ACT>
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ x, int ldx, const float* __restrict__ w,
                                                   const float* __restrict__ bias, const float* residual, int ldr,
                                                   float* y, int ldy, int T, int K, int N) {
    __shared__ float xs[16][64 + 1], ws[16][64 + 1];
    const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
    const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += 16) {
        __syncthreads();
        for (int e = threadIdx.x; e < 64 * 16; e += 256) {
            const int r = e / 16, c = e % 16;
            const int k = k0 + c;
            xs[c][r] = (m0 + r < T && k < K) ? x[(int64_t)(m0 + r) * ldx + k] : 0.f;
            ws[c][r] = (n0 + r < N && k < K) ? w[(int64_t)(n0 + r) * K + k] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            float a[4], b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                a[u] = xs[c][ty * 4 + u];
                b[u] = ws[c][tx + 16 * u];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(a[u], b[v], acc[u][v]);
        }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int m = m0 + ty * 4 + u;
        if (m >= T) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int n = n0 + tx + 16 * v;
            if (n >= N) continue;
            float o = acc[u][v] + (bias ? bias[n] : 0.f);
            o = activate<ACT>(o);
            if (residual) o += residual[(int64_t)m * ldr + n];
            y[(int64_t)m * ldy + n] = o;
        }
    }
}

template <int ACT, bool HB, bool HR>
hipError_t launch_bf16_variant(const void* x, int ldx, const void* w, const void* bias, const void* residual,
                               int ldr, void* y, int ldy, int T, int K, int N, hipStream_t s) {
    const int tiles_m = (T + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    const size_t lds = 2 * (BM + BN) * BK * sizeof(uint16_t);
    static bool attr_set = false;  // benign race: every thread sets the same value
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm_bf16<ACT, HB, HR>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    hipLaunchKernelGGL((k_gemm_bf16<ACT, HB, HR>), dim3(tiles_m * tiles_n), dim3(kGemmThreads), lds, s,
                       static_cast<const uint16_t*>(x), ldx, static_cast<const uint16_t*>(w),
                       static_cast<const uint16_t*>(bias), static_cast<const uint16_t*>(residual), ldr,
                       static_cast<uint16_t*>(y), ldy, T, K, N, tiles_n);
    return hipGetLastError();
}

template <int ACT>
hipError_t launch_bf16_act(const void* x, int ldx, const void* w, const void* bias, const void* residual, int ldr,
                           void* y, int ldy, int T, int K, int N, hipStream_t s) {
    if (bias && residual) return launch_bf16_variant<ACT, true, true>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
    if (bias) return launch_bf16_variant<ACT, true, false>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
    if (residual) return launch_bf16_variant<ACT, false, true>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
    return launch_bf16_variant<ACT, false, false>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
}

}  // namespace

hipError_t launch_linear(int dtype, const void* x, int ldx, const void* w, const void* bias, const void* residual,
                         int ldr, int act, void* y, int ldy, int T, int K, int N, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (dtype == 1) {
        if (act == 1) return launch_bf16_act<1>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
        if (act == 2) return launch_bf16_act<2>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
        return launch_bf16_act<0>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
    }
    const dim3 grid((T + 63) / 64, (N + 63) / 64);
    const float* xf = static_cast<const float*>(x);
    const float* wf = static_cast<const float*>(w);
    const float* bf = static_cast<const float*>(bias);
    const float* rf = static_cast<const float*>(residual);
    float* yf = static_cast<float*>(y);
    if (act == 1) hipLaunchKernelGGL(k_gemm_f32<1>, grid, dim3(256), 0, s, xf, ldx, wf, bf, rf, ldr, yf, ldy, T, K, N);
    else if (act == 2) hipLaunchKernelGGL(k_gemm_f32<2>, grid, dim3(256), 0, s, xf, ldx, wf, bf, rf, ldr, yf, ldy, T, K, N);
    else hipLaunchKernelGGL(k_gemm_f32<0>, grid, dim3(256), 0, s, xf, ldx, wf, bf, rf, ldr, yf, ldy, T, K, N);
    return hipGetLastError();
}

}  // namespace rag
