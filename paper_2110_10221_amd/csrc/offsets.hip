// The prelude on the GPU: prefix sums of the lengths, the longest-first order,
// the token -> sequence map and the (sequence, head, tile) work lists.
//
// The paper builds these auxiliary arrays on the host and copies them over
// (Section 2 pipeline; its Section 7.4 finds the copy to dominate the prelude's
// cost).  Here the lengths already live in device memory and four small
// kernels build everything in place, so nothing crosses PCIe:
//   1. scan   (one workgroup): tok_off, att_off, validation, largest length
//   2. rank   (B/256 workgroups): stable longest-first rank -> order
//   3. items  (one workgroup): per-sequence item counts scanned in `order`
//   4. fill   (B workgroups): work-list entries and the token map
// Batches of up to 1024 sequences run steps 1-3 as one single-workgroup kernel,
// and batches of up to 256 the whole prelude as one launch.
#include <climits>

#include "device_common.h"
#include "launch.h"
#include "plan_device.h"

namespace rag {
namespace {

constexpr int kScanThreads = 1024;
constexpr int kScanWaves = kScanThreads / kWave;

__global__ __launch_bounds__(kScanThreads) void k_plan_scan(const int32_t* __restrict__ lengths, int B,
                                                             int T_expected, int max_len, int H,
                                                             int32_t* __restrict__ tok_off,
                                                             int64_t* __restrict__ att_off,
                                                             int32_t* __restrict__ status) {
    __shared__ int64_t sh_a[kScanWaves], sh_b[kScanWaves];
    __shared__ int sh_flags, sh_max;
    if (threadIdx.x == 0) {
        sh_flags = 0;
        sh_max = 0;
    }
    __syncthreads();
    int flags = 0, mx = 0;
    int64_t carry_tok = 0, carry_att = 0;
    for (int base = 0; base < B; base += kScanThreads) {
        const int b = base + threadIdx.x;
        int L = b < B ? lengths[b] : 0;
        if (b < B) {
            if (L < 0) flags |= kDataNegLength;
            if (L > max_len) flags |= kDataLongLength;
            mx = max(mx, L);
        }
        const int64_t Lc = L > 0 ? L : 0;  // negative lengths are flagged, counted as 0
        int64_t et, ea, tt, ta;
        block_exclusive_scan2(Lc, (int64_t)H * Lc * Lc, et, ea, tt, ta, sh_a, sh_b);
        if (b < B) {
            tok_off[b] = static_cast<int32_t>(carry_tok + et);
            att_off[b] = carry_att + ea;
        }
        carry_tok += tt;
        carry_att += ta;
    }
    if (flags) atomicOr(&sh_flags, flags);
    atomicMax(&sh_max, mx);
    __syncthreads();
    if (threadIdx.x == 0) {
        int f = sh_flags;
        if (carry_tok != T_expected) f |= kDataTokenCount;
        tok_off[B] = static_cast<int32_t>(carry_tok);
        att_off[B] = carry_att;
        status[0] = f;
        status[1] = 0;
        status[2] = 0;
        status[3] = sh_max;
    }
}

// rank(b) = #{b' : L_b' > L_b} + #{b' < b : L_b' = L_b}: a strict total order, so
// `order[rank(b)] = b` writes every slot of order exactly once for any lengths.
__global__ __launch_bounds__(256) void k_plan_rank(const int32_t* __restrict__ lengths, int B,
                                                    int32_t* __restrict__ order) {
    __shared__ int32_t Ls[256];
    const int b = blockIdx.x * 256 + threadIdx.x;
    const int Lb = b < B ? lengths[b] : 0;
    int rank = 0;
    for (int base = 0; base < B; base += 256) {
        __syncthreads();
        Ls[threadIdx.x] = base + threadIdx.x < B ? lengths[base + threadIdx.x] : 0;
        __syncthreads();
        const int n = min(256, B - base);
        for (int k = 0; k < n; ++k) {
            const int Lk = Ls[k];
            rank += (Lk > Lb) | ((Lk == Lb) & (base + k < b));
        }
    }
    if (b < B) order[rank] = b;
}

__global__ __launch_bounds__(kScanThreads) void k_plan_items(const int32_t* __restrict__ lengths,
                                                              const int32_t* __restrict__ order, int B,
                                                              int H, int64_t qkt_cap, int64_t av_cap,
                                                              int32_t* __restrict__ qkt_item_off,
                                                              int32_t* __restrict__ av_item_off,
                                                              int32_t* __restrict__ status) {
    __shared__ int64_t sh_a[kScanWaves], sh_b[kScanWaves];
    const int flags0 = status[0];
    int64_t carry_q = 0, carry_a = 0;
    for (int base = 0; base < B; base += kScanThreads) {
        const int k = base + threadIdx.x;
        int64_t nq = 0, na = 0;
        if (k < B && flags0 == 0) {
            const int64_t nt = (lengths[order[k]] + kTile - 1) / kTile;
            na = (int64_t)H * nt;
            nq = na * nt;
        }
        int64_t eq, ea, tq, ta;
        block_exclusive_scan2(nq, na, eq, ea, tq, ta, sh_a, sh_b);
        if (k < B) {
            qkt_item_off[k] = static_cast<int32_t>(min(carry_q + eq, (int64_t)INT_MAX));
            av_item_off[k] = static_cast<int32_t>(min(carry_a + ea, (int64_t)INT_MAX));
        }
        carry_q += tq;
        carry_a += ta;
    }
    if (threadIdx.x == 0) {
        int f = flags0;
        if (carry_q > qkt_cap) f |= kDataQktCap;
        if (carry_a > av_cap) f |= kDataAvCap;
        qkt_item_off[B] = static_cast<int32_t>(min(carry_q, (int64_t)INT_MAX));
        av_item_off[B] = static_cast<int32_t>(min(carry_a, (int64_t)INT_MAX));
        status[0] = f;
        status[1] = f ? 0 : static_cast<int32_t>(carry_q);
        status[2] = f ? 0 : static_cast<int32_t>(carry_a);
    }
}

// Batches of at most kScanThreads sequences: scan, rank and item counting in one
// workgroup (one thread per sequence, lengths and order kept in LDS), with the
// same results as k_plan_scan + k_plan_rank + k_plan_items.
__global__ __launch_bounds__(kScanThreads) void k_plan_small(const int32_t* __restrict__ lengths, int B,
                                                              int T_expected, int max_len, int H, int64_t qkt_cap,
                                                              int64_t av_cap, int32_t* __restrict__ tok_off,
                                                              int64_t* __restrict__ att_off,
                                                              int32_t* __restrict__ order,
                                                              int32_t* __restrict__ qkt_item_off,
                                                              int32_t* __restrict__ av_item_off,
                                                              int32_t* __restrict__ status) {
    __shared__ int64_t sh_a[kScanWaves], sh_b[kScanWaves];
    __shared__ __attribute__((aligned(16))) int32_t sL[kScanThreads];
    __shared__ int32_t sOrder[kScanThreads];
    __shared__ int sh_flags, sh_max;
    const int b = threadIdx.x;
    if (b == 0) {
        sh_flags = 0;
        sh_max = 0;
    }
    const int L = b < B ? lengths[b] : 0;
    sL[b] = b < B ? L : -1;  // padding never outranks a length (negative lengths are flagged anyway)
    int flags = 0;
    if (b < B) {
        if (L < 0) flags |= kDataNegLength;
        if (L > max_len) flags |= kDataLongLength;
    }
    __syncthreads();
    if (flags) atomicOr(&sh_flags, flags);
    if (b < B) atomicMax(&sh_max, L);
    // offsets (negative lengths are flagged and counted as 0)
    const int64_t Lc = L > 0 ? L : 0;
    int64_t et, ea, tt, ta;
    block_exclusive_scan2(Lc, (int64_t)H * Lc * Lc, et, ea, tt, ta, sh_a, sh_b);
    if (b < B) {
        tok_off[b] = static_cast<int32_t>(et);
        att_off[b] = ea;
    }
    // longest-first rank (a strict total order: every slot written once)
    if (b < B) {
        int rank = 0;
        // four lengths per LDS read, so the reads pipeline instead of each waiting in turn
#pragma unroll 2
        for (int k = 0; k < B; k += 4) {
            const int4 l4 = *reinterpret_cast<const int4*>(sL + k);
            rank += (l4.x > L) | ((l4.x == L) & (k < b));
            rank += (l4.y > L) | ((l4.y == L) & (k + 1 < b));
            rank += (l4.z > L) | ((l4.z == L) & (k + 2 < b));
            rank += (l4.w > L) | ((l4.w == L) & (k + 3 < b));
        }
        sOrder[rank] = b;
        order[rank] = b;
    }
    __syncthreads();
    int f = sh_flags;
    if (tt != T_expected) f |= kDataTokenCount;
    // per-sequence item counts scanned in longest-first order
    int64_t nq = 0, na = 0;
    if (b < B && f == 0) {
        const int64_t nt = (sL[sOrder[b]] + kTile - 1) / kTile;
        na = (int64_t)H * nt;
        nq = na * nt;
    }
    int64_t eq, ea2, tq, ta2;
    block_exclusive_scan2(nq, na, eq, ea2, tq, ta2, sh_a, sh_b);
    if (b < B) {
        qkt_item_off[b] = static_cast<int32_t>(min(eq, (int64_t)INT_MAX));
        av_item_off[b] = static_cast<int32_t>(min(ea2, (int64_t)INT_MAX));
    }
    if (b == 0) {
        if (tq > qkt_cap) f |= kDataQktCap;
        if (ta2 > av_cap) f |= kDataAvCap;
        tok_off[B] = static_cast<int32_t>(tt);
        att_off[B] = ta;
        qkt_item_off[B] = static_cast<int32_t>(min(tq, (int64_t)INT_MAX));
        av_item_off[B] = static_cast<int32_t>(min(ta2, (int64_t)INT_MAX));
        status[0] = f;
        status[1] = f ? 0 : static_cast<int32_t>(tq);
        status[2] = f ? 0 : static_cast<int32_t>(ta2);
        status[3] = sh_max;
    }
}

// Batches of at most kFusedBatch sequences: the whole prelude in one launch of B
// workgroups (plan_fused_body in plan_device.h, which the QKV projection's launch
// can also carry).
__global__ __launch_bounds__(kFusedBatch) void k_plan_fused(PlanFillArgs a) {
    __shared__ PlanSmem sm;
    plan_fused_body(a, blockIdx.x, sm);
}

// Workgroup k writes the items of the k-th longest sequence and its token map.
__global__ __launch_bounds__(256) void k_plan_fill(const int32_t* __restrict__ lengths,
                                                    const int32_t* __restrict__ order,
                                                    const int32_t* __restrict__ tok_off, int H,
                                                    const int32_t* __restrict__ qkt_item_off,
                                                    const int32_t* __restrict__ av_item_off,
                                                    int32_t* __restrict__ qkt_items,
                                                    int32_t* __restrict__ av_items,
                                                    int32_t* __restrict__ tok_seq,
                                                    const int32_t* __restrict__ status) {
    if (status[0] != 0) return;
    const int k = blockIdx.x;
    const int b = order[k];
    const int L = lengths[b];
    const int nt = (L + kTile - 1) / kTile;
    const int nq = H * nt * nt, na = H * nt;
    int4* q = reinterpret_cast<int4*>(qkt_items) + qkt_item_off[k];
    for (int idx = threadIdx.x; idx < nq; idx += 256) {
        const int h = idx / (nt * nt), r = idx - h * nt * nt;
        const int ti = r / nt, tj = r - ti * nt;
        q[idx] = make_int4(b, h, ti, tj);
    }
    int32_t* a = av_items + 3 * (int64_t)av_item_off[k];
    for (int idx = threadIdx.x; idx < na; idx += 256) {
        const int h = idx / nt, ti = idx - h * nt;
        a[3 * idx + 0] = b;
        a[3 * idx + 1] = h;
        a[3 * idx + 2] = ti;
    }
    const int t0 = tok_off[b];
    for (int t = threadIdx.x; t < L; t += 256) tok_seq[t0 + t] = b;
}

// ---------------------------------------------------------------------------
// Variable-sized batched GEMM prelude: packed-storage offsets, largest-first
// order, tile prefix and the flat tile list, in four launches like the plan
// above (scan, rank, tile scan, fill).
// ---------------------------------------------------------------------------

// Sizes as the offsets count them: negative ones are flagged and counted as 0,
// oversized ones flagged and clamped (so no sum can overflow).
__device__ __forceinline__ int64_t vgemm_dim(int v) { return v < 0 ? 0 : (v > kVgemmMaxDim ? kVgemmMaxDim : v); }

__global__ __launch_bounds__(kScanThreads) void k_vgemm_scan(const int32_t* __restrict__ dims, int B,
                                                              int64_t* __restrict__ a_off,
                                                              int64_t* __restrict__ b_off,
                                                              int64_t* __restrict__ c_off,
                                                              int32_t* __restrict__ status) {
    __shared__ int64_t sh_a[kScanWaves], sh_b[kScanWaves];
    __shared__ int sh_flags, sh_shape;
    if (threadIdx.x == 0) {
        sh_flags = 0;
        sh_shape = 0;
    }
    __syncthreads();
    int flags = 0, shape = 0;
    int64_t carry_a = 0, carry_b = 0, carry_c = 0;
    for (int base = 0; base < B; base += blockDim.x) {
        const int p = base + threadIdx.x;
        int64_t m = 0, n = 0, k = 0;
        if (p < B) {
            const int dm = dims[3 * p], dn = dims[3 * p + 1], dk = dims[3 * p + 2];
            if (dm < 0 || dn < 0 || dk < 0) flags |= kVgemmNegSize;
            if (dm > kVgemmMaxDim || dn > kVgemmMaxDim || dk > kVgemmMaxDim) flags |= kVgemmLargeSize;
            if (dk % 64 != 0 || dn % 8 != 0) shape = 1;
            m = vgemm_dim(dm);
            n = vgemm_dim(dn);
            k = vgemm_dim(dk);
        }
        int64_t ea, eb, ta, tb, ec, unused, tc, tu;
        block_exclusive_scan2(m * k, n * k, ea, eb, ta, tb, sh_a, sh_b);
        block_exclusive_scan2(m * n, 0, ec, unused, tc, tu, sh_a, sh_b);
        if (p < B) {
            a_off[p] = carry_a + ea;
            b_off[p] = carry_b + eb;
            c_off[p] = carry_c + ec;
        }
        carry_a += ta;
        carry_b += tb;
        carry_c += tc;
    }
    if (flags) atomicOr(&sh_flags, flags);
    if (shape) atomicOr(&sh_shape, shape);
    __syncthreads();
    if (threadIdx.x == 0) {
        a_off[B] = carry_a;
        b_off[B] = carry_b;
        c_off[B] = carry_c;
        status[0] = sh_flags;
        status[1] = 0;
        status[2] = sh_shape;
    }
}

// Same strict total order as k_plan_rank, on the multiply-add count m n k.
__global__ __launch_bounds__(256) void k_vgemm_rank(const int32_t* __restrict__ dims, int B,
                                                     int32_t* __restrict__ order) {
    __shared__ int64_t ws[256];
    const int p = blockIdx.x * 256 + threadIdx.x;
    const int64_t wp = p < B ? vgemm_dim(dims[3 * p]) * vgemm_dim(dims[3 * p + 1]) * vgemm_dim(dims[3 * p + 2]) : 0;
    int rank = 0;
    for (int base = 0; base < B; base += 256) {
        __syncthreads();
        const int q = base + threadIdx.x;
        ws[threadIdx.x] = q < B ? vgemm_dim(dims[3 * q]) * vgemm_dim(dims[3 * q + 1]) * vgemm_dim(dims[3 * q + 2]) : 0;
        __syncthreads();
        const int n = min(256, B - base);
        for (int j = 0; j < n; ++j) {
            const int64_t wq = ws[j];
            rank += (wq > wp) | ((wq == wp) & (base + j < p));
        }
    }
    if (p < B) order[rank] = p;
}

__device__ __forceinline__ int64_t vgemm_tiles(const int32_t* dims, int p) {
    return ((vgemm_dim(dims[3 * p]) + kVgemmTileM - 1) / kVgemmTileM) *
           ((vgemm_dim(dims[3 * p + 1]) + kVgemmTileN - 1) / kVgemmTileN);
}

__global__ __launch_bounds__(kScanThreads) void k_vgemm_tile_scan(const int32_t* __restrict__ dims,
                                                                   const int32_t* __restrict__ order, int B,
                                                                   int64_t tile_cap,
                                                                   int64_t* __restrict__ tile_off,
                                                                   int32_t* __restrict__ status) {
    __shared__ int64_t sh_a[kScanWaves], sh_b[kScanWaves];
    int64_t carry = 0;
    for (int base = 0; base < B; base += blockDim.x) {
        const int r = base + threadIdx.x;
        const int64_t nt = r < B ? vgemm_tiles(dims, order[r]) : 0;
        int64_t e, unused, t, tu;
        block_exclusive_scan2(nt, 0, e, unused, t, tu, sh_a, sh_b);
        if (r < B) tile_off[r] = carry + e;
        carry += t;
    }
    if (threadIdx.x == 0) {
        int f = status[0];
        if (carry > tile_cap) f |= kVgemmTileCap;
        tile_off[B] = carry;
        status[0] = f;
        status[1] = f ? 0 : static_cast<int32_t>(carry);
    }
}

// Workgroup r writes the tiles of the r-th largest problem, tile rows fastest.
__global__ __launch_bounds__(256) void k_vgemm_fill(const int32_t* __restrict__ dims,
                                                     const int32_t* __restrict__ order,
                                                     const int64_t* __restrict__ tile_off,
                                                     int32_t* __restrict__ tile_items,
                                                     const int32_t* __restrict__ status) {
    if (status[0] != 0) return;
    const int r = blockIdx.x;
    const int p = order[r];
    const int tm = static_cast<int>((vgemm_dim(dims[3 * p]) + kVgemmTileM - 1) / kVgemmTileM);
    const int n = static_cast<int>(tile_off[r + 1] - tile_off[r]);
    int4* out = reinterpret_cast<int4*>(tile_items) + tile_off[r];
    for (int idx = threadIdx.x; idx < n; idx += 256) out[idx] = make_int4(p, idx % tm, idx / tm, 0);
}

}  // namespace

hipError_t launch_vgemm_offsets(const VgemmView& p, hipStream_t s) {
    // one thread per problem up to kScanThreads (a smaller workgroup synchronises faster)
    const int threads = std::min(kScanThreads, (p.batch + kWave - 1) / kWave * kWave);
    hipLaunchKernelGGL(k_vgemm_scan, dim3(1), dim3(threads), 0, s, p.dims, p.batch, p.a_off, p.b_off, p.c_off,
                       p.status);
    hipLaunchKernelGGL(k_vgemm_rank, dim3((p.batch + 255) / 256), dim3(256), 0, s, p.dims, p.batch, p.order);
    hipLaunchKernelGGL(k_vgemm_tile_scan, dim3(1), dim3(threads), 0, s, p.dims, p.order, p.batch, p.tile_cap,
                       p.tile_off, p.status);
    hipLaunchKernelGGL(k_vgemm_fill, dim3(p.batch), dim3(256), 0, s, p.dims, p.order, p.tile_off, p.tile_items,
                       p.status);
    return hipGetLastError();
}

hipError_t launch_offsets(const PlanView& p, hipStream_t s) {
    if (p.batch <= kFusedBatch) {
        hipLaunchKernelGGL(k_plan_fused, dim3(p.batch), dim3(kFusedBatch), 0, s, plan_fill_args(p));
        return hipGetLastError();
    }
    if (p.batch <= kScanThreads) {
        const int threads = (p.batch + kWave - 1) / kWave * kWave;  // one thread per sequence
        hipLaunchKernelGGL(k_plan_small, dim3(1), dim3(threads), 0, s, p.lengths, p.batch, p.total_tokens,
                           p.max_len, p.heads, p.qkt_cap, p.av_cap, p.tok_off, p.att_off, p.order, p.qkt_item_off,
                           p.av_item_off, p.status);
        hipLaunchKernelGGL(k_plan_fill, dim3(p.batch), dim3(256), 0, s, p.lengths, p.order, p.tok_off, p.heads,
                           p.qkt_item_off, p.av_item_off, p.qkt_items, p.av_items, p.tok_seq, p.status);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(k_plan_scan, dim3(1), dim3(kScanThreads), 0, s, p.lengths, p.batch, p.total_tokens,
                       p.max_len, p.heads, p.tok_off, p.att_off, p.status);
    hipLaunchKernelGGL(k_plan_rank, dim3((p.batch + 255) / 256), dim3(256), 0, s, p.lengths, p.batch, p.order);
    hipLaunchKernelGGL(k_plan_items, dim3(1), dim3(kScanThreads), 0, s, p.lengths, p.order, p.batch, p.heads,
                       p.qkt_cap, p.av_cap, p.qkt_item_off, p.av_item_off, p.status);
    hipLaunchKernelGGL(k_plan_fill, dim3(p.batch), dim3(256), 0, s, p.lengths, p.order, p.tok_off, p.heads,
                       p.qkt_item_off, p.av_item_off, p.qkt_items, p.av_items, p.tok_seq, p.status);
    return hipGetLastError();
}

}  // namespace rag
