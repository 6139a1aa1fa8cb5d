// The prelude of batches of at most kFusedBatch sequences as one workgroup's
// work: every workgroup computes the scans, the rank and the item offsets itself
// (one thread per sequence; a few hundred LDS operations), so none waits for
// another: workgroup 0 also writes the global arrays and the status, and
// workgroup `me` writes the items and token map of the me-th longest sequence.
// Shared by the prelude's own launch and the QKV projection's launch, which can
// carry these workgroups behind its tiles (the projection does not read the plan).
#pragma once

#include <climits>

#include "device_common.h"
#include "launch.h"

namespace rag {

constexpr int kFusedBatch = 256;        // the largest batch (one thread per sequence)
constexpr int kFusedMaxThreads = 512;   // workgroups of kFusedBatch or kFusedMaxThreads threads

struct PlanFillArgs {
    const int32_t* lengths;
    int B, T_expected, max_len, H;
    int64_t qkt_cap, av_cap;
    int32_t* tok_off;
    int64_t* att_off;
    int32_t* order;
    int32_t* qkt_item_off;
    int32_t* av_item_off;
    int32_t* qkt_items;
    int32_t* av_items;
    int32_t* tok_seq;
    int32_t* status;
};

struct PlanSmem {
    int64_t sh_a[kFusedMaxThreads / kWave], sh_b[kFusedMaxThreads / kWave];
    __attribute__((aligned(16))) int32_t sL[kFusedBatch];
    int32_t sOrder[kFusedBatch];
    int flags, max, t0, qoff, aoff;
};

// Inclusive prefix sum across one wave (64-bit values).
__device__ __forceinline__ int64_t wave_inclusive_scan(int64_t v, int lane) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int64_t t = __shfl_up(v, o, kWave);
        if (lane >= o) v += t;
    }
    return v;
}

// Block-wide exclusive scan of two 64-bit sequences (one value per thread);
// returns each thread's exclusive prefixes and the block totals.  All threads
// of the block must call it.
__device__ __forceinline__ void block_exclusive_scan2(int64_t a, int64_t b, int64_t& ea, int64_t& eb,
                                                      int64_t& ta, int64_t& tb, int64_t* sh_a,
                                                      int64_t* sh_b) {
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    int64_t ia = wave_inclusive_scan(a, lane);
    int64_t ib = wave_inclusive_scan(b, lane);
    if (lane == kWave - 1) {
        sh_a[wid] = ia;
        sh_b[wid] = ib;
    }
    __syncthreads();
    int64_t pa = 0, pb = 0;
    ta = 0;
    tb = 0;
    const int nw = blockDim.x / kWave;  // the launch may use fewer than kScanThreads threads
    for (int w = 0; w < nw; ++w) {
        if (w < wid) {
            pa += sh_a[w];
            pb += sh_b[w];
        }
        ta += sh_a[w];
        tb += sh_b[w];
    }
    ea = pa + ia - a;
    eb = pb + ib - b;
    __syncthreads();  // the shared totals may be overwritten by the next call
}

inline PlanFillArgs plan_fill_args(const PlanView& p) {
    return PlanFillArgs{p.lengths, p.batch,       p.total_tokens, p.max_len,      p.heads,
                        p.qkt_cap, p.av_cap,      p.tok_off,      p.att_off,      p.order,
                        p.qkt_item_off, p.av_item_off, p.qkt_items, p.av_items,   p.tok_seq,
                        p.status};
}

// Called by every thread of a workgroup of kFusedBatch or kFusedMaxThreads
// threads; thread b < B stands for sequence b, the others only take part in the
// scans and share the item filling.
__device__ __forceinline__ void plan_fused_body(const PlanFillArgs& a, int me, PlanSmem& sm) {
    int64_t* const sh_a = sm.sh_a;
    int64_t* const sh_b = sm.sh_b;
    int32_t* const sL = sm.sL;
    int32_t* const sOrder = sm.sOrder;
    int& sh_flags = sm.flags;
    int& sh_max = sm.max;
    int& sh_t0 = sm.t0;
    int& sh_qoff = sm.qoff;
    int& sh_aoff = sm.aoff;
    const int b = threadIdx.x;
    const int* const lengths = a.lengths;
    const int B = a.B, T_expected = a.T_expected, max_len = a.max_len, H = a.H;
    const int64_t qkt_cap = a.qkt_cap, av_cap = a.av_cap;
    int32_t* const tok_off = a.tok_off;
    int64_t* const att_off = a.att_off;
    int32_t* const order = a.order;
    int32_t* const qkt_item_off = a.qkt_item_off;
    int32_t* const av_item_off = a.av_item_off;
    int32_t* const qkt_items = a.qkt_items;
    int32_t* const av_items = a.av_items;
    int32_t* const tok_seq = a.tok_seq;
    int32_t* const status = a.status;
    const bool lead = me == 0;
    if (b == 0) {
        sh_flags = 0;
        sh_max = 0;
    }
    const int L = b < B ? lengths[b] : 0;
    if (b < kFusedBatch) sL[b] = b < B ? L : -1;  // padding never outranks a length
    int flags = 0;
    if (b < B) {
        if (L < 0) flags |= kDataNegLength;
        if (L > max_len) flags |= kDataLongLength;
    }
    __syncthreads();
    if (flags) atomicOr(&sh_flags, flags);
    if (b < B) atomicMax(&sh_max, L);
    const int64_t Lc = L > 0 ? L : 0;
    int64_t et, ea, tt, ta;
    block_exclusive_scan2(Lc, (int64_t)H * Lc * Lc, et, ea, tt, ta, sh_a, sh_b);
    if (lead && b < B) {
        tok_off[b] = static_cast<int32_t>(et);
        att_off[b] = ea;
    }
    if (b < B) {
        int rank = 0;
#pragma unroll 2
        for (int k = 0; k < B; k += 4) {
            const int4 l4 = *reinterpret_cast<const int4*>(sL + k);
            rank += (l4.x > L) | ((l4.x == L) & (k < b));
            rank += (l4.y > L) | ((l4.y == L) & (k + 1 < b));
            rank += (l4.z > L) | ((l4.z == L) & (k + 2 < b));
            rank += (l4.w > L) | ((l4.w == L) & (k + 3 < b));
        }
        sOrder[rank] = b;
        if (lead) order[rank] = b;
    }
    __syncthreads();
    int f = sh_flags;
    if (tt != T_expected) f |= kDataTokenCount;
    int64_t nq = 0, na = 0;
    if (b < B && f == 0) {
        const int64_t nt = (sL[sOrder[b]] + kTile - 1) / kTile;
        na = (int64_t)H * nt;
        nq = na * nt;
    }
    int64_t eq, ea2, tq, ta2;
    block_exclusive_scan2(nq, na, eq, ea2, tq, ta2, sh_a, sh_b);
    if (tq > qkt_cap) f |= kDataQktCap;
    if (ta2 > av_cap) f |= kDataAvCap;
    if (lead) {
        if (b < B) {
            qkt_item_off[b] = static_cast<int32_t>(min(eq, (int64_t)INT_MAX));
            av_item_off[b] = static_cast<int32_t>(min(ea2, (int64_t)INT_MAX));
        }
        if (b == 0) {
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
    if (f != 0) return;  // uniform: every workgroup derived the same flags
    // this workgroup's sequence: the me-th longest
    if (b == me) {
        sh_qoff = static_cast<int32_t>(eq);
        sh_aoff = static_cast<int32_t>(ea2);
    }
    if (b < B && b == sOrder[me]) sh_t0 = static_cast<int32_t>(et);
    __syncthreads();
    const int sb = sOrder[me];
    const int Ls = sL[sb];
    const int nt = (Ls + kTile - 1) / kTile;
    const int nqs = H * nt * nt, nas = H * nt;
    int4* q = reinterpret_cast<int4*>(qkt_items) + sh_qoff;
    for (int idx = b; idx < nqs; idx += blockDim.x) {
        const int h = idx / (nt * nt), r = idx - h * nt * nt;
        const int ti = r / nt, tj = r - ti * nt;
        q[idx] = make_int4(sb, h, ti, tj);
    }
    int32_t* const av = av_items + 3 * (int64_t)sh_aoff;
    for (int idx = b; idx < nas; idx += blockDim.x) {
        const int h = idx / nt, ti = idx - h * nt;
        av[3 * idx + 0] = sb;
        av[3 * idx + 1] = h;
        av[3 * idx + 2] = ti;
    }
    const int t0 = sh_t0;
    for (int t = b; t < Ls; t += blockDim.x) tok_seq[t0 + t] = sb;
}

}  // namespace rag
