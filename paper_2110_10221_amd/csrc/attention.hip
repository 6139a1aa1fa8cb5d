// Ragged scaled dot-product attention over the plan's work lists: the paper's
// QK^T, Softmax and AttnV operators one by one, and the three fused.
//   ragged QK^T     bf16: one workgroup item = one (sequence, head, 64-query
//                   block), walking every 64-key tile of its rows; fp32: one
//                   item = one 64x64 score tile.  No tile crosses a sequence
//                   boundary, so no padded work is done beyond predicated edges
//   ragged softmax  one wave per token: the token's H rows (each L_b scores)
//                   are contiguous in the X[b][i][h][j] layout
//   ragged Attn.V   one workgroup item = 64 query rows of one sequence and head,
//                   reducing over that sequence's L_b keys
//   fused           one (sequence, head, 64-query tile) item per two-wave
//                   workgroup, keys streamed through LDS (details further down)
// The operators' persistent grids walk the lists in order: sequences longest first.
//
// The unfused bf16 kernels use v_mfma_f32_16x16x32_bf16.  In a 16x16x32 MFMA lane l
// supplies row (l % 16) of A and column (l % 16) of B, each with the 8 consecutive
// k values 8*(l/16) .. 8*(l/16)+7, and receives C rows 4*(l/16) .. 4*(l/16)+3 of
// column l % 16.
#include <algorithm>
#include <cfloat>

#include "device_common.h"
#include "launch.h"

namespace rag {
namespace {

struct PlanArgs {
    const int32_t* lengths;
    const int32_t* tok_off;
    const int64_t* att_off;
    const int32_t* tok_seq;
    const int32_t* qkt_items;
    const int32_t* av_items;
    const int32_t* order;
    const int32_t* av_item_off;
    int32_t* status;
    int batch, heads;
};

PlanArgs plan_args(const PlanView& p) {
    return PlanArgs{p.lengths, p.tok_off, p.att_off, p.tok_seq, p.qkt_items, p.av_items, p.order, p.av_item_off,
                    p.status, p.batch, p.heads};
}

// True if the plan is valid and the score buffer large enough; otherwise one
// thread records the overflow and every workgroup returns.
__device__ __forceinline__ bool plan_ok(const PlanArgs& pa, int64_t score_cap) {
    if (pa.status[0] != 0) return false;
    if (pa.att_off[pa.batch] > score_cap) {
        if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(pa.status, kDataScoreCap);
        return false;
    }
    return true;
}

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }

// The status word is written in these kernels (atomicOr), so the compiler cannot
// keep plan reads in scalar registers by itself; values that are uniform over the
// workgroup are made so explicitly (a buffer descriptor built from a per-lane value
// becomes a loop over lanes).
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int64_t uni64(int64_t v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(static_cast<uint64_t>(v) >> 32));
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// ---------------------------------------------------------------------------
// QK^T
// ---------------------------------------------------------------------------

typedef __attribute__((address_space(3))) void lds_void_t;

// Element offset of (row, col) in [rows][64 channels] LDS storage (128-byte rows,
// two per 256-byte bank line) whose 16-byte chunks are XOR-swizzled by row bits
// 1-3: the K-operand reads (16 consecutive rows, one chunk each) then meet 16
// distinct bank groups, and in the transposed V reads (rows r..r+3, four
// adjacent chunks each) rows r and r+2 use opposite halves of the row.
__device__ __forceinline__ int kv_swz(int row) { return (((row >> 1) & 1) << 2) | ((row >> 2) & 3); }
__device__ __forceinline__ int kv_off(int row, int col) { return row * kHeadDim + ((((col >> 3) ^ kv_swz(row)) & 7) << 3) + (col & 7); }

// The bf16 operators take one work item per (sequence, 64-query block, group of
// G consecutive heads), G a divisor of H chosen at launch so that the batch
// makes enough items to fill the GPU.  In the X[b][i][h][j] layout the item's
// scores are G * L_b contiguous values per query row (all of them, one region,
// when G = H), so a workgroup reads or writes whole cache lines, and the item
// reads each of its heads' K (or V) panels of the sequence once.  Items follow
// the plan's Attn.V list (sequences longest first, then head groups, then query
// blocks); a workgroup finds its item's sequence by a wave-wide search of the
// per-sequence item prefix, and consecutive items (the query blocks of one head
// group) go to one XCD in runs, so they share its K / V panels in that L2.
constexpr int kOpRun = 8;  // consecutive items per XCD

// Largest k with off[k] / G <= g: the sorted sequence holding item g (off holds
// H entries per 64-query block of each sequence, so off[k] / G counts the items
// of G heads each, G a divisor of H).
__device__ __forceinline__ int item_sequence(const int32_t* off, int B, int G, int g) {
    const int lane = threadIdx.x % kWave;
    int lo = 0, span = B;
    while (span > 1) {
        const int st = (span + kWave - 1) / kWave;
        const bool le = lane * st < span && off[lo + lane * st] / G <= g;
        const uint64_t m = __ballot(le);  // lane 0 always holds (off[lo] / G <= g)
        const int last = 63 - __builtin_clzll(m);
        lo += last * st;
        span = min(st, span - last * st);
    }
    return lo;
}

__device__ __forceinline__ int op_item(int bid, int grid) {  // grid: a multiple of 8 * kOpRun
    const int xcd = bid % 8, j = bid / 8;
    return ((j / kOpRun) * 8 + xcd) * kOpRun + j % kOpRun;
}

// bf16 QK^T.  Per head of the item and piece of kPiece keys, wave w computes the
// piece's key tile w for all 64 query rows of the block (v_mfma_f32_16x16x32_bf16,
// K fragments straight from memory, the next piece's tile loaded while this one
// is computed), scaled and rounded into the workgroup's LDS rows; then all
// threads write the piece's row pieces as aligned 16-byte chunks (a row starts at
// any element, so a chunk is cut from two LDS chunks by a funnel shift), and
// 2-byte stores for the partial chunks at both ends of each row piece.
constexpr int kPiece = 4 * kTile;         // keys per written row piece: one tile per wave
constexpr int kPieceRow = kPiece + 4;     // LDS row (elements): room for the shifted read
constexpr int kQkWaves = 8, kQkThreads = kQkWaves * kWave;
constexpr int kQkKeys = kPiece / kQkWaves;  // keys of a piece per wave
constexpr int kQkJb = kQkKeys / 16;         // 16-key MFMA blocks per wave

__global__ __launch_bounds__(kQkThreads) void k_qkt_bf16(PlanArgs pa, const uint16_t* __restrict__ q, int ldq,
                                                   const uint16_t* __restrict__ k, int ldk, float scale,
                                                   uint16_t* __restrict__ S, int64_t score_cap, int causal, int G) {
    if (!plan_ok(pa, score_cap)) return;
    __shared__ __attribute__((aligned(16))) uint16_t st[kTile][kPieceRow];
    __shared__ __attribute__((aligned(16))) uint16_t qs[2][kTile * kHeadDim];  // a head's Q block, two buffers
    const int H = pa.heads;
    const int n_items = pa.status[2] / G;
    const int wave = uni(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const int l16 = lane % 16, q4 = lane / 16;
    for (int base_it = 0; base_it < n_items; base_it += gridDim.x) {
        const int g = base_it + op_item(blockIdx.x, gridDim.x);
        if (g >= n_items) break;
        const int kk = uni(item_sequence(pa.av_item_off, pa.batch, G, g));
        const int b = uni(pa.order[kk]);
        const int local = g - uni(pa.av_item_off[kk]) / G;
        const int nb = (uni(pa.lengths[b]) + kTile - 1) / kTile;  // query blocks of the sequence
        const int hg = local / nb, ti = local - hg * nb, h0 = hg * G;  // heads h0 .. h0 + G - 1
        const int L = uni(pa.lengths[b]);
        const int t0 = uni(pa.tok_off[b]);
        const int64_t base = uni64(pa.att_off[b]);
        const int i0 = ti * kTile;                // the block's first query row
        const int rows = min(kTile, L - i0);
        // keys the block needs: all, or (masked) up to its last row
        const int kend = causal ? min(L, i0 + rows) : L;
        const int npc = (kend + kPiece - 1) / kPiece;  // pieces per head
        const int F = G * npc;
        // this wave's keys of piece f: head h0 + f / npc, keys (f % npc) * kPiece + kQkKeys wave ..
        bf16x8 kc[kQkJb][2], kn[kQkJb][2], qf[4][2];
        // the Q block (rows i0 .. i0 + 63, rows past L as zeros) of head h0 + j into
        // qs[j & 1] by direct copies: wave w fills rows 8 w .. 8 w + 7 (one 1 KB
        // block), 16-byte chunks swizzled as in kv_off
        auto copy_q = [&](int j) {
            const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<uint16_t*>(q + (int64_t)(t0 + i0) * ldq + (h0 + j) * kHeadDim), 0,
                (uint32_t)rows * ldq * 2u, 0x00020000);
            static_assert(kQkWaves * 8 == kTile, "one 8-row block of Q per wave");
            const int row = wave * 8 + lane / 8;
            const int off = row * ldq * 2 + (((lane % 8) ^ kv_swz(row)) * 16);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (lds_void_t*)(&qs[j & 1][wave * 512]), 16, off, 0, 0, 0);
        };
        copy_q(0);
        auto load_k = [&](int f, bf16x8 (&kb)[kQkJb][2]) {
            const int h = h0 + f / npc, k0 = (f % npc) * kPiece + wave * kQkKeys;
#pragma unroll
            for (int jb = 0; jb < kQkJb; ++jb) {
                const int kj = min(k0 + jb * 16 + l16, L - 1);
                const uint16_t* krow = k + (int64_t)(t0 + kj) * ldk + h * kHeadDim + 8 * q4;
                kb[jb][0] = as_bf16x8(ld16(krow));
                kb[jb][1] = as_bf16x8(ld16(krow + 32));
            }
        };
        load_k(0, kc);
        for (int f = 0; f < F; ++f) {
            const int h = h0 + f / npc, p0 = (f % npc) * kPiece;
            if (f % npc == 0) {  // a new head: its Q block has landed (all waves' copies)
                const int j = f / npc;
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                __syncthreads();
                // its Q fragments, rows rg*16 + l16, read before the next head's copy goes
                // out (an LDS read after a pending LDS copy waits for the copy)
                const uint16_t* qb = qs[j & 1];
#pragma unroll
                for (int rg = 0; rg < 4; ++rg) {
                    qf[rg][0] = as_bf16x8(*reinterpret_cast<const u32x4*>(qb + kv_off(rg * 16 + l16, 8 * q4)));
                    qf[rg][1] = as_bf16x8(*reinterpret_cast<const u32x4*>(qb + kv_off(rg * 16 + l16, 32 + 8 * q4)));
                }
                if (j + 1 < G) copy_q(j + 1);  // qs[(j + 1) & 1] was last read by head j - 1
            }
            if (f + 1 < F) load_k(f + 1, kn);
            const int pn = min(kPiece, kend - p0);
            const bool mine = wave * kQkKeys < pn;  // this wave's keys include keys of the piece
            floatx4 acc[kQkJb][4];
            if (mine) {
#pragma unroll
                for (int jb = 0; jb < kQkJb; ++jb)
#pragma unroll
                    for (int rg = 0; rg < 4; ++rg) {
                        acc[jb][rg] = floatx4{0.f, 0.f, 0.f, 0.f};
                        acc[jb][rg] = mfma16x16x32(kc[jb][0], qf[rg][0], acc[jb][rg]);  // C[j][i] = K[j] . Q[i]
                        acc[jb][rg] = mfma16x16x32(kc[jb][1], qf[rg][1], acc[jb][rg]);
                    }
            }
            __syncthreads();  // the previous piece's LDS rows are written out
            if (mine) {
#pragma unroll
                for (int jb = 0; jb < kQkJb; ++jb)
#pragma unroll
                    for (int rg = 0; rg < 4; ++rg)
                        *reinterpret_cast<u32x2*>(&st[rg * 16 + l16][wave * kQkKeys + jb * 16 + 4 * q4]) =
                            u32x2{pack_bf16x2(acc[jb][rg][0] * scale, acc[jb][rg][1] * scale),
                                  pack_bf16x2(acc[jb][rg][2] * scale, acc[jb][rg][3] * scale)};
            }
            __syncthreads();
            // Row r (threads 8 r .. 8 r + 7) holds keys p0 .. p0 + n - 1 at elements G0 ..
            // G0 + n - 1 of S.  Its whole 16-byte chunks fa .. fb - 1 start at local key
            // sh + 8 (c - fa), sh = 8 fa - G0 the same for every chunk of the row: five
            // dwords read from LDS at dword 4 (c - fa) + sh / 2, funneled by 2 (sh & 1)
            // bytes, give the chunk.  The partial chunks at both ends (under 8 elements
            // each) are 2-byte stores, one per thread and end.
            {
                const int r = threadIdx.x >> 3, sub = threadIdx.x & 7;
                const int n = causal ? min(pn, i0 + r + 1 - p0) : pn;
                if (r < rows && n > 0) {
                    const int64_t G0 = base + ((int64_t)(i0 + r) * H + h) * L + p0;
                    const int64_t fa = (G0 + 7) >> 3, fb = (G0 + n) >> 3;
                    const int sh = (int)(8 * fa - G0);  // 0 .. 7
                    const int nch = (int)(fb - fa);     // may be negative for a short row
                    const uint32_t* const src = reinterpret_cast<const uint32_t*>(&st[r][0]) + (sh >> 1);
                    const uint32_t rb = (sh & 1) * 2;
                    uint16_t* const dst = S + 8 * fa;
                    for (int cc = sub; cc < nch; cc += 8) {
                        // the five dwords by LDS reads the compiler does not see, so it adds
                        // no wait for the Q copy that may be in flight (it cannot tell the
                        // buffers apart)
                        const uint32_t da = (uint32_t)(uintptr_t)(src + 4 * cc);
                        u32x2 d01, d23;
                        uint32_t d4;
                        asm volatile(
                            "ds_read2_b32 %0, %3 offset1:1\n\tds_read2_b32 %1, %3 offset0:2 offset1:3\n\t"
                            "ds_read_b32 %2, %3 offset:16\n\ts_waitcnt lgkmcnt(0)"
                            : "=&v"(d01), "=&v"(d23), "=&v"(d4)
                            : "v"(da)
                            : "memory");
                        const uint32_t d0 = d01[0], d1 = d01[1], d2 = d23[0], d3 = d23[1];
                        *reinterpret_cast<u32x4*>(dst + 8 * cc) =
                            u32x4{__builtin_amdgcn_alignbyte(d1, d0, rb), __builtin_amdgcn_alignbyte(d2, d1, rb),
                                  __builtin_amdgcn_alignbyte(d3, d2, rb), __builtin_amdgcn_alignbyte(d4, d3, rb)};
                    }
                    const int head = min(sh, n), tail0 = max((int)(8 * fb - G0), head);
                    if (sub < head) S[G0 + sub] = st[r][sub];
                    if (tail0 + sub < n) S[G0 + tail0 + sub] = st[r][tail0 + sub];
                }
            }
            if (f + 1 < F) {
#pragma unroll
                for (int jb = 0; jb < kQkJb; ++jb) {
                    kc[jb][0] = kn[jb][0];
                    kc[jb][1] = kn[jb][1];
                }
            }
        }
        __syncthreads();  // the last piece's rows are written out before the next item stages
    }
}

// fp32 QK^T: one 64 x 64 score tile per item, Q and K rows staged in LDS; wave w
// computes the 32 x 32 block (queries 32 (w / 2) .., keys 32 (w % 2) ..) on
// v_mfma_f32_32x32x2f32 (fp32 products and accumulation).  A lane holds key
// l % 32 of the block and queries 8 (r / 4) + 4 (l / 32) + r % 4, so each
// accumulator register is stored as 32 consecutive floats of one score row.
// Row stride 66 floats: the 64 lanes of an operand read (row l % 32, column
// c + l / 32) fall in 64 distinct banks.
constexpr int kF32Row = kHeadDim + 2;

__global__ __launch_bounds__(256) void k_qkt_f32(PlanArgs pa, const float* __restrict__ q, int ldq,
                                                  const float* __restrict__ k, int ldk, float scale,
                                                  float* __restrict__ S, int64_t score_cap, int causal) {
    if (!plan_ok(pa, score_cap)) return;
    __shared__ float Qs[kTile][kF32Row], Ks[kTile][kF32Row];
    const int n_items = pa.status[1];
    const int H = pa.heads;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int l32 = lane % 32, h2 = lane / 32;
    const int wq = wave >> 1, wk = wave & 1;
    for (int it = blockIdx.x; it < n_items; it += gridDim.x) {
        const int4 item = reinterpret_cast<const int4*>(pa.qkt_items)[it];
        const int b = item.x, h = item.y, ti = item.z, tj = item.w;
        if (causal && tj > ti) continue;
        const int L = pa.lengths[b];
        const int t0 = pa.tok_off[b];
        const int64_t base = pa.att_off[b];
        __syncthreads();
        for (int e = threadIdx.x; e < kTile * kHeadDim; e += 256) {
            const int r = e / kHeadDim, c = e % kHeadDim;
            const int qi = min(ti * kTile + r, L - 1), kj = min(tj * kTile + r, L - 1);
            Qs[r][c] = q[(int64_t)(t0 + qi) * ldq + h * kHeadDim + c];
            Ks[r][c] = k[(int64_t)(t0 + kj) * ldk + h * kHeadDim + c];
        }
        __syncthreads();
        floatx16 acc;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll 8
        for (int c = 0; c < kHeadDim; c += 2)
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(Qs[wq * 32 + l32][c + h2], Ks[wk * 32 + l32][c + h2], acc, 0, 0, 0);
        const int rows = min(kTile, L - ti * kTile), cols = min(kTile, L - tj * kTile);
        const int j = wk * 32 + l32;
        if (j < cols) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int i = wq * 32 + 8 * (r / 4) + 4 * h2 + r % 4;
                if (i < rows && (!causal || tj * kTile + j <= ti * kTile + i))
                    S[base + ((int64_t)(ti * kTile + i) * H + h) * L + tj * kTile + j] = acc[r] * scale;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Softmax
// ---------------------------------------------------------------------------

template <bool BF16>
struct Elem;
template <>
struct Elem<true> {
    using T = uint16_t;
    static __device__ __forceinline__ float load(const T* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ void store(T* p, float v) { *p = f32_to_bf16(v); }
    static __device__ __forceinline__ float exp(float x) { return __expf(x); }
};
template <>
struct Elem<false> {
    using T = float;
    static __device__ __forceinline__ float load(const T* p) { return *p; }
    static __device__ __forceinline__ void store(T* p, float v) { *p = v; }
    static __device__ __forceinline__ float exp(float x) { return expf(x); }
};

constexpr int kSoftmaxRegs = 8;  // rows up to 64 * 8 = 512 scores stay in registers

// One bf16 score row of n values starting at element E (any alignment) with R
// aligned 16-byte chunks per lane (n + 7 <= 512 R): loads through the
// range-checked descriptor rs (based at element e_base, a multiple of 8), an
// exact max and sum over the row, whole chunks stored with 16-byte stores and
// the partial chunks at both ends element by element (their other elements
// belong to the neighbouring rows, so a whole-chunk store could race with them).
template <int R>
__device__ __forceinline__ void softmax_row_chunks(__amdgpu_buffer_rsrc_t rs, int64_t e_base, int64_t E, int n,
                                                   uint16_t* P, int lane) {
    const int64_t c0 = E >> 3;        // first chunk of the row
    const int sh = (int)(E & 7);      // the row's first element within it
    const int nch = (sh + n + 7) >> 3;
    float x[R][8];
    float m = -FLT_MAX;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int c = lane + kWave * r;
        u32x4 raw = {0u, 0u, 0u, 0u};
        if (c < nch)
            raw = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)((c0 + c) * 8 - e_base) * 2, 0, 0));
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int j = 8 * c + e - sh;
            const uint32_t w = raw[e >> 1];
            const float v = __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
            x[r][e] = (j >= 0 && j < n) ? v : -FLT_MAX;
            m = fmaxf(m, x[r][e]);
        }
    }
    m = wave_max(m);
    float sum = 0.f;
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int j = 8 * (lane + kWave * r) + e - sh;
            x[r][e] = (j >= 0 && j < n) ? __expf(x[r][e] - m) : 0.f;
            sum += x[r][e];
        }
    const float inv = 1.0f / wave_sum(sum);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int c = lane + kWave * r;
        if (c >= nch) continue;
        const int j0 = 8 * c - sh;  // row position of the chunk's first element
        uint16_t* dst = P + (c0 + c) * 8;
        if (j0 >= 0 && j0 + 8 <= n) {
            u32x4 o;
#pragma unroll
            for (int d = 0; d < 4; ++d) o[d] = pack_bf16x2(x[r][2 * d] * inv, x[r][2 * d + 1] * inv);
            *reinterpret_cast<u32x4*>(dst) = o;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (j0 + e >= 0 && j0 + e < n) dst[e] = f32_to_bf16(x[r][e] * inv);
        }
    }
}

template <bool BF16>
__global__ __launch_bounds__(256) void k_softmax(PlanArgs pa, const typename Elem<BF16>::T* S,
                                                  typename Elem<BF16>::T* P, int64_t score_cap, int T, int causal) {
    using E = Elem<BF16>;
    if (!plan_ok(pa, score_cap)) return;
    // wave-uniform by construction; made explicit so that the token's offsets and
    // the score rows' buffer descriptor stay in scalar registers
    const int wave = uni(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const int t = blockIdx.x * 4 + wave;
    if (t >= T) return;
    const int b = pa.tok_seq[t];
    const int H = pa.heads;
    const int ld = pa.lengths[b];                 // row stride: the sequence length
    const int pos = t - pa.tok_off[b];
    const int L = causal ? pos + 1 : ld;          // scores in each of this token's rows
    const int64_t row0 = pa.att_off[b] + (int64_t)pos * H * ld;
    if (L <= kWave) {
        // 64/G rows per pass, G = next power of two >= L lanes per row
        int G = 1;
        while (G < L) G <<= 1;
        const int R = kWave / G, r = lane / G, e = lane % G;
        for (int h0 = 0; h0 < H; h0 += R) {
            const int h = h0 + r;
            const bool valid = (h < H) && (e < L);
            const int64_t off = row0 + (int64_t)h * ld + e;
            const float x = valid ? E::load(S + off) : -FLT_MAX;
            const float m = group_max(x, G);
            const float ex = valid ? E::exp(x - m) : 0.f;
            const float s = group_sum(ex, G);
            if (valid) E::store(P + off, ex * (1.0f / s));
        }
    } else if (BF16 && L + 7 <= 8 * kWave * 2) {
        // aligned 16-byte chunks: the token's rows are one span of H * ld scores
        const int64_t e_base = row0 & ~(int64_t)7;
        const int64_t span_end = min(score_cap, row0 + (int64_t)(H - 1) * ld + L);
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<void*>(static_cast<const void*>(S + e_base)), 0,
            (uint32_t)min<int64_t>(((span_end - e_base) * 2 + 3) & ~(int64_t)3, (int64_t)0x7ffffffc), 0x00020000);
        uint16_t* const Pb = reinterpret_cast<uint16_t*>(P);
        if (L + 7 <= 8 * kWave) {
            for (int h = 0; h < H; ++h) softmax_row_chunks<1>(rs, e_base, row0 + (int64_t)h * ld, L, Pb, lane);
        } else {
            for (int h = 0; h < H; ++h) softmax_row_chunks<2>(rs, e_base, row0 + (int64_t)h * ld, L, Pb, lane);
        }
    } else if (L <= kWave * kSoftmaxRegs) {
        for (int h = 0; h < H; ++h) {
            const int64_t rp = row0 + (int64_t)h * ld;
            float x[kSoftmaxRegs];
            float m = -FLT_MAX;
#pragma unroll
            for (int u = 0; u < kSoftmaxRegs; ++u) {
                const int j = lane + kWave * u;
                x[u] = j < L ? E::load(S + rp + j) : -FLT_MAX;
                m = fmaxf(m, x[u]);
            }
            m = wave_max(m);
            float s = 0.f;
#pragma unroll
            for (int u = 0; u < kSoftmaxRegs; ++u) {
                const int j = lane + kWave * u;
                x[u] = j < L ? E::exp(x[u] - m) : 0.f;
                s += x[u];
            }
            const float inv = 1.0f / wave_sum(s);
#pragma unroll
            for (int u = 0; u < kSoftmaxRegs; ++u) {
                const int j = lane + kWave * u;
                if (j < L) E::store(P + rp + j, x[u] * inv);
            }
        }
    } else {
        // long rows: max pass, sum pass, write pass (each element is read before
        // the same lane overwrites it, so in-place use is safe)
        for (int h = 0; h < H; ++h) {
            const int64_t rp = row0 + (int64_t)h * ld;
            float m = -FLT_MAX;
            for (int j = lane; j < L; j += kWave) m = fmaxf(m, E::load(S + rp + j));
            m = wave_max(m);
            float s = 0.f;
            for (int j = lane; j < L; j += kWave) s += E::exp(E::load(S + rp + j) - m);
            const float inv = 1.0f / wave_sum(s);
            for (int j = lane; j < L; j += kWave) E::store(P + rp + j, E::exp(E::load(S + rp + j) - m) * inv);
        }
    }
}

// ---------------------------------------------------------------------------
// Attn.V
// ---------------------------------------------------------------------------

// bf16 Attn.V over the same items as QK^T (one sequence's 64-query block, all
// heads): the probabilities of the item are one contiguous region.  Per tile of
// 64 keys, each of the block's 64 probability rows is copied to LDS as the ten
// aligned 16-byte chunks from the one holding its first key on (range-checked
// direct copies; chunks past the item read as zeros and are masked), and a lane
// takes its 8 keys as five dwords at the row's element shift, funneled by one
// byte-align per dword.  V tiles (64 keys x 64
// channels) reach LDS row-major by bounds-checked direct copies (rows past L_b as
// zeros) into two buffers, one tile ahead, 16-byte chunks swizzled as in kv_off;
// the MFMA's V^T operand comes from transposed reads (ds_read_b64_tr_b16: within
// each 16-lane group, lane 4 e + q addresses row e, columns 4 q .. 4 q + 3 of a
// 4 x 16 block and lane t receives column t of the four rows), issued as inline
// assembly with their own wait so that the compiler does not first wait for the
// next tile's copies.
constexpr int kAvBuf = kTile * kHeadDim;  // elements of one V buffer
constexpr int kAvPRow = 10;               // 16-byte chunks staged per probability row
constexpr int kAvPBlocks = 12;            // 1 KB copy blocks per tile: 64 rows x 10 chunks, rounded to 3 per wave
constexpr int kAvPBuf = kAvPBlocks * 512; // elements of one probability buffer

__global__ __launch_bounds__(256) void k_attn_v_bf16(PlanArgs pa, const uint16_t* __restrict__ P,
                                                      int64_t score_cap, const uint16_t* __restrict__ v,
                                                      int ldv, uint16_t* __restrict__ O, int ldo, int causal,
                                                      int G) {
    if (!plan_ok(pa, score_cap)) return;
    __shared__ __attribute__((aligned(16))) uint16_t vb[2 * kAvBuf];  // [buffer][key][64 channels]
    __shared__ __attribute__((aligned(16))) uint16_t pb[2 * kAvPBuf];  // [buffer][row][10 chunks]
    const int H = pa.heads;
    const int n_items = pa.status[2] / G;
    const int wave = uni(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const int l16 = lane % 16, q4 = lane / 16;
    // transposed-read addresses (buffer 0, keys 0..31): group q4 reads keys 8 q4 + e (+ 4),
    // channels 16 cb + 4 q of its 4 x 16 blocks; keys 32 .. 63 and buffer 1 are immediates
    // (32 rows leave the swizzle's row bits 1-3 unchanged)
    const int tr_e = (lane % 16) / 4, tr_q = lane % 4;
    uint32_t vaddr[4][2];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int hi = 0; hi < 2; ++hi)
            vaddr[cb][hi] = (uint32_t)(uintptr_t)(vb + kv_off(8 * q4 + tr_e + 4 * hi, 16 * cb + 4 * tr_q));
    for (int base_it = 0; base_it < n_items; base_it += gridDim.x) {
        const int g = base_it + op_item(blockIdx.x, gridDim.x);
        if (g >= n_items) break;  // uniform over the workgroup
        const int kk = uni(item_sequence(pa.av_item_off, pa.batch, G, g));
        const int b = uni(pa.order[kk]);
        const int local = g - uni(pa.av_item_off[kk]) / G;
        const int nb = (uni(pa.lengths[b]) + kTile - 1) / kTile;  // query blocks of the sequence
        const int hg = local / nb, ti = local - hg * nb, h0 = hg * G;  // heads h0 .. h0 + G - 1
        const int L = uni(pa.lengths[b]);
        const int t0 = uni(pa.tok_off[b]);
        const int64_t base = uni64(pa.att_off[b]);
        const int rows = min(kTile, L - ti * kTile);
        const int i = ti * kTile + wave * 16 + l16;  // this lane's query row (valid if < ti*64 + rows)
        const bool row_ok = wave * 16 + l16 < rows;
        // the item reads rows ti*64 .. ti*64 + rows - 1 of heads h0 .. h0 + G - 1: from element e_lo on
        const int64_t e_lo = base + (int64_t)ti * kTile * H * L;
        const int64_t e_al = e_lo & ~(int64_t)7;
        // Range: through the item's last element (a chunk read past it is masked), in
        // whole dwords (the range check drops a dword that is only partly inside; a
        // dword never straddles a page), and never past the caller's score_cap.
        const int64_t e_end = min(score_cap, base + (int64_t)(ti * kTile + rows) * H * L);
        const int64_t nbytes = min<int64_t>(((e_end - e_al) * 2 + 3) & ~(int64_t)3, (int64_t)0x7ffffffc);
        const __amdgpu_buffer_rsrc_t rp =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(P + e_al), 0, (uint32_t)nbytes, 0x00020000);
        const int jend = causal ? min(L, (ti + 1) * kTile) : L;  // masked: keys up to the diagonal tile
        const int kmax = causal ? min(L - 1, i) : L - 1;          // last key this row uses
        // Tiles (head h0 + f / nt, keys 64 (f % nt) ..) in one stream: tile f + 1's V
        // copies and probability chunks are issued while tile f is computed.
        const int nt = (jend + kTile - 1) / kTile;
        const int F = G * nt;
        // V tile f into buffer f & 1: wave w copies rows 16 w .. 16 w + 15 (two 1 KB blocks)
        auto copy_v = [&](int f, auto buf) {
            const int h = h0 + f / nt, j0 = (f % nt) * kTile;
            const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<uint16_t*>(v + (int64_t)(t0 + j0) * ldv + h * kHeadDim), 0,
                (uint32_t)min(kTile, L - j0) * ldv * 2u, 0x00020000);
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int blk = 2 * wave + u, row = blk * 8 + lane / 8;
                const int chunk = (lane % 8) ^ kv_swz(row);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void_t*)(vb + decltype(buf)::value * kAvBuf + blk * 512),
                                                         16, (row * ldv + chunk * 8) * 2, 0, 0, 0);
            }
        };
        // probability rows of tile f into buffer f & 1: slot x = 64 blk + lane is row x / 10,
        // chunk x % 10 (slots past 640 copy nothing useful), wave w taking blocks w, w + 4, w + 8
        auto copy_p = [&](int f, auto buf) {
            const int h = h0 + f / nt, j0 = (f % nt) * kTile;
#pragma unroll
            for (int u = 0; u < kAvPBlocks / 4; ++u) {
                const int blk = wave + 4 * u, x = blk * 64 + lane;
                const int r = min(x / kAvPRow, kTile - 1), c = x - (x / kAvPRow) * kAvPRow;
                const int64_t e = (e_lo - e_al) + ((int64_t)r * H + h) * L + j0;  // the row's first key
                const int off = x < kTile * kAvPRow ? (int)((e & ~(int64_t)7) + 8 * c) * 2 : 0x7ffffff0;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rp, (lds_void_t*)(pb + decltype(buf)::value * kAvPBuf + blk * 512),
                                                         16, off, 0, 0, 0);
            }
        };
        // the element shift of every row piece: row starts differ by multiples of L only
        const int64_t row_e0 = (int64_t)(wave * 16 + l16) * H * L;
        floatx4 acc[4];
        auto step = [&](int f, auto buf) {
            constexpr int BUF = decltype(buf)::value;
            const int h = h0 + f / nt, j0 = (f % nt) * kTile;
            if (f % nt == 0) {
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
            }
            // this wave's copies of tile f, then every wave's; buffers f + 1 were last read in step f - 1
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
            // This tile's probability pieces are read before tile f + 1's copies go
            // out: the compiler makes an LDS read wait for every LDS copy in flight,
            // which would hold the tile for the next one's copies.
            const int sh = (int)((e_lo - e_al + row_e0 + (int64_t)h * L + j0) & 7);
            const uint32_t rb = (sh & 1) * 2;
            const uint32_t* const prow =
                reinterpret_cast<const uint32_t*>(pb + BUF * kAvPBuf) + (wave * 16 + l16) * (kAvPRow * 4) + (sh >> 1);
            bf16x8 pk[2];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const int jk = j0 + 32 * ks + 8 * q4;
                const uint32_t* d = prow + 16 * ks + 4 * q4;
                const uint32_t d0 = d[0], d1 = d[1], d2 = d[2], d3 = d[3], d4 = d[4];
                u32x4 pw = {__builtin_amdgcn_alignbyte(d1, d0, rb), __builtin_amdgcn_alignbyte(d2, d1, rb),
                            __builtin_amdgcn_alignbyte(d3, d2, rb), __builtin_amdgcn_alignbyte(d4, d3, rb)};
                // keys past the row's last used key (and rows past the block) count as zero
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int j = jk + 2 * e;
                    const uint32_t keep = (row_ok && j <= kmax ? 0x0000ffffu : 0u) |
                                          (row_ok && j + 1 <= kmax ? 0xffff0000u : 0u);
                    pw[e] &= keep;
                }
                pk[ks] = as_bf16x8(pw);
            }
            if (f + 1 < F) {
                copy_v(f + 1, std::integral_constant<int, 1 - BUF>{});
                copy_p(f + 1, std::integral_constant<int, 1 - BUF>{});
            }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x8 pb = pk[ks];
                u32x2 t[4][2];
                asm volatile(
                    "ds_read_b64_tr_b16 %0, %8 offset:%16\n\t"
                    "ds_read_b64_tr_b16 %1, %9 offset:%16\n\t"
                    "ds_read_b64_tr_b16 %2, %10 offset:%16\n\t"
                    "ds_read_b64_tr_b16 %3, %11 offset:%16\n\t"
                    "ds_read_b64_tr_b16 %4, %12 offset:%16\n\t"
                    "ds_read_b64_tr_b16 %5, %13 offset:%16\n\t"
                    "ds_read_b64_tr_b16 %6, %14 offset:%16\n\t"
                    "ds_read_b64_tr_b16 %7, %15 offset:%16\n\t"
                    "s_waitcnt lgkmcnt(0)"
                    : "=&v"(t[0][0]), "=&v"(t[0][1]), "=&v"(t[1][0]), "=&v"(t[1][1]), "=&v"(t[2][0]), "=&v"(t[2][1]),
                      "=&v"(t[3][0]), "=&v"(t[3][1])
                    : "v"(vaddr[0][0]), "v"(vaddr[0][1]), "v"(vaddr[1][0]), "v"(vaddr[1][1]), "v"(vaddr[2][0]),
                      "v"(vaddr[2][1]), "v"(vaddr[3][0]), "v"(vaddr[3][1]),
                      "i"((BUF * kAvBuf + 32 * ks * kHeadDim) * 2)
                    : "memory");
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) {
                    const bf16x8 va = as_bf16x8(u32x4{t[cb][0][0], t[cb][0][1], t[cb][1][0], t[cb][1][1]});
                    acc[cb] = mfma16x16x32(va, pb, acc[cb]);  // C[c][i] = sum_j V[j][c] P[i][j]
                }
            }
            if (f % nt == nt - 1 && row_ok) {
                // C[c][i]: the lane holds channels cb*16 + 4 q4 .. + 3 of query row i
                uint16_t* orow = O + (int64_t)(t0 + i) * ldo + h * kHeadDim;
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) {
                    u32x2 w2 = {pack_bf16x2(acc[cb][0], acc[cb][1]), pack_bf16x2(acc[cb][2], acc[cb][3])};
                    *reinterpret_cast<u32x2*>(orow + cb * 16 + 4 * q4) = w2;
                }
            }
        };
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");  // the previous item's reads are done
        copy_v(0, std::integral_constant<int, 0>{});
        copy_p(0, std::integral_constant<int, 0>{});
        for (int f = 0; f < F; f += 2) {
            step(f, std::integral_constant<int, 0>{});
            if (f + 1 < F) step(f + 1, std::integral_constant<int, 1>{});
        }
    }
}

// fp32 Attn.V: one 64-query block of one head per item, probabilities and V
// staged in LDS 64 keys at a time; wave w accumulates the 32 x 32 block
// (queries 32 (w / 2) .., channels 32 (w % 2) ..) on v_mfma_f32_32x32x2f32.  V's
// row stride 96 puts the operand read (row kk + l / 32, column l % 32) in 64
// distinct banks.
__global__ __launch_bounds__(256) void k_attn_v_f32(PlanArgs pa, const float* __restrict__ P, int64_t score_cap,
                                                     const float* __restrict__ v, int ldv, float* __restrict__ O,
                                                     int ldo, int causal) {
    if (!plan_ok(pa, score_cap)) return;
    __shared__ float Ps[kTile][kF32Row], Vs[kTile][kHeadDim + 32];
    const int n_items = pa.status[2];
    const int H = pa.heads;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int l32 = lane % 32, h2 = lane / 32;
    const int wq = wave >> 1, wc = wave & 1;
    for (int it = blockIdx.x; it < n_items; it += gridDim.x) {
        const int b = pa.av_items[3 * it], h = pa.av_items[3 * it + 1], ti = pa.av_items[3 * it + 2];
        const int L = pa.lengths[b];
        const int t0 = pa.tok_off[b];
        const int64_t base = pa.att_off[b];
        const int rows = min(kTile, L - ti * kTile);
        floatx16 acc;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.f;
        const int jend = causal ? min(L, (ti + 1) * kTile) : L;
        for (int j0 = 0; j0 < jend; j0 += kTile) {
            const int cols = min(kTile, L - j0);
            // every load unconditional at an index clamped into the block, the masked
            // elements zeroed afterwards: loads under the range tests were each waited
            // for before the next was issued
            float pv[kTile * kTile / 256], vv[kTile * kTile / 256];
#pragma unroll
            for (int u = 0; u < kTile * kTile / 256; ++u) {
                const int e = threadIdx.x + 256 * u, r = e / kTile, c = e % kTile;
                pv[u] = P[base + ((int64_t)(ti * kTile + min(r, rows - 1)) * H + h) * L + j0 + min(c, cols - 1)];
                vv[u] = v[(int64_t)(t0 + j0 + min(r, cols - 1)) * ldv + h * kHeadDim + c];
            }
            __syncthreads();  // the previous block's operand reads are done
#pragma unroll
            for (int u = 0; u < kTile * kTile / 256; ++u) {
                const int e = threadIdx.x + 256 * u, r = e / kTile, c = e % kTile;
                Ps[r][c] = (r < rows && c < cols && (!causal || j0 + c <= ti * kTile + r)) ? pv[u] : 0.f;
                Vs[r][c] = r < cols ? vv[u] : 0.f;
            }
            __syncthreads();
#pragma unroll 8
            for (int kk = 0; kk < kTile; kk += 2)
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(Ps[wq * 32 + l32][kk + h2], Vs[kk + h2][wc * 32 + l32], acc,
                                                           0, 0, 0);
        }
        float* orow = O + (int64_t)(t0 + ti * kTile) * ldo + h * kHeadDim + wc * 32 + l32;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = wq * 32 + 8 * (r / 4) + 4 * h2 + r % 4;
            if (i < rows) orow[(int64_t)i * ldo] = acc[r];
        }
    }
}

// ---------------------------------------------------------------------------
// Fused ragged attention: QK^T, softmax and Attn.V in one pass over the keys; no
// score reaches memory.  One (sequence b, head h, 64-query tile) item of the
// plan's Attn.V list per workgroup of two waves, 32 queries per wave, items
// longest sequence first (the plan's order).
//   keys   stream through two LDS stages of 32 K rows and 32 V rows (16 KB per
//          workgroup, so eight workgroups share a CU: while one waits for its
//          next chunk the others compute, and every SIMD keeps four busy waves
//          whatever the lengths); bounds-checked buffer loads write LDS
//          directly, 16-byte chunks XOR-swizzled by row, rows past L_b as zeros
//   scores S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (lane holds query
//          i = lane % 32 and keys 8*(r/4) + 4*(lane/32) + r%4), kept in fp32
//   softmax online: z = s * scale * log2(e); a per-row reference m, the
//          first chunk's maximum; a later chunk takes e = exp2(z - m) at once
//          and only if a lane's sum of its 16 exponentials passes 2^16 does
//          the wave recompute the chunk, raise m to its maximum and rescale
//          the running sum and output (rare); e rounded to bf16 is the MFMA
//          operand
//   output O^T += V^T E^T.  The lane's eight keys of each 16-key step
//          {4h..4h+3, 8+4h..8+4h+3} (h = lane/32) are its k values (the MFMA
//          pairs the k-th element of A with the k-th element of B), and
//          ds_read_b64_tr_b16 gathers the V operand for exactly those keys
//          from the row-major V rows; O is divided by the row sum at the end.
// Relative to the three separate operators, the fused path skips the bf16
// rounding of the scores and rounds the unnormalised exponentials instead of
// the probabilities (the flash-attention order); both differ from the
// separate path by rounding only.  Items are dealt to the XCDs in runs of
// kStreamRun consecutive list entries (a sequence's tiles of one head share its
// K / V rows in that XCD's L2), the runs round-robin.
// ---------------------------------------------------------------------------

constexpr float kSumCap = 65536.f;  // largest lane sum of a chunk's exponentials kept (2^16)
constexpr int kStreamWaves = 2, kStreamThreads = kStreamWaves * kWave;
constexpr int kStreamBlocks = 4 / kStreamWaves;                 // 1 KB copies of K (and of V) per wave and chunk
constexpr int kStreamChunk = 32;                                // keys per LDS stage
constexpr int kStreamStageElems = 2 * kStreamChunk * kHeadDim;  // K rows, then V rows
constexpr int kStreamRun = 8;
constexpr int kStreamPerCu = 64;  // grid cap in workgroups per CU (they then loop over the list)

__device__ __forceinline__ int stream_item(int bid, int nb) {  // nb: a multiple of 8 * kStreamRun
    const int xcd = bid % 8, j = bid / 8;
    return ((j / kStreamRun) * 8 + xcd) * kStreamRun + j % kStreamRun;
}

__device__ __forceinline__ void attn_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Combine a value with the one held by the lane 32 apart (the other half of
// the same query row): v_permlane32_swap hands each half the other's value.
__device__ __forceinline__ float max_xor32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float sum_xor32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <bool CAUSAL>
__global__ __launch_bounds__(kStreamThreads) __attribute__((amdgpu_waves_per_eu(4)))
void k_attention_bf16(PlanArgs pa, const uint16_t* __restrict__ q, int ldq, const uint16_t* __restrict__ k,
                             int ldk, const uint16_t* __restrict__ v, int ldv, float scale,
                             uint16_t* __restrict__ O, int ldo) {
    if (pa.status[0] != 0) return;
    __shared__ __attribute__((aligned(16))) uint16_t kvs[2 * kStreamStageElems];
    const int n_items = pa.status[2];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const int l32 = lane % 32, h2 = lane / 32;
    const int tr_e = (lane % 16) / 4, tr_q = lane % 4, tr_g = lane / 16;
    // A zero scale would turn the masked keys' -inf into NaN (-inf * 0); any
    // |scale| below 1e-30 already makes every exponential round to 1 (the
    // uniform softmax of a zero scale), so the factor is kept at least that.
    const float zs = fmaxf(fabsf(scale) * 1.4426950408889634f, 1e-30f);
    const uint32_t qsign = scale < 0.f ? 0x80008000u : 0u;
    // a stage holds keys 32c .. 32c + 31 at rows 0..31; 32c leaves the swizzle's
    // row bits 1-3 unchanged, so the offsets are those of chunk 0
    int koff[4], voff[2][2];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) koff[ks] = kv_off(l32, 16 * ks + 8 * h2);
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int hi = 0; hi < 2; ++hi)
            voff[cb][hi] = kv_off(4 * (tr_g >> 1) + tr_e + 8 * hi, 32 * cb + 16 * (tr_g & 1) + 4 * tr_q);
    // LDS byte addresses of the transposed V reads in stage 0, key step 0
    uint32_t vaddr[2][2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int hi = 0; hi < 2; ++hi)
            vaddr[cb][hi] = (uint32_t)(uintptr_t)(kvs + kStreamChunk * kHeadDim + voff[cb][hi]);

    for (int base = 0; base < n_items; base += gridDim.x) {
        const int it = base + stream_item(blockIdx.x, gridDim.x);
        if (it >= n_items) break;
        const int b = pa.av_items[3 * it], h = pa.av_items[3 * it + 1], ti = pa.av_items[3 * it + 2];
        const int L = pa.lengths[b];
        const int t0 = pa.tok_off[b];
        const int qb = 2 * ti + wave;  // this wave's 32-query block
        const bool active = qb * 32 < L;
        const int nc_all = (L + 31) / 32;
        const int nc_wg = CAUSAL ? min(nc_all, 2 * ti + kStreamWaves) : nc_all;  // chunks the workgroup loads
        const int nc_me = CAUSAL ? qb + 1 : nc_all;                    // chunks this wave uses
        const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t*>(k + (int64_t)t0 * ldk + h * kHeadDim), 0, (uint32_t)L * ldk * 2u, 0x00020000);
        const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t*>(v + (int64_t)t0 * ldv + h * kHeadDim), 0, (uint32_t)L * ldv * 2u, 0x00020000);
        // wave w copies rows 16w .. 16w + 15 of the chunk's K and V (two 1 KB blocks
        // of 8 rows each); rows past L arrive as zeros.  Chunk c adds 32c rows to
        // the lane offsets of chunk 0 (32c leaves the swizzle's row bits alone).
        int vko[kStreamBlocks], vvo[kStreamBlocks];
#pragma unroll
        for (int i = 0; i < kStreamBlocks; ++i) {
            const int row = (wave * kStreamBlocks + i) * 8 + lane / 8;
            const int logical = (lane % 8) ^ kv_swz(row);
            vko[i] = row * ldk * 2 + logical * 16;
            vvo[i] = row * ldv * 2 + logical * 16;
        }
        auto issue = [&](int c, auto stg) {
            uint16_t* st = kvs + decltype(stg)::value * kStreamStageElems;
            const int dk = c * kStreamChunk * ldk * 2, dv = c * kStreamChunk * ldv * 2;
#pragma unroll
            for (int i = 0; i < kStreamBlocks; ++i) {
                const int blk = wave * kStreamBlocks + i;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void_t*)(st + blk * 512), 16, vko[i] + dk, 0, 0, 0);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void_t*)(st + kStreamChunk * kHeadDim + blk * 512),
                                                         16, vvo[i] + dv, 0, 0, 0);
            }
        };
        bf16x8 qf[4];
        {
            const int qi = min(qb * 32 + l32, L - 1);
            const uint16_t* qrow = q + (int64_t)(t0 + qi) * ldq + h * kHeadDim + 8 * h2;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                u32x4 raw = active ? ld16(qrow + 16 * ks) : u32x4{0u, 0u, 0u, 0u};
                raw ^= qsign;
                qf[ks] = as_bf16x8(raw);
            }
        }
        float m = -INFINITY, lsum = 0.f;
        floatx16 oacc[2];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int r = 0; r < 16; ++r) oacc[cb][r] = 0.f;
        // chunk c in stage STG (c's parity, a compile-time constant, so every LDS
        // address is a fixed per-lane register plus an immediate offset)
        auto step = [&](int c, auto stg) {
            constexpr int STG = decltype(stg)::value;
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's copies of chunk c
            attn_barrier();  // ... and the other wave's; chunk c + 1's stage was last read in step c - 1
            if (c + 1 < nc_wg) issue(c + 1, std::integral_constant<int, 1 - STG>{});
            if (!active || c >= nc_me) return;
            const uint16_t* kst = kvs + STG * kStreamStageElems;
            floatx16 acc;
            // scores of the chunk (rows past L and, causal, keys past the query as -inf)
            // (LEAN: one K fragment at a time, for the rare recomputation, where the
            // transposed V reads are already held)
            auto scores = [&](auto lean) {
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[r] = 0.f;
                if constexpr (decltype(lean)::value) {
#pragma unroll
                    for (int ks = 0; ks < 4; ++ks)
                        acc = mfma32x32x16(as_bf16x8(*reinterpret_cast<const u32x4*>(kst + koff[ks])), qf[ks], acc);
                } else {
                    bf16x8 kf[4];
#pragma unroll
                    for (int ks = 0; ks < 4; ++ks) kf[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(kst + koff[ks]));
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int ks = 0; ks < 4; ++ks) acc = mfma32x32x16(kf[ks], qf[ks], acc);
                }
                if (32 * (c + 1) > L || (CAUSAL && c == qb)) {
                    const int kmax = CAUSAL && c == qb ? min(L - 1, qb * 32 + l32) : L - 1;
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        if (32 * c + 8 * (r / 4) + 4 * h2 + (r % 4) > kmax) acc[r] = -INFINITY;
                }
            };
            // the row's largest z = s * scale * log2(e) in the chunk (both half-waves)
            auto chunk_max = [&]() {
                float cmax = acc[0];
#pragma unroll
                for (int r = 1; r < 16; ++r) cmax = fmaxf(cmax, acc[r]);
                return max_xor32(cmax) * zs;
            };
            // exponentials exp2(z - m) in place of the scores; the lane's sum of them
            auto exps = [&]() {
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[r] = __builtin_amdgcn_exp2f(fmaf(acc[r], zs, -m));
                float p[8];
#pragma unroll
                for (int r = 0; r < 8; ++r) p[r] = acc[2 * r] + acc[2 * r + 1];
#pragma unroll
                for (int r = 0; r < 4; ++r) p[r] += p[r + 4];
                return (p[0] + p[2]) + (p[1] + p[3]);
            };
            scores(std::false_type{});
            // the V^T operand of both 16-key halves by transposed reads, issued now
            // and waited for just before the P.V products, so their latency passes
            // under the exponentials (inline assembly: the builtin makes the
            // compiler wait first for every LDS copy in flight, chunk c + 1's included)
            u32x2 tr[2][2][2];
            asm volatile(
                "ds_read_b64_tr_b16 %0, %8 offset:%12\n\t"
                "ds_read_b64_tr_b16 %1, %9 offset:%12\n\t"
                "ds_read_b64_tr_b16 %2, %10 offset:%12\n\t"
                "ds_read_b64_tr_b16 %3, %11 offset:%12\n\t"
                "ds_read_b64_tr_b16 %4, %8 offset:%13\n\t"
                "ds_read_b64_tr_b16 %5, %9 offset:%13\n\t"
                "ds_read_b64_tr_b16 %6, %10 offset:%13\n\t"
                "ds_read_b64_tr_b16 %7, %11 offset:%13"
                : "=&v"(tr[0][0][0]), "=&v"(tr[0][0][1]), "=&v"(tr[0][1][0]), "=&v"(tr[0][1][1]),
                  "=&v"(tr[1][0][0]), "=&v"(tr[1][0][1]), "=&v"(tr[1][1][0]), "=&v"(tr[1][1][1])
                : "v"(vaddr[0][0]), "v"(vaddr[0][1]), "v"(vaddr[1][0]), "v"(vaddr[1][1]),
                  "i"(STG * kStreamStageElems * 2), "i"((STG * kStreamStageElems + 16 * kHeadDim) * 2)
                : "memory");
            if (c == 0) m = chunk_max();  // the reference starts at the first chunk's maximum
            float ps = exps();
            // a lane sum above kSumCap (or NaN) means a score well above m: the wave
            // recomputes its scores, raises m to the chunk maximum and rescales what
            // it has summed so far (rare after the first chunks)
            if (c > 0 && __ballot(!(ps <= kSumCap)) != 0) {
                scores(std::true_type{});
                const float mn = fmaxf(m, chunk_max());
                const float alpha = __builtin_amdgcn_exp2f(m - mn);
                lsum *= alpha;
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) oacc[cb][r] *= alpha;
                m = mn;
                ps = exps();
            }
            lsum += ps;
            // the transposed reads have landed (the registers pass through the wait,
            // so no use of them moves above it)
            asm volatile("s_waitcnt lgkmcnt(0)"
                         : "+v"(tr[0][0][0]), "+v"(tr[0][0][1]), "+v"(tr[0][1][0]), "+v"(tr[0][1][1]),
                           "+v"(tr[1][0][0]), "+v"(tr[1][0][1]), "+v"(tr[1][1][0]), "+v"(tr[1][1][1])
                         :
                         : "memory");
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                u32x4 pw;
#pragma unroll
                for (int e = 0; e < 4; ++e) pw[e] = pack_bf16x2(acc[8 * t + 2 * e], acc[8 * t + 2 * e + 1]);
                const bf16x8 pb = as_bf16x8(pw);
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
                    oacc[cb] = mfma32x32x16(
                        as_bf16x8(u32x4{tr[t][cb][0][0], tr[t][cb][0][1], tr[t][cb][1][0], tr[t][cb][1][1]}), pb,
                        oacc[cb]);
            }
        };
        attn_barrier();  // both stages are free: the previous item's reads are done
        issue(0, std::integral_constant<int, 0>{});
        for (int c = 0; c < nc_wg; c += 2) {
            step(c, std::integral_constant<int, 0>{});
            if (c + 1 < nc_wg) step(c + 1, std::integral_constant<int, 1>{});
        }
        if (active) {
            const float inv = 1.0f / sum_xor32(lsum);
            const int i = qb * 32 + l32;
            if (i < L) {
                uint16_t* orow = O + (int64_t)(t0 + i) * ldo + h * kHeadDim;
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const u32x2 w2 = {pack_bf16x2(oacc[cb][4 * g] * inv, oacc[cb][4 * g + 1] * inv),
                                          pack_bf16x2(oacc[cb][4 * g + 2] * inv, oacc[cb][4 * g + 3] * inv)};
                        *reinterpret_cast<u32x2*>(orow + 32 * cb + 8 * g + 4 * h2) = w2;
                    }
            }
        }
    }
}

int persistent_grid(int64_t cap, int per_cu) {
    const int64_t g = (int64_t)device_cu_count() * per_cu;
    return static_cast<int>(cap < g ? (cap > 0 ? cap : 1) : g);
}

// Grid of the bf16 operators: at most four workgroups per CU, no more than the
// items a plan of this capacity can hold (av_cap / H), and a multiple of
// 8 * kOpRun so the XCD dealing is a permutation.
int op_grid(const PlanView& p, int G) {
    constexpr int64_t kUnit = 8 * kOpRun;
    const int64_t items = std::max<int64_t>((p.av_cap + G - 1) / G, 1);
    const int64_t g = std::min<int64_t>(items, (int64_t)device_cu_count() * 4);
    return static_cast<int>((g + kUnit - 1) / kUnit * kUnit);
}

// Heads per item: the largest divisor of H that still leaves a plan of this
// capacity (av_cap / G items at most) eight items per CU.  Fewer, larger items
// balance worse over the grid: at the batch-128, 16-head shape G = 8 (about five
// items per CU) took Attn.V 0.171 ms against 0.149 at G = 4; QK^T is within 2%
// from G = 2 to 8 and 15% slower at G = 1.
int op_heads(const PlanView& p) {
    const int64_t want = (int64_t)device_cu_count() * 8;
    for (int G = p.heads; G > 1; --G)
        if (p.heads % G == 0 && p.av_cap / G >= want) return G;
    return 1;
}

}  // namespace

hipError_t launch_qkt(const PlanView& p, int dtype, const void* q, int ldq, const void* k, int ldk, float scale,
                      void* scores, int64_t score_cap, bool causal, hipStream_t s) {
    const PlanArgs pa = plan_args(p);
    const int G = op_heads(p);
    const int grid = dtype == 1 ? op_grid(p, G) : persistent_grid(p.qkt_cap, 8);
    if (dtype == 1)
        hipLaunchKernelGGL(k_qkt_bf16, dim3(grid), dim3(kQkThreads), 0, s, pa, static_cast<const uint16_t*>(q), ldq,
                           static_cast<const uint16_t*>(k), ldk, scale, static_cast<uint16_t*>(scores), score_cap,
                           int(causal), G);
    else
        hipLaunchKernelGGL(k_qkt_f32, dim3(grid), dim3(256), 0, s, pa, static_cast<const float*>(q), ldq,
                           static_cast<const float*>(k), ldk, scale, static_cast<float*>(scores), score_cap,
                           int(causal));
    return hipGetLastError();
}

hipError_t launch_softmax(const PlanView& p, int dtype, const void* scores, void* probs, int64_t score_cap,
                          bool causal, hipStream_t s) {
    if (p.total_tokens == 0) return hipSuccess;
    const PlanArgs pa = plan_args(p);
    const int grid = (p.total_tokens + 3) / 4;
    if (dtype == 1)
        hipLaunchKernelGGL(k_softmax<true>, dim3(grid), dim3(256), 0, s, pa, static_cast<const uint16_t*>(scores),
                           static_cast<uint16_t*>(probs), score_cap, p.total_tokens, int(causal));
    else
        hipLaunchKernelGGL(k_softmax<false>, dim3(grid), dim3(256), 0, s, pa, static_cast<const float*>(scores),
                           static_cast<float*>(probs), score_cap, p.total_tokens, int(causal));
    return hipGetLastError();
}

hipError_t launch_attn_v(const PlanView& p, int dtype, const void* probs, int64_t score_cap, const void* v, int ldv,
                         void* out, int ldo, bool causal, hipStream_t s) {
    const PlanArgs pa = plan_args(p);
    const int G = op_heads(p);
    const int grid = dtype == 1 ? op_grid(p, G) : persistent_grid(p.av_cap, 8);
    if (dtype == 1)
        hipLaunchKernelGGL(k_attn_v_bf16, dim3(grid), dim3(256), 0, s, pa, static_cast<const uint16_t*>(probs),
                           score_cap, static_cast<const uint16_t*>(v), ldv, static_cast<uint16_t*>(out), ldo, int(causal),
                           G);
    else
        hipLaunchKernelGGL(k_attn_v_f32, dim3(grid), dim3(256), 0, s, pa, static_cast<const float*>(probs),
                           score_cap, static_cast<const float*>(v), ldv, static_cast<float*>(out), ldo, int(causal));
    return hipGetLastError();
}

namespace {
template <bool CAUSAL>
hipError_t launch_fused_variant(const PlanView& p, const void* q, int ldq, const void* k, int ldk, const void* v,
                                int ldv, float scale, void* out, int ldo, hipStream_t s) {
    // one workgroup per item, at most kStreamPerCu per CU (the workgroups then
    // loop over the list); a multiple of 8 * kStreamRun so the XCD dealing is a
    // permutation
    constexpr int64_t kUnit = 8 * kStreamRun;
    const int64_t cap = std::max<int64_t>(p.av_cap, 1);
    const int64_t limit = (int64_t)device_cu_count() * kStreamPerCu;
    const int64_t g = (std::min(cap, limit) + kUnit - 1) / kUnit * kUnit;
    hipLaunchKernelGGL(k_attention_bf16<CAUSAL>, dim3((unsigned)g), dim3(kStreamThreads), 0, s, plan_args(p),
                       static_cast<const uint16_t*>(q), ldq, static_cast<const uint16_t*>(k), ldk,
                       static_cast<const uint16_t*>(v), ldv, scale, static_cast<uint16_t*>(out), ldo);
    return hipGetLastError();
}
}  // namespace

hipError_t launch_fused_attention(const PlanView& p, int dtype, const void* q, int ldq, const void* k, int ldk,
                                  const void* v, int ldv, float scale, void* out, int ldo, bool causal,
                                  hipStream_t s) {
    if (dtype != 1) return hipErrorInvalidValue;
    return causal ? launch_fused_variant<true>(p, q, ldq, k, ldk, v, ldv, scale, out, ldo, s)
                  : launch_fused_variant<false>(p, q, ldq, k, ldk, v, ldv, scale, out, ldo, s);
}

}  // namespace rag
