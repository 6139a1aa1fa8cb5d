// Packed-token linear operator y = act(x w^T + bias) + residual over the T real
// tokens (the layer's Proj1 / Proj2 / FF1 / FF2; Section 7.2 runs them as one
// fused loop over the batch and length loops, so they are plain GEMMs with
// M = T and no padding).
//
// bf16: a 128 x 256 output tile per workgroup of 4 waves, each wave a 128
// (tokens) x 64 (features) sub-tile of v_mfma_f32_32x32x16_bf16 accumulators
// (the full-rate bf16 MFMA on gfx950).  A tile needs at most 80 KB of LDS, so two
// workgroups share a CU and one's prologue / epilogue overlaps the other's K
// loop.  (256-token tiles of 8 waves, measured against this design, were no
// faster on 8192^3 and 8% slower on the QKV projection.)
//  - Both operands are K-contiguous in memory (x is [T, K], w is [N, K]), the
//    operand layout the MFMA wants, so tiles go to LDS untransposed.
//  - Global -> LDS copies are bounds-checked buffer loads that write LDS
//    directly (no register staging): each wave instruction fills one 1 KB block
//    of consecutive rows, lane l landing at byte 16*l of the block.  Rows past
//    T (or N) lie outside the buffer range and arrive as zeros, so the ragged
//    last token tile needs no clamping.
//  - The 16-byte chunk index inside an LDS row is XOR-swizzled with the row, so
//    the fragment reads of 16 consecutive rows hit 16 distinct bank groups; the
//    copies pick their source chunk so that the swizzled slot is filled.
//  - Software pipeline over K steps of 32: the x fragments of step k+1 are read
//    into a second register set right after the step's barrier and its w
//    fragments are streamed in while the MFMAs of step k run; the barrier waits
//    only for the copies the next step needs, and the copies of later steps are
//    issued one MFMA group apart.  Two LDS layouts:
//      paired-w (GEMM, vgemm): x in two stages of 32 k, w in two stages of 64 k
//        (one 128-byte row per feature), 80 KB.  Every w copy reads whole
//        128-byte lines, which halves the L2 requests of the dominant operand
//        (64-byte K-step rows cost one request per half line; measured 11-15%
//        faster on the layer's GEMMs).
//      ring (trmm): three stages of 32 k, copies issued three steps ahead, 72 KB.
//  - The MFMA computes the transposed tile C[n][m] = sum_k w[n][k] x[m][k], so each
//    lane ends with four consecutive output features of one token.  Results pass
//    through LDS so that whole 512-byte rows move to memory: without a residual,
//    bias and activation are applied to the accumulators and the whole tile is
//    staged as bf16 rows at once (one barrier pair); with a residual, fp32
//    results are staged in 32-token slices and bias / activation / residual are
//    applied in the row phase, so the sum is rounded once.
//
// The same tile body (gemm_tile_bf16) also serves the variable-sized batched
// GEMM (one workgroup per entry of a plan's tile list, Section 7.1) and the
// triangular product C = tril(L) B (a [K][N] right operand read through
// transposing LDS loads, and a triangular left operand whose last K steps are
// masked), both further down.
#include <type_traits>

#include "device_common.h"
#include "launch.h"
#include "plan_device.h"

namespace rag {
namespace {

typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int BN = 256, BK = 32;
constexpr int WN = 64, FN = WN / 32;        // wave tile: all BM tokens x WN features
constexpr int KSTEPS = BK / 16;             // MFMA k-steps per K step
constexpr int kChunks = BK / 8;             // 16-byte chunks per LDS row
constexpr int kRowsPerBlock = 64 / kChunks; // rows filled by one 1 KB wave copy
constexpr int kEpiRows = 32;                // tokens per epilogue slice
constexpr int kGroupM = 8;                  // token tiles per group in the tile order

// Tile configuration: BM tokens x BN features per workgroup of 4 waves, wave w
// holding all BM tokens x features [64 w, 64 w + 64); BM = 128, or 64 for the
// halves of a last round's tiles.  Two workgroups share a CU.
template <int BM>
struct Cfg {
    static_assert(BM == 64 || BM == 128, "tile height");
    static constexpr int kWaves = 4, kThreads = kWaves * kWave;
    static constexpr int kFM = BM / 32;                 // 32-token fragments per wave
    static constexpr int kStages = 3;
    static constexpr int kStageElems = (BM + BN) * BK;  // one LDS stage: x tile then w tile
    static constexpr int kXBlocks = BM / kRowsPerBlock / kWaves;  // 1 KB copies of x per wave and step
    static constexpr int kWBlocks = BN / kRowsPerBlock / kWaves;  // 1 KB copies of w per wave and step
    static constexpr int kCopies = kXBlocks + kWBlocks;
    static constexpr int kStageBytes = kStages * kStageElems * 2, kEpilogueBytes = kEpiRows * BN * 4;
    static constexpr int kLdsBytes = kStageBytes > kEpilogueBytes ? kStageBytes : kEpilogueBytes;
    static_assert(kLdsBytes <= 160 * 1024, "LDS budget");
    static_assert(kXBlocks >= 1 && kWBlocks >= 1, "copy split");
    // Paired-w pipeline (w stored [N][K]): two x stages of BK and two w stages of
    // 2 BK, at most 80 KB, still two workgroups per CU.
    static constexpr int kPairXElems = BM * BK, kPairWElems = BN * 2 * BK;
    static constexpr int kPairWBlocks = BN / 8 / kWaves;  // 1 KB copies of w per wave and w stage
    static constexpr int kPairBytes = (2 * kPairXElems + 2 * kPairWElems) * 2;
    static constexpr int kPairLdsBytes = kPairBytes > kEpilogueBytes ? kPairBytes : kEpilogueBytes;
    static_assert(2 * kPairLdsBytes <= 160 * 1024, "two paired-w workgroups per CU");
};

// The pipeline a tile runs: paired-w with w stored [N][K], the kStages ring
// otherwise (the [K][N] and triangular operands of trmm).
constexpr bool pair_w(bool w_kn, bool tri) { return !w_kn && !tri; }
template <int BM, bool W_KN, bool TRI = false>
constexpr int tile_lds_bytes() { return pair_w(W_KN, TRI) ? Cfg<BM>::kPairLdsBytes : Cfg<BM>::kLdsBytes; }

// The 16-byte chunk index inside an LDS row is XOR-swizzled with bits 2-3 of the
// row: a ds_read_b128 serves 16 lanes per cycle, here 16 consecutive rows (four
// 64-byte rows per 256-byte bank line), which then fall on 16 distinct 16-byte
// bank groups.
__device__ __forceinline__ int swz(int row) { return (row >> 2) & (kChunks - 1); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}

// Per-lane byte offset for copying a block of kRowsPerBlock rows starting at
// row0: lane l fills LDS slot l (row row0 + l / kChunks, physical chunk
// l % kChunks) and so reads the logical chunk that the swizzle maps there.
__device__ __forceinline__ int copy_voffset(int lane, int row0, int ld_bytes) {
    const int row = row0 + lane / kChunks;
    return row * ld_bytes + ((lane % kChunks) ^ swz(row)) * 16;
}

// One wave fills the 1 KB LDS block `dst`; k0b (the K offset in bytes) is
// wave-uniform and travels in the scalar offset.
__device__ __forceinline__ void copy_block(__amdgpu_buffer_rsrc_t rsrc, uint16_t* dst, int voff, int k0b) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)dst, 16, voff, k0b, 0, 0);
}

// Workgroup barrier that waits for LDS traffic but not for the copies still in
// flight (a __syncthreads() fence would drain them all): the caller has already
// waited for the copies it needs.
__device__ __forceinline__ void barrier_lds() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ bf16x8 lds_frag(const uint16_t* tile, int row, int chunk) {
    return as_bf16x8(*reinterpret_cast<const u32x4*>(tile + row * BK + ((chunk ^ swz(row)) * 8)));
}

// w operand stored [K][N] (N contiguous; the dense right factor of trmm): an LDS
// stage holds BK rows of BN columns, 512-byte rows of kKnChunks 16-byte chunks
// whose index is XOR-swizzled by (row & 3) << 2.  The transposed fragment reads
// below take rows r..r+3 (64 bytes each per half-wave), which the swizzle puts
// on four distinct 64-byte bank segments.
constexpr int kKnChunks = BN / 8;
constexpr int kKnRowsPerBlock = 64 / kKnChunks;  // rows one 1 KB wave copy fills
__device__ __forceinline__ int swz_kn(int row) { return (row & 3) << 2; }

// Paired-w stages: BN rows of 2 BK (128 bytes, eight 16-byte chunks) whose chunk
// index is XOR-swizzled with bits 1-3 of the row, so the fragment reads of 16
// consecutive rows (two rows per 256-byte bank line) hit 16 distinct bank groups.
// A 1 KB wave copy fills 8 whole rows, so every copy request is a full 128-byte
// line: half as many L2 requests as 64-byte K-step rows.
__device__ __forceinline__ int swz2(int row) { return (row >> 1) & 7; }

template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

typedef __attribute__((ext_vector_type(4))) short short4_t;
typedef __attribute__((address_space(3))) short4_t lds_short4_t;

// ds_read_b64_tr_b16: within each 16-lane group, lane 4e + q supplies the
// address of row e, columns 4q..4q+3 of a 4 x 16 block; lane t of the group
// receives column t of rows 0..3.  Two such reads (rows +0..3 and +4..7) give a
// lane eight consecutive k of one column: the MFMA operand layout.
__device__ __forceinline__ bf16x8 lds_frag_tr(const uint16_t* lo_addr, const uint16_t* hi_addr) {
    const u32x2 lo = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4_t*)lo_addr));
    const u32x2 hi = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4_t*)hi_addr));
    return as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]});
}

// Output tile of a linear workgroup id.  Workgroups are dealt to the 8 XCDs
// round-robin, so the id is first remapped to give each XCD a contiguous range.
// That range is walked in groups of kGroupM token tiles, token tile fastest, so
// the tiles an XCD runs at once share both x rows and w rows in its L2 (groups of
// 2 to 16 measured alike on the layer's GEMMs except FF1, slower below 8).
__device__ __forceinline__ void group_walk(int t, int tiles_m, int tiles_n, int& tm, int& tn) {
    const int gsz = kGroupM * tiles_n, first = (t / gsz) * kGroupM;
    const int gm = min(tiles_m - first, kGroupM);
    tm = first + (t % gsz) % gm;
    tn = (t % gsz) / gm;
}

__device__ __forceinline__ void tile_coords(int bid, int nblocks, int tiles_m, int tiles_n, int& tm, int& tn) {
    const int per = nblocks / 8, rem = nblocks % 8;
    const int xcd = bid % 8, idx = bid / 8;
    const int t = xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
    group_walk(t, tiles_m, tiles_n, tm, tn);
}

// Wait until at most `n` copy instructions of this wave are outstanding (the
// copies complete in issue order).
template <int C>
__device__ __forceinline__ void wait_copies(int n) {
    if (n >= 3 * C) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * C) : "memory");
    else if (n >= 2 * C) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * C) : "memory");
    else if (n >= C) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(C) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// One BM x BN output tile at (m0, n0) of y = act(x w^T + bias) + residual, w being
// [N, K] with K contiguous; smem holds tile_lds_bytes<BM, W_KN, TRI>().  Called by the workgroup
// as a whole (it synchronises on LDS).  K (a multiple of 64) is the extent of the
// reduction the tile runs.
//   W_KN  w is instead [K rows][N] with leading dimension ldw and kvalid valid
//         rows (rows past it read as zeros): y = x w.
//   GROUPS = 2  the workgroup has eight waves in two groups of four; group g
//         runs the K loop over k in [g K / 2, (g + 1) K / 2) in LDS of its own
//         (smem holds twice tile_lds_bytes), and the epilogue adds the two
//         groups' fp32 tiles (group 0's first) before bias, activation and
//         residual: twice the waves on a tile, for launches with fewer tiles
//         than CUs.  K / 2 is then a multiple of 64.
//   TRI   x is lower triangular: x[i][k] counts only for k <= i.  The K steps
//         wholly below the tile's first row run unchecked; the others zero the
//         fragment entries with k > i after reading them (operation splitting of
//         the reduction loop's last iterations, Section 4).
template <int BM, int ACT, bool HAS_BIAS, bool HAS_RES, bool W_KN = false, bool TRI = false, int GROUPS = 1>
__device__ __forceinline__ void gemm_tile_bf16(const uint16_t* __restrict__ x, int ldx, const uint16_t* __restrict__ w,
                                               const uint16_t* __restrict__ bias, const uint16_t* residual, int ldr,
                                               uint16_t* y, int ldy, int T, int K, int N, int m0, int n0,
                                               uint16_t* smem, int ldw = 0, int kvalid = 0) {
    using C = Cfg<BM>;
    static_assert(GROUPS == 1 || (GROUPS == 2 && !W_KN && !TRI), "K halves: the plain GEMM only");
    constexpr int kStages = C::kStages, kStageElems = C::kStageElems, kCopies = C::kCopies;
    constexpr bool kPW = pair_w(W_KN, TRI);
    constexpr int FM = C::kFM;
    // wave-uniform by construction; made explicit so that LDS copy addresses stay scalar
    const int wave_all = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const int grp = wave_all / C::kWaves;  // the K half (GROUPS = 2)
    const int wave = wave_all % C::kWaves;
    const int wn = wave;  // the wave's 64 output features
    const int l32 = lane % 32, h2 = lane / 32;
    uint16_t* const smem_all = smem;
    if constexpr (GROUPS > 1) smem += grp * (tile_lds_bytes<BM, W_KN, TRI>() / 2);
    const int kofs = grp * (K / GROUPS);  // the group's first k

    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc(x + (int64_t)m0 * ldx + kofs, (uint32_t)min(T - m0, BM) * ldx * 2u);
    __amdgpu_buffer_rsrc_t rw;
    if constexpr (W_KN)  // through the last valid column of the last valid row
        rw = make_rsrc(w + n0, kvalid > 0 ? (uint32_t)(((int64_t)(kvalid - 1) * ldw + min(N - n0, BN)) * 2) : 0u);
    else
        rw = make_rsrc(w + (int64_t)n0 * K + kofs, (uint32_t)min(N - n0, BN) * K * 2u);
    int vx[C::kXBlocks], vw[C::kWBlocks];
#pragma unroll
    for (int i = 0; i < C::kXBlocks; ++i) vx[i] = copy_voffset(lane, (wave * C::kXBlocks + i) * kRowsPerBlock, ldx * 2);
#pragma unroll
    for (int i = 0; i < C::kWBlocks; ++i) {
        if constexpr (W_KN) {  // lane l fills slot l of rows 2 blk, 2 blk + 1 (physical chunk l % 32)
            const int row = (wave * C::kWBlocks + i) * kKnRowsPerBlock + lane / kKnChunks;
            vw[i] = row * ldw * 2 + ((lane % kKnChunks) ^ swz_kn(row)) * 16;
        } else {
            vw[i] = copy_voffset(lane, (wave * C::kWBlocks + i) * kRowsPerBlock, K * 2);
        }
    }
    // copy c of this wave for `step`: x blocks first, then w blocks
    auto issue_one = [&](int step, int c) {
        uint16_t* xs = smem + (step % kStages) * kStageElems;
        uint16_t* ws = xs + BM * BK;
        const int k0b = step * BK * 2;
        if (c < C::kXBlocks) {
            copy_block(rx, xs + (wave * C::kXBlocks + c) * 512, vx[c], k0b);
        } else {
            const int i = c - C::kXBlocks;
            if constexpr (W_KN)  // the step moves down the rows: keep it in the range-checked offset
                copy_block(rw, ws + (wave * C::kWBlocks + i) * 512, vw[i] + step * BK * ldw * 2, 0);
            else
                copy_block(rw, ws + (wave * C::kWBlocks + i) * 512, vw[i], k0b);
        }
    };
    auto issue = [&](int step) {
#pragma unroll
        for (int c = 0; c < kCopies; ++c) issue_one(step, c);
    };
    // transposed-read addresses of the [K][N] layout: rows 8 h2 + e (+4), columns
    // wn*WN + i*32 + 16 (g & 1) + 4q, g = lane / 16 (so the lane's column is l32)
    int tr_row = 0, tr_col[FN];
    if constexpr (W_KN) {
        const int e = (lane % 16) / 4, q = lane % 4, g = lane / 16;
        tr_row = (8 * h2 + e) * BN;
#pragma unroll
        for (int i = 0; i < FN; ++i) {
            const int col = wn * WN + i * 32 + 16 * (g & 1) + 4 * q;
            tr_col[i] = (((col >> 3) ^ swz_kn(e)) << 3) + (col & 7);
        }
    }

    floatx16 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // Fragments of one K step: fa[ks][i] (w rows), fb[ks][j] (x rows).
    bf16x8 fa0[KSTEPS][FN], fb0[KSTEPS][FM], fa1[KSTEPS][FN], fb1[KSTEPS][FM];
    auto read_x = [&](bf16x8 (&fb)[KSTEPS][FM], int step) {
        const uint16_t* xb = smem + (step % kStages) * kStageElems;
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
            for (int j = 0; j < FM; ++j) fb[ks][j] = lds_frag(xb, j * 32 + l32, ks * 2 + h2);
    };
    // TRI edge steps: zero the x entries with k > i of a landed stage in LDS, then
    // a barrier (the stage is read only after it).  In registers the masks would
    // push the loop past the register budget.
    auto mask_x = [&](int step) {
        uint32_t* xs = reinterpret_cast<uint32_t*>(smem + (step % kStages) * kStageElems);
        constexpr int kDwords = BM * BK / 2, kPerRow = BK / 2;
#pragma unroll
        for (int d = threadIdx.x; d < kDwords; d += C::kThreads) {
            const int r = d / kPerRow, p = d % kPerRow;
            const int k = step * BK + (((p / 4) ^ swz(r)) * 8) + (p % 4) * 2;  // the dword's first k
            const int i = m0 + r;
            if (k + 1 > i) xs[d] = k > i ? 0u : (xs[d] & 0x0000ffffu);
        }
        barrier_lds();
    };
    auto read_w1 = [&](bf16x8 (&fa)[KSTEPS][FN], int step, int ks, int i) {
        const uint16_t* wb = smem + (step % kStages) * kStageElems + BM * BK;
        if constexpr (W_KN)
            fa[ks][i] = lds_frag_tr(wb + tr_row + ks * 16 * BN + tr_col[i], wb + tr_row + (ks * 16 + 4) * BN + tr_col[i]);
        else
            fa[ks][i] = lds_frag(wb, wn * WN + i * 32 + l32, ks * 2 + h2);
    };
    // one K step with a successor: prefetch its fragments while the MFMAs run
    auto step_next = [&](bf16x8 (&fa)[KSTEPS][FN], bf16x8 (&fb)[KSTEPS][FM], bf16x8 (&na)[KSTEPS][FN],
                         bf16x8 (&nb)[KSTEPS][FM], int kt, int nk, auto masked) {
        wait_copies<kCopies>(min(kStages - 2, nk - 2 - kt) * kCopies);
        barrier_lds();  // step kt+1's stage is visible; step kt's stage is no longer read
        // TRI issues the step's copies at once (spread over the MFMAs they push the
        // edge loop past the register budget); otherwise one MFMA group apart
        const bool copy = kt + kStages < nk;
        if (TRI && copy) issue(kt + kStages);
        if constexpr (decltype(masked)::value) mask_x(kt + 1);
        read_x(nb, kt + 1);
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
            for (int i = 0; i < FN; ++i) {
#pragma unroll
                for (int j = 0; j < FM; ++j) acc[i][j] = mfma32x32x16(fa[ks][i], fb[ks][j], acc[i][j]);
                read_w1(na, kt + 1, ks, i);
                if (!TRI && copy) {
#pragma unroll
                    for (int c = 0; c < kCopies; ++c)
                        if (c % (KSTEPS * FN) == ks * FN + i) issue_one(kt + kStages, c);
                }
            }
    };
    auto step_last = [&](bf16x8 (&fa)[KSTEPS][FN], bf16x8 (&fb)[KSTEPS][FM]) {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j) acc[i][j] = mfma32x32x16(fa[ks][i], fb[ks][j], acc[i][j]);
    };

    const int nk = K / GROUPS / BK;
    constexpr std::bool_constant<false> plain{};
    constexpr std::bool_constant<TRI> edge{};
    if constexpr (kPW) {
        // Paired-w pipeline.  x step s lives in x stage s & 1, w steps 2q and 2q + 1 in
        // w stage q & 1 (one 128-byte row per feature).  Step kt (after its barrier)
        // copies x of step kt + 2 into the x stage step kt has left, and an odd step
        // also copies w pair (kt + 3) / 2 into the w stage steps kt - 1 and kt have
        // left.  Each step's x copies go out first, so the barrier of step kt waits
        // for x of step kt + 1 with only that step's later w copies still allowed in
        // flight.
        const int np = nk / 2;  // K is a multiple of 64
        constexpr int kXE = C::kPairXElems, kWE = C::kPairWElems, kPWB = C::kPairWBlocks;
        uint16_t* const xs0 = smem;
        uint16_t* const ws0 = smem + 2 * kXE;
        // w copy i of this wave fills rows 8 b .. 8 b + 7, b = wave * kPWB + i, lane l
        // landing in slot l (row 8 b + l / 8, physical chunk l % 8).  Blocks i and
        // i + 2 are 16 rows apart and share the swizzle, so two offsets serve all.
        int vwp[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int row = (wave * kPWB + h) * 8 + lane / 8;
            vwp[h] = row * K * 2 + ((lane % 8) ^ swz2(row)) * 16;
        }
        auto issue_x = [&](int step) {
            uint16_t* xs = xs0 + (step & 1) * kXE;
#pragma unroll
            for (int i = 0; i < C::kXBlocks; ++i)
                copy_block(rx, xs + (wave * C::kXBlocks + i) * 512, vx[i], step * BK * 2);
        };
        auto issue_w = [&](int pair, int i) {
            copy_block(rw, ws0 + (pair & 1) * kWE + (wave * kPWB + i) * 512, vwp[i & 1] + (i >> 1) * 32 * K,
                       pair * 4 * BK);
        };
        auto read_xp = [&](bf16x8 (&fb)[KSTEPS][FM], int step) {
            const uint16_t* xb = xs0 + (step & 1) * kXE;
#pragma unroll
            for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
                for (int j = 0; j < FM; ++j) fb[ks][j] = lds_frag(xb, j * 32 + l32, ks * 2 + h2);
        };
        // step's parity is a compile-time constant at every call
        auto read_wp = [&](bf16x8 (&fa)[KSTEPS][FN], int step, int ks, int i, auto odd) {
            const uint16_t* wb = ws0 + ((step >> 1) & 1) * kWE;
            const int row = wn * WN + i * 32 + l32;
            const int chunk = (decltype(odd)::value ? 4 : 0) + ks * 2 + h2;
            fa[ks][i] = as_bf16x8(*reinterpret_cast<const u32x4*>(wb + row * 2 * BK + ((chunk ^ swz2(row)) * 8)));
        };
        constexpr std::bool_constant<false> even{};
        constexpr std::bool_constant<true> odd{};
        auto step_pair = [&](bf16x8 (&fa)[KSTEPS][FN], bf16x8 (&fb)[KSTEPS][FM], bf16x8 (&na)[KSTEPS][FN],
                             bf16x8 (&nb)[KSTEPS][FM], int kt, auto kt_odd) {
            constexpr bool kOdd = decltype(kt_odd)::value;
            if constexpr (kOdd) wait_vm<0>();  // x of step kt + 1 was the last copy issued
            else if ((kt >> 1) + 1 < np) wait_vm<kPWB>();
            else wait_vm<0>();
            barrier_lds();  // step kt+1's operands are visible; step kt's x stage is free
            if (kt + 2 < nk) issue_x(kt + 2);
            const bool wcopy = kOdd && ((kt + 3) >> 1) < np;
            read_xp(nb, kt + 1);
#pragma unroll
            for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
                for (int i = 0; i < FN; ++i) {
#pragma unroll
                    for (int j = 0; j < FM; ++j) acc[i][j] = mfma32x32x16(fa[ks][i], fb[ks][j], acc[i][j]);
                    read_wp(na, kt + 1, ks, i, std::bool_constant<!kOdd>{});
                    if (wcopy) {  // spread over the step's MFMAs
#pragma unroll
                        for (int c = 0; c < kPWB; ++c)
                            if (c % (KSTEPS * FN) == ks * FN + i) issue_w((kt + 3) >> 1, c);
                    }
                }
        };
        issue_x(0);
#pragma unroll
        for (int c = 0; c < kPWB; ++c) issue_w(0, c);
        issue_x(1);
        if (np > 1) {
#pragma unroll
            for (int c = 0; c < kPWB; ++c) issue_w(1, c);
            wait_vm<C::kXBlocks + kPWB>();
        } else {
            wait_vm<C::kXBlocks>();
        }
        barrier_lds();
        read_xp(fb0, 0);
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
            for (int i = 0; i < FN; ++i) read_wp(fa0, 0, ks, i, even);
        int kt = 0;
        for (; kt + 2 < nk; kt += 2) {
            step_pair(fa0, fb0, fa1, fb1, kt, even);
            step_pair(fa1, fb1, fa0, fb0, kt + 1, odd);
        }
        step_pair(fa0, fb0, fa1, fb1, nk - 2, even);
        step_last(fa1, fb1);
    } else {
    // TRI: steps below kfree have every k under the tile's first row (no check);
    // the rest form the separately compiled edge loop
    const int kfree = TRI ? min(m0 / BK, nk) : nk;
#pragma unroll
    for (int st = 0; st < kStages; ++st)
        if (st < nk) issue(st);
    wait_copies<kCopies>(min(kStages - 1, nk - 1) * kCopies);
    barrier_lds();
    if (TRI && kfree == 0) mask_x(0);
    read_x(fb0, 0);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
        for (int i = 0; i < FN; ++i) read_w1(fa0, 0, ks, i);
    // K is a multiple of 64, so nk = K / 32 is even: steps pair up with one exit path
    int kt = 0;
    for (; kt + 2 < nk && kt + 2 < kfree; kt += 2) {
        step_next(fa0, fb0, fa1, fb1, kt, nk, plain);
        step_next(fa1, fb1, fa0, fb0, kt + 1, nk, plain);
    }
    if constexpr (TRI) {
        for (; kt + 2 < nk; kt += 2) {
            step_next(fa0, fb0, fa1, fb1, kt, nk, edge);
            step_next(fa1, fb1, fa0, fb0, kt + 1, nk, edge);
        }
    }
    step_next(fa0, fb0, fa1, fb1, nk - 2, nk, edge);
    step_last(fa1, fb1);
    }

    if constexpr (!HAS_RES && !W_KN && !TRI && GROUPS == 1) {
        // no residual: bias and activation on the accumulators, bf16 rows staged in
        // LDS all at once (BM rows of 512 bytes, 16-byte chunk c of row r at
        // physical chunk c ^ (r & 31)), then whole rows stored
        uint32_t* eb = reinterpret_cast<uint32_t*>(smem);
        // the wave's bias groups, all loaded before the first is used (one wait, not
        // one per group); features past N read a group in range and count as zero
        u32x2 braw[FN][4];
        if constexpr (HAS_BIAS) {
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    braw[i][g] = *reinterpret_cast<const u32x2*>(
                        bias + min(n0 + wn * WN + i * 32 + 8 * g + 4 * h2, N - 4));
        }
        barrier_lds();  // the K loop is done with LDS
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int f0 = wn * WN + i * 32 + 8 * g + 4 * h2;  // feature (in the tile) of acc[.][.][4g]
                float bv[4] = {0.f, 0.f, 0.f, 0.f};
                if constexpr (HAS_BIAS) {
                    const u32x2 bb = n0 + f0 < N ? braw[i][g] : u32x2{0u, 0u};
                    bv[0] = lo_bf16(bb[0]);
                    bv[1] = hi_bf16(bb[0]);
                    bv[2] = lo_bf16(bb[1]);
                    bv[3] = hi_bf16(bb[1]);
                }
#pragma unroll
                for (int j = 0; j < FM; ++j) {
                    const int r = j * 32 + l32;
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = activate_bf16<ACT>(acc[i][j][4 * g + e] + bv[e]);
                    const int pc = (f0 >> 3) ^ (r & 31);
                    *reinterpret_cast<u32x2*>(eb + r * 128 + pc * 4 + h2 * 2) =
                        u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                }
            }
        barrier_lds();
        // each wave instruction stores two 512-byte rows: lane / 32 picks the row, lane % 32 its chunk
        const int cl = lane % 32;
        const int n = n0 + 8 * cl;
#pragma unroll
        for (int rr = 0; rr < BM / 8; ++rr) {
            const int r = (rr * C::kWaves + wave) * 2 + h2;
            const int m = m0 + r;
            if (m < T && n < N)
                *reinterpret_cast<u32x4*>(y + (int64_t)m * ldy + n) =
                    *reinterpret_cast<const u32x4*>(eb + r * 128 + ((cl ^ (r & 31)) * 4));
        }
        return;
    }
    // Epilogue through LDS, 32 tokens at a time: the waves holding a slice write
    // their fp32 accumulators there, then all waves read whole rows back (32
    // bytes per lane, two rows of 256 features per wave instruction), apply bias,
    // activation and residual and store 512-byte rows as 16-byte chunks.
    // acc[i][j][4g + r] holds (token j*32 + l32, feature i*32 + 8g + 4*h2 + r) of
    // the wave's sub-tile.  LDS layout: row r of 64 16-byte chunks, chunk c at
    // physical slot c ^ r.
    // (GROUPS = 2: one 32-token slice region per group, the row phase adds them)
    float* ep = reinterpret_cast<float*>(smem_all);
    float* const ep_mine = ep + grp * kEpiRows * BN;
    const int cl = lane % 32;        // this lane's 16-byte output chunk of a row in the row phase
    const int ncol = n0 + 8 * cl;    // its eight output features
    float bv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    // two 8-byte bias loads (the bias need only be 8-byte aligned), unconditional so
    // that they go out with the residual loads below; features past N read a group in
    // range and count as zero.  They are unpacked only after the first slice is
    // staged, so that their wait (and the residual loads' behind them) falls there.
    u32x2 bb[2] = {u32x2{0u, 0u}, u32x2{0u, 0u}};
    if constexpr (HAS_BIAS) {
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) bb[hb] = *reinterpret_cast<const u32x2*>(bias + min(ncol, N - 8) + 4 * hb);
    }
    constexpr int kRowsPerWave = kEpiRows / (C::kWaves * GROUPS);
    constexpr int kRowPairs = kRowsPerWave / 2;  // wave instructions per slice: rows 2 p + h2
    // Residual rows are fetched for every slice at once, so their latency is paid once per tile.
    u32x4 res[HAS_RES ? BM / kEpiRows : 1][kRowPairs];
    if constexpr (HAS_RES) {
#pragma unroll
        for (int slice = 0; slice < BM / kEpiRows; ++slice)
#pragma unroll
            for (int rp = 0; rp < kRowPairs; ++rp) {
                const int m = m0 + slice * kEpiRows + wave_all * kRowsPerWave + 2 * rp + h2;
                res[slice][rp] = (m < T && ncol < N) ? *reinterpret_cast<const u32x4*>(residual + (int64_t)m * ldr + ncol)
                                                     : u32x4{0u, 0u, 0u, 0u};
            }
    }
#pragma unroll
    for (int slice = 0; slice < BM / kEpiRows; ++slice) {
        barrier_lds();  // the K loop (first slice) or the previous slice is done with LDS
        // every wave holds the slice's 32 tokens (fragment column `slice`) for its 64 features
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c = (wn * WN + i * 32 + 8 * g + 4 * h2) >> 2;
                const floatx16& a = acc[i][slice];
                const floatx4 o = {a[4 * g], a[4 * g + 1], a[4 * g + 2], a[4 * g + 3]};
                *reinterpret_cast<floatx4*>(ep_mine + (l32 * 64 + (c ^ l32)) * 4) = o;
            }
        barrier_lds();
        if constexpr (HAS_BIAS) {
            if (slice == 0) {
                asm volatile("" : "+v"(bb[0]), "+v"(bb[1]));  // not before this point
#pragma unroll
                for (int hb = 0; hb < 2; ++hb) {
                    const u32x2 b2 = ncol < N ? bb[hb] : u32x2{0u, 0u};
                    bv[4 * hb] = lo_bf16(b2[0]);
                    bv[4 * hb + 1] = hi_bf16(b2[0]);
                    bv[4 * hb + 2] = lo_bf16(b2[1]);
                    bv[4 * hb + 3] = hi_bf16(b2[1]);
                }
            }
        }
#pragma unroll
        for (int rp = 0; rp < kRowPairs; ++rp) {
            const int r = wave_all * kRowsPerWave + 2 * rp + h2;
            const int m = m0 + slice * kEpiRows + r;
            if (m < T && ncol < N) {
                float o[8];
#pragma unroll
                for (int hc = 0; hc < 2; ++hc) {
                    const int slot = ((2 * cl + hc) ^ r) * 4;
                    floatx4 t = *reinterpret_cast<const floatx4*>(ep + r * 256 + slot);
                    if constexpr (GROUPS == 2) {
                        const floatx4 t1 = *reinterpret_cast<const floatx4*>(ep + kEpiRows * BN + r * 256 + slot);
#pragma unroll
                        for (int e = 0; e < 4; ++e) t[e] += t1[e];
                    }
#pragma unroll
                    for (int e = 0; e < 4; ++e) o[4 * hc + e] = t[e];
                }
                float v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = activate_bf16<ACT>(o[e] + bv[e]);
                if constexpr (HAS_RES) {
                    const u32x4 rv = res[HAS_RES ? slice : 0][rp];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        v[2 * e] += lo_bf16(rv[e]);
                        v[2 * e + 1] += hi_bf16(rv[e]);
                    }
                }
                *reinterpret_cast<u32x4*>(y + (int64_t)m * ldy + ncol) =
                    u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                          pack_bf16x2(v[6], v[7])};
            }
        }
    }
}

// Packed linear: workgroups [0, n_full) run 128-token tiles in the grouped
// XCD-aware order; when the last round of tiles would fill at most half the
// workgroup slots (two per CU), its tiles instead run as two 64-token halves
// each, workgroups n_full onwards, so that round takes about half a tile's time.
// Workgroups from n_gemm on (if any) build a batch's plan instead: the layer's
// QKV projection carries the prelude that way, in the slots its last round of
// tiles leaves free.
static_assert(sizeof(PlanSmem) <= tile_lds_bytes<64, false>(), "the plan's LDS fits the GEMM's");
static_assert(Cfg<128>::kThreads == kFusedBatch && 2 * Cfg<64>::kThreads == kFusedMaxThreads,
              "the plan body's workgroup sizes");

template <int ACT, bool HAS_BIAS, bool HAS_RES>
__global__ __launch_bounds__(Cfg<128>::kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_gemm_bf16(const uint16_t* __restrict__ x, int ldx, const uint16_t* __restrict__ w,
                 const uint16_t* __restrict__ bias, const uint16_t* residual, int ldr, uint16_t* y, int ldy,
                 int T, int K, int N, int tiles_m, int tiles_n, int n_full, int n_gemm, PlanFillArgs pf) {
    extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
    if ((int)blockIdx.x >= n_gemm) {
        plan_fused_body(pf, blockIdx.x - n_gemm, *reinterpret_cast<PlanSmem*>(smem));
        return;
    }
    int tm, tn;
    if ((int)blockIdx.x < n_full) {
        tile_coords(blockIdx.x, n_full, tiles_m, tiles_n, tm, tn);
        gemm_tile_bf16<128, ACT, HAS_BIAS, HAS_RES>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, tm * 128,
                                                    tn * BN, smem);
    } else {
        const int u = blockIdx.x - n_full;
        group_walk(n_full + (u >> 1), tiles_m, tiles_n, tm, tn);
        const int m0 = tm * 128 + (u & 1) * 64;
        if (m0 >= T) return;  // the lower half of a tile past the last token
        gemm_tile_bf16<64, ACT, HAS_BIAS, HAS_RES>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, m0, tn * BN,
                                                   smem);
    }
}

// Launches with at most one 64-token tile per CU (small batches): one tile per
// workgroup of eight waves, the two groups of four splitting K (GROUPS = 2), so
// each SIMD holds two waves of the tile instead of one.  Workgroups from n_gemm
// on build a batch's plan (all eight waves; threads past the batch only help).
constexpr int kDualLds = 2 * tile_lds_bytes<64, false>();
static_assert(kDualLds <= 160 * 1024, "LDS budget");
static_assert(sizeof(PlanSmem) <= kDualLds, "the plan's LDS fits the GEMM's");

template <int ACT, bool HAS_BIAS, bool HAS_RES>
__global__ __launch_bounds__(2 * Cfg<64>::kThreads)
void k_gemm_bf16_dual(const uint16_t* __restrict__ x, int ldx, const uint16_t* __restrict__ w,
                      const uint16_t* __restrict__ bias, const uint16_t* residual, int ldr, uint16_t* y, int ldy,
                      int T, int K, int N, int tiles_m, int tiles_n, int n_gemm, PlanFillArgs pf) {
    extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
    if ((int)blockIdx.x >= n_gemm) {
        plan_fused_body(pf, blockIdx.x - n_gemm, *reinterpret_cast<PlanSmem*>(smem));
        return;
    }
    int tm, tn;
    tile_coords(blockIdx.x, n_gemm, tiles_m, tiles_n, tm, tn);
    gemm_tile_bf16<64, ACT, HAS_BIAS, HAS_RES, false, false, 2>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N,
                                                                tm * 64, tn * BN, smem);
}

// fp32: 64x64 tiles, K step 16, 4x4 outputs per thread, plain FMA.
template <int ACT>
__device__ __forceinline__ void gemm_tile_f32(const float* __restrict__ x, int ldx, const float* __restrict__ w,
                                              const float* __restrict__ bias, const float* residual, int ldr,
                                              float* y, int ldy, int T, int K, int N, int m0, int n0) {
    __shared__ float xs[16][64 + 1], ws[16][64 + 1];
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

template <int ACT>
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ x, int ldx, const float* __restrict__ w,
                                                   const float* __restrict__ bias, const float* residual, int ldr,
                                                   float* y, int ldy, int T, int K, int N) {
    gemm_tile_f32<ACT>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, blockIdx.x * 64, blockIdx.y * 64);
}

// fp32 on the matrix cores: v_mfma_f32_32x32x2f32 (fp32 products and fp32
// accumulation, as the VALU kernel above).  128 x 128 output tiles, four waves
// of 64 x 64; operands go global -> LDS with bounds-checked buffer loads (rows
// past T or N read as zeros) into two stages of 32 k, 128-byte rows whose
// 16-byte chunks are XOR-swizzled like the bf16 paired-w rows.  In MFMA step s
// of an 8-k group a lane supplies k = 4 (lane / 32) + s (the same k order for
// both operands), so one 16-byte LDS read feeds four MFMAs.  The MFMA computes
// C^T = W X^T: a lane holds four consecutive output features of one token,
// stored as one 16-byte vector.
constexpr int kF32K = 32;
template <int TS>
constexpr int f32_stage_floats() { return 2 * TS * kF32K; }  // TS x rows, then TS w rows

// TS = 128 (four waves of 64 x 64) or, for launches that would leave most CUs
// idle, TS = 64 (four waves of 32 x 32: four times the tiles; a wave's single
// accumulator chain still issues an fp32 MFMA every cycle the pipe allows).
template <int ACT, bool HB, bool HR, int TS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_gemm_f32_mfma(const float* __restrict__ x, int ldx, const float* __restrict__ w,
                     const float* __restrict__ bias, const float* residual, int ldr, float* y, int ldy, int T,
                     int K, int N, int tiles_m, int tiles_n) {
    static_assert(TS == 128 || TS == 64, "tile side");
    constexpr int WS = TS / 2, F = WS / 32;          // the wave's sub-tile side and 32-wide blocks
    constexpr int kStage = f32_stage_floats<TS>();
    constexpr int kBx = TS / 8, kPerWave = 2 * kBx / 4;  // 1 KB x blocks; copies per wave and step
    extern __shared__ __attribute__((aligned(16))) float fsm[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    const int l32 = lane % 32, h2 = lane / 32;
    const int wm = wave >> 1, wn = wave & 1;  // the wave's WS tokens and WS features
    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * TS, n0 = tn * TS;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x + (int64_t)m0 * ldx, (uint32_t)min(T - m0, TS) * ldx * 4u);
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(w + (int64_t)n0 * K, (uint32_t)min(N - n0, TS) * K * 4u);
    // copy block b (1 KB: 8 rows of 128 bytes; blocks 0 .. kBx - 1 x rows, then w rows):
    // this wave fills blocks kPerWave wave .. + kPerWave - 1, lane l slot l (row 8 b' + l / 8,
    // physical chunk l % 8, which holds logical chunk (l % 8) ^ swz2(row))
    int voff[8];  // first kPerWave used (a size that depends on TS made hipcc drop the host stub)
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
        const int blk = wave * kPerWave + i, bl = blk % kBx, row = bl * 8 + lane / 8;
        voff[i] = row * (blk < kBx ? ldx : K) * 4 + ((lane % 8) ^ swz2(row)) * 16;
    }
    auto issue = [&](int step) {
        float* st = fsm + (step & 1) * kStage;
#pragma unroll
        for (int i = 0; i < kPerWave; ++i) {
            const int blk = wave * kPerWave + i;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(blk < kBx ? rx : rw, (lds_void_t*)(st + blk * 256), 16, voff[i],
                                                     step * kF32K * 4, 0, 0);
        }
    };
    floatx16 acc[F][F];
#pragma unroll
    for (int i = 0; i < F; ++i)
#pragma unroll
        for (int j = 0; j < F; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    const int nk = K / kF32K;
    issue(0);
    for (int k = 0; k < nk; ++k) {
        wait_vm<0>();
        barrier_lds();  // step k's stage is visible; the other stage is no longer read
        if (k + 1 < nk) issue(k + 1);
        const float* xs = fsm + (k & 1) * kStage;
        const float* ws = xs + TS * kF32K;
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            floatx4 a[F], bq[F];
#pragma unroll
            for (int i = 0; i < F; ++i) {
                const int r = wn * WS + i * 32 + l32;
                a[i] = *reinterpret_cast<const floatx4*>(ws + r * kF32K + (((gq * 2 + h2) ^ swz2(r)) * 4));
            }
#pragma unroll
            for (int j = 0; j < F; ++j) {
                const int r = wm * WS + j * 32 + l32;
                bq[j] = *reinterpret_cast<const floatx4*>(xs + r * kF32K + (((gq * 2 + h2) ^ swz2(r)) * 4));
            }
#pragma unroll
            for (int st = 0; st < 4; ++st)
#pragma unroll
                for (int i = 0; i < F; ++i)
#pragma unroll
                    for (int j = 0; j < F; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][st], bq[j][st], acc[i][j], 0, 0, 0);
        }
    }
    // acc[i][j][4g + r]: token wm*WS + j*32 + l32, feature wn*WS + i*32 + 8g + 4 h2 + r.
    // The bias groups, and per 32-feature block the residual chunks, are loaded
    // before their first use (indexes clamped into range; one wait for each batch):
    // loaded under the range tests, each was waited for before the next was issued.
    floatx4 bv[F][4];
#pragma unroll
    for (int i = 0; i < F; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            bv[i][g] = floatx4{0.f, 0.f, 0.f, 0.f};
            if constexpr (HB) bv[i][g] = *reinterpret_cast<const floatx4*>(bias + min(n0 + wn * WS + i * 32 + 8 * g + 4 * h2, N - 4));
        }
#pragma unroll
    for (int i = 0; i < F; ++i) {
        floatx4 rv[4][F];
        if constexpr (HR) {
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int j = 0; j < F; ++j)
                    rv[g][j] = *reinterpret_cast<const floatx4*>(
                        residual + (int64_t)min(m0 + wm * WS + j * 32 + l32, T - 1) * ldr +
                        min(n0 + wn * WS + i * 32 + 8 * g + 4 * h2, N - 4));
        }
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int n = n0 + wn * WS + i * 32 + 8 * g + 4 * h2;
            if (n >= N) continue;
#pragma unroll
            for (int j = 0; j < F; ++j) {
                const int m = m0 + wm * WS + j * 32 + l32;
                if (m >= T) continue;
                floatx4 o;
#pragma unroll
                for (int r = 0; r < 4; ++r) o[r] = activate<ACT>(acc[i][j][4 * g + r] + bv[i][g][r]);
                if constexpr (HR) o += rv[g][j];
                *reinterpret_cast<floatx4*>(y + (int64_t)m * ldy + n) = o;
            }
        }
    }
}

template <int ACT, bool HB, bool HR, int TS>
hipError_t launch_f32_mfma_ts(const float* x, int ldx, const float* w, const float* bias, const float* residual,
                              int ldr, float* y, int ldy, int T, int K, int N, hipStream_t s) {
    constexpr int kLds = 2 * f32_stage_floats<TS>() * 4;
    static bool attr_set = false;  // benign race: every thread sets the same value
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm_f32_mfma<ACT, HB, HR, TS>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int tiles_m = (T + TS - 1) / TS, tiles_n = (N + TS - 1) / TS;
    hipLaunchKernelGGL((k_gemm_f32_mfma<ACT, HB, HR, TS>), dim3(tiles_m * tiles_n), dim3(256), kLds, s, x, ldx, w,
                       bias, residual, ldr, y, ldy, T, K, N, tiles_m, tiles_n);
    return hipGetLastError();
}

// 64 x 64 tiles when they cut the busiest CU's share of work, counted in rounds of
// one tile per CU (a 128 x 128 tile being four 64 x 64 ones), by a fifth or more:
// they re-read each operand twice as often, which large launches notice (35475 x
// 1024 x 4096: 139 rounds of 64 x 64 against 35 of 128 x 128 ran 7% slower)
template <int ACT, bool HB, bool HR>
hipError_t launch_f32_mfma(const float* x, int ldx, const float* w, const float* bias, const float* residual, int ldr,
                           float* y, int ldy, int T, int K, int N, hipStream_t s) {
    const int64_t cus = device_cu_count();
    const int64_t tiles128 = (int64_t)((T + 127) / 128) * ((N + 127) / 128);
    const int64_t tiles64 = (int64_t)((T + 63) / 64) * ((N + 63) / 64);
    if (5 * ((tiles64 + cus - 1) / cus) <= 16 * ((tiles128 + cus - 1) / cus))
        return launch_f32_mfma_ts<ACT, HB, HR, 64>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
    return launch_f32_mfma_ts<ACT, HB, HR, 128>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
}

template <int ACT>
hipError_t launch_f32_mfma_act(const float* x, int ldx, const float* w, const float* bias, const float* residual,
                               int ldr, float* y, int ldy, int T, int K, int N, hipStream_t s) {
    if (bias && residual) return launch_f32_mfma<ACT, true, true>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
    if (bias) return launch_f32_mfma<ACT, true, false>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
    if (residual) return launch_f32_mfma<ACT, false, true>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
    return launch_f32_mfma<ACT, false, false>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, s);
}

// The matrix-core fp32 kernel needs whole 32-k steps, 16-byte vectors (rows of x,
// w, y and residual and the bias 16-byte aligned) and N % 4 == 0.
bool f32_mfma_ok(const void* x, int ldx, const void* w, const void* bias, const void* residual, int ldr,
                 const void* y, int ldy, int K, int N) {
    auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    return K % kF32K == 0 && N % 4 == 0 && ldx % 4 == 0 && ldy % 4 == 0 && al(x) && al(w) && al(y) &&
           (!bias || al(bias)) && (!residual || (al(residual) && ldr % 4 == 0));
}

// ---------------------------------------------------------------------------
// Variable-sized batched GEMM: one workgroup per entry of the plan's tile list
// (problems largest first).  The workgroup -> entry map deals the list to the
// 8 XCDs in chunks of kVgemmChunk consecutive entries (workgroups go to the
// XCDs round-robin), so the tiles an XCD runs together mostly come from one
// problem and share its operand panels in that XCD's L2, while every XCD still
// gets a share of the large problems first.
// ---------------------------------------------------------------------------
constexpr int kVgemmChunk = 32;
constexpr int kVgemmGridQuantum = 8 * kVgemmChunk;  // the grid is a multiple of this

struct VgemmArgs {
    const int32_t* dims;
    const int64_t* a_off;
    const int64_t* b_off;
    const int64_t* c_off;
    const int4* items;
    int32_t* status;
    int batch;
    int64_t a_cap, b_cap, c_cap;
};

// The status word may be written in these kernels (atomicOr), so the compiler
// cannot keep the plan reads in scalar registers by itself; these are
// workgroup-uniform and are made so explicitly (otherwise every buffer
// descriptor built from them becomes a per-lane loop).
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int64_t uni64(int64_t v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(static_cast<uint64_t>(v) >> 32));
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// The tile one workgroup computes: problem p, output rows [m0, m0 + 128) and
// columns [n0, n0 + 256) of C_p = A_p B_p^T.
struct VgemmTile {
    int m, n, k, m0, n0;
    int64_t a_off, b_off, c_off;
};

__device__ __forceinline__ VgemmTile vgemm_tile(const VgemmArgs& va, int e) {
    const int4 it = va.items[e];
    const int p = uni(it.x);
    VgemmTile t;
    t.m = uni(va.dims[3 * p]);
    t.n = uni(va.dims[3 * p + 1]);
    t.k = uni(va.dims[3 * p + 2]);
    t.m0 = uni(it.y) * kVgemmTileM;
    t.n0 = uni(it.z) * kVgemmTileN;
    t.a_off = uni64(va.a_off[p]);
    t.b_off = uni64(va.b_off[p]);
    t.c_off = uni64(va.c_off[p]);
    return t;
}

__device__ __forceinline__ int vgemm_entry(int bid) {
    const int xcd = bid % 8, idx = bid / 8;
    return ((idx / kVgemmChunk) * 8 + xcd) * kVgemmChunk + idx % kVgemmChunk;
}

// False if the plan reports a data error or this call cannot run on it; one
// thread then records why and every workgroup returns.
__device__ __forceinline__ bool vgemm_ok(const VgemmArgs& va, bool bf16) {
    if (va.status[0] != 0) return false;
    int bad = 0;
    if (va.a_off[va.batch] > va.a_cap || va.b_off[va.batch] > va.b_cap || va.c_off[va.batch] > va.c_cap)
        bad |= kVgemmOperandCap;
    if (bf16 && va.status[2] != 0) bad |= kVgemmBf16Shape;
    if (bad) {
        if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(va.status, bad);
        return false;
    }
    return true;
}

// C = 0 over the rows [m0, m) x columns [n0, n) of a tile (problems with k = 0).
template <typename E>
__device__ __forceinline__ void vgemm_zero_tile(E* c, int m, int n, int m0, int n0, int threads) {
    const int rows = min(m - m0, kVgemmTileM), cols = min(n - n0, kVgemmTileN);
    for (int e = threadIdx.x; e < rows * cols; e += threads)
        c[(int64_t)(m0 + e / cols) * n + n0 + e % cols] = E(0);
}

__global__ __launch_bounds__(Cfg<kVgemmTileM>::kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_vgemm_bf16(VgemmArgs va, const uint16_t* __restrict__ a, const uint16_t* __restrict__ b, uint16_t* c) {
    static_assert(kVgemmTileN == BN, "vgemm tiles are the GEMM's 128 x 256 tiles");
    extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
    if (!vgemm_ok(va, true)) return;
    const int e = vgemm_entry(blockIdx.x);
    if (e >= uni(va.status[1])) return;
    const VgemmTile t = vgemm_tile(va, e);
    uint16_t* cp = c + t.c_off;
    if (t.k == 0) {
        vgemm_zero_tile(cp, t.m, t.n, t.m0, t.n0, Cfg<kVgemmTileM>::kThreads);
        return;
    }
    gemm_tile_bf16<kVgemmTileM, 0, false, false>(a + t.a_off, t.k, b + t.b_off, nullptr, nullptr, 0, cp, t.n, t.m,
                                                 t.k, t.n, t.m0, t.n0, smem);
}

// fp32: the 128 x 256 tile as eight 64 x 64 sub-tiles of the fp32 GEMM.
__global__ __launch_bounds__(256) void k_vgemm_f32(VgemmArgs va, const float* __restrict__ a,
                                                    const float* __restrict__ b, float* c) {
    if (!vgemm_ok(va, false)) return;
    const int e = vgemm_entry(blockIdx.x);
    if (e >= uni(va.status[1])) return;
    const VgemmTile t = vgemm_tile(va, e);
    for (int sub = 0; sub < (kVgemmTileM / 64) * (kVgemmTileN / 64); ++sub) {
        const int sm = t.m0 + (sub % (kVgemmTileM / 64)) * 64, sn = t.n0 + (sub / (kVgemmTileM / 64)) * 64;
        if (sm < t.m && sn < t.n)
            gemm_tile_f32<0>(a + t.a_off, t.k, b + t.b_off, nullptr, nullptr, 0, c + t.c_off, t.n, t.m, t.k, t.n, sm, sn);
    }
}

// ---------------------------------------------------------------------------
// Triangular matrix multiplication C = tril(L) B (trmm; Section 7.1): L is
// n x n, B and C are n x m, all row-major.  The reduction over k is a variable
// loop (k <= i), so the output row tile tm needs k < min(128 (tm + 1), n) only:
// tile work grows with tm.  The tiles run heaviest first (thread remapping,
// Section 4).
// ---------------------------------------------------------------------------
constexpr int kTrmmTile = 128;  // output rows per tile (the BM = 128 GEMM tile)


// Tiles are listed heaviest row first, columns ascending, and dealt to the XCDs
// in chunks of `chunk` consecutive columns (workgroups go to the XCDs
// round-robin).  With chunk = tiles_n / 8 each XCD owns the same column panels
// of B in every row (so B is fetched into one L2, not eight) and gets the same
// share of every row, hence the same total work.
__device__ __forceinline__ bool trmm_tile_coords(int bid, int tiles_m, int tiles_n, int chunk, int& tm, int& tn) {
    const int xcd = bid % 8, idx = bid / 8;
    const int t = ((idx / chunk) * 8 + xcd) * chunk + idx % chunk;
    if (t >= tiles_m * tiles_n) return false;
    tm = tiles_m - 1 - t / tiles_n;
    tn = t % tiles_n;
    return true;
}

__global__ __launch_bounds__(Cfg<kTrmmTile>::kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_trmm_bf16(const uint16_t* __restrict__ l, int ldl, const uint16_t* __restrict__ b, int ldb, uint16_t* c,
                 int ldc, int n, int m, int tiles_m, int tiles_n) {
    extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
    int tm, tn;
    if (!trmm_tile_coords(blockIdx.x, tiles_m, tiles_n, max(1, tiles_n / 8), tm, tn)) return;
    const int m0 = tm * kTrmmTile;
    const int k_end = min(m0 + kTrmmTile, (n + 63) & ~63);  // a multiple of 64; L and B past n read as zeros
    gemm_tile_bf16<kTrmmTile, 0, false, false, true, true>(l, ldl, b, nullptr, nullptr, 0, c, ldc, n, k_end, m, m0,
                                                            tn * BN, smem, ldb, n);
}

// fp32: 64 x 64 tiles of plain FMA, the reduction stopping at the tile's last row
// and L entries past the diagonal read as zero.
__global__ __launch_bounds__(256) void k_trmm_f32(const float* __restrict__ l, int ldl, const float* __restrict__ b,
                                                   int ldb, float* c, int ldc, int n, int m) {
    __shared__ float ls[16][64 + 1], bs[16][64 + 1];
    const int tiles_m = (n + 63) / 64;
    const int m0 = (tiles_m - 1 - (int)blockIdx.x) * 64, n0 = blockIdx.y * 64;  // heaviest rows first
    const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
    const int k_end = min(m0 + 64, n);
    float acc[4][4] = {};
    for (int k0 = 0; k0 < k_end; k0 += 16) {
        __syncthreads();
        for (int e = threadIdx.x; e < 64 * 16; e += 256) {
            const int r = e / 16, cc = e % 16, k = k0 + cc;
            ls[cc][r] = (m0 + r < n && k <= m0 + r) ? l[(int64_t)(m0 + r) * ldl + k] : 0.f;
            const int kr = k0 + e / 64, col = n0 + e % 64;
            bs[e / 64][e % 64] = (kr < n && col < m) ? b[(int64_t)kr * ldb + col] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int cc = 0; cc < 16; ++cc) {
            float av[4], bv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                av[u] = ls[cc][ty * 4 + u];
                bv[u] = bs[cc][tx + 16 * u];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(av[u], bv[v], acc[u][v]);
        }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int i = m0 + ty * 4 + u;
        if (i >= n) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = n0 + tx + 16 * v;
            if (j < m) c[(int64_t)i * ldc + j] = acc[u][v];
        }
    }
}

template <int ACT, bool HB, bool HR>
hipError_t launch_bf16_tiles(const void* x, int ldx, const void* w, const void* bias, const void* residual, int ldr,
                             void* y, int ldy, int T, int K, int N, const PlanView* plan, hipStream_t s) {
    constexpr int kLds = tile_lds_bytes<128, false>() > tile_lds_bytes<64, false>() ? tile_lds_bytes<128, false>()
                                                                                    : tile_lds_bytes<64, false>();
    const int tiles_m = (T + 127) / 128, tiles_n = (N + BN - 1) / BN, tiles = tiles_m * tiles_n;
    const int tiles64 = (T + 63) / 64 * tiles_n;
    const PlanFillArgs pf = plan ? plan_fill_args(*plan) : PlanFillArgs{};
    if (tiles64 <= device_cu_count() && K % 128 == 0) {  // a small launch: eight waves per tile
        static bool dual_set = false;  // benign race: every thread sets the same value
        if (!dual_set) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm_bf16_dual<ACT, HB, HR>),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, kDualLds);
            if (e != hipSuccess) return e;
            dual_set = true;
        }
        hipLaunchKernelGGL((k_gemm_bf16_dual<ACT, HB, HR>), dim3(tiles64 + (plan ? plan->batch : 0)),
                           dim3(2 * Cfg<64>::kThreads), kDualLds, s, static_cast<const uint16_t*>(x), ldx,
                           static_cast<const uint16_t*>(w), static_cast<const uint16_t*>(bias),
                           static_cast<const uint16_t*>(residual), ldr, static_cast<uint16_t*>(y), ldy, T, K, N,
                           (T + 63) / 64, tiles_n, tiles64, pf);
        return hipGetLastError();
    }
    const int slots = 2 * device_cu_count();                      // resident workgroups
    const int last = tiles - (tiles - 1) / slots * slots;         // tiles in the last round, 1..slots
    const int n_full = 2 * last <= slots ? tiles - last : tiles;  // the rest run as halves
    static bool attr_set = false;  // benign race: every thread sets the same value
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm_bf16<ACT, HB, HR>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int n_gemm = n_full + 2 * (tiles - n_full);
    hipLaunchKernelGGL((k_gemm_bf16<ACT, HB, HR>), dim3(n_gemm + (plan ? plan->batch : 0)), dim3(Cfg<128>::kThreads),
                       kLds, s, static_cast<const uint16_t*>(x), ldx, static_cast<const uint16_t*>(w),
                       static_cast<const uint16_t*>(bias), static_cast<const uint16_t*>(residual), ldr,
                       static_cast<uint16_t*>(y), ldy, T, K, N, tiles_m, tiles_n, n_full, n_gemm, pf);
    return hipGetLastError();
}

template <int ACT>
hipError_t launch_bf16_act(const void* x, int ldx, const void* w, const void* bias, const void* residual, int ldr,
                           void* y, int ldy, int T, int K, int N, const PlanView* plan, hipStream_t s) {
    auto* f = &launch_bf16_tiles<ACT, false, false>;
    if (bias && residual) f = &launch_bf16_tiles<ACT, true, true>;
    else if (bias) f = &launch_bf16_tiles<ACT, true, false>;
    else if (residual) f = &launch_bf16_tiles<ACT, false, true>;
    return f(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, plan, s);
}

}  // namespace

hipError_t launch_vgemm(const VgemmView& p, int dtype, const void* a, int64_t a_cap, const void* b, int64_t b_cap,
                        void* c, int64_t c_cap, hipStream_t s) {
    if (p.tile_cap == 0) return hipSuccess;
    const VgemmArgs va{p.dims, p.a_off, p.b_off, p.c_off, reinterpret_cast<const int4*>(p.tile_items), p.status,
                       p.batch, a_cap, b_cap, c_cap};
    const int64_t grid = (p.tile_cap + kVgemmGridQuantum - 1) / kVgemmGridQuantum * kVgemmGridQuantum;
    if (dtype == 1) {
        using C = Cfg<kVgemmTileM>;
        constexpr int kLds = tile_lds_bytes<kVgemmTileM, false>();
        static bool attr_set = false;  // benign race: every thread sets the same value
        if (!attr_set) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_vgemm_bf16),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
            if (e != hipSuccess) return e;
            attr_set = true;
        }
        hipLaunchKernelGGL(k_vgemm_bf16, dim3((unsigned)grid), dim3(C::kThreads), kLds, s, va,
                           static_cast<const uint16_t*>(a), static_cast<const uint16_t*>(b), static_cast<uint16_t*>(c));
    } else {
        hipLaunchKernelGGL(k_vgemm_f32, dim3((unsigned)grid), dim3(256), 0, s, va, static_cast<const float*>(a),
                           static_cast<const float*>(b), static_cast<float*>(c));
    }
    return hipGetLastError();
}

hipError_t launch_trmm(int dtype, const void* l, int ldl, const void* b, int ldb, void* c, int ldc, int n, int m,
                       hipStream_t s) {
    if (n == 0 || m == 0) return hipSuccess;
    if (dtype == 1) {
        using C = Cfg<kTrmmTile>;
        constexpr int kLds = tile_lds_bytes<kTrmmTile, true, true>();
        const int tiles_m = (n + kTrmmTile - 1) / kTrmmTile, tiles_n = (m + BN - 1) / BN;
        const int q = 8 * max(1, tiles_n / 8);  // the grid covers whole rounds of chunks
        const int per_xcd = (tiles_m * tiles_n + q - 1) / q * q / 8;
        static bool attr_set = false;  // benign race: every thread sets the same value
        if (!attr_set) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_trmm_bf16),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
            if (e != hipSuccess) return e;
            attr_set = true;
        }
        hipLaunchKernelGGL(k_trmm_bf16, dim3(8 * per_xcd), dim3(C::kThreads), kLds, s,
                           static_cast<const uint16_t*>(l), ldl, static_cast<const uint16_t*>(b), ldb,
                           static_cast<uint16_t*>(c), ldc, n, m, tiles_m, tiles_n);
    } else {
        hipLaunchKernelGGL(k_trmm_f32, dim3((n + 63) / 64, (m + 63) / 64), dim3(256), 0, s,
                           static_cast<const float*>(l), ldl, static_cast<const float*>(b), ldb, static_cast<float*>(c),
                           ldc, n, m);
    }
    return hipGetLastError();
}

hipError_t launch_linear(int dtype, const void* x, int ldx, const void* w, const void* bias, const void* residual,
                         int ldr, int act, void* y, int ldy, int T, int K, int N, hipStream_t s,
                         const PlanView* plan) {
    if (plan && (dtype != 1 || T == 0 || plan->batch > kFusedBatch)) {
        // the plan rides along only with a bf16 projection; otherwise its own launch goes first
        const hipError_t e = launch_offsets(*plan, s);
        if (e != hipSuccess) return e;
        plan = nullptr;
    }
    if (T == 0) return hipSuccess;
    if (dtype == 1) {
        if (act == 1) return launch_bf16_act<1>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, plan, s);
        if (act == 2) return launch_bf16_act<2>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, plan, s);
        return launch_bf16_act<0>(x, ldx, w, bias, residual, ldr, y, ldy, T, K, N, plan, s);
    }
    const dim3 grid((T + 63) / 64, (N + 63) / 64);
    const float* xf = static_cast<const float*>(x);
    const float* wf = static_cast<const float*>(w);
    const float* bf = static_cast<const float*>(bias);
    const float* rf = static_cast<const float*>(residual);
    float* yf = static_cast<float*>(y);
    if (f32_mfma_ok(x, ldx, w, bias, residual, ldr, y, ldy, K, N)) {
        if (act == 1) return launch_f32_mfma_act<1>(xf, ldx, wf, bf, rf, ldr, yf, ldy, T, K, N, s);
        if (act == 2) return launch_f32_mfma_act<2>(xf, ldx, wf, bf, rf, ldr, yf, ldy, T, K, N, s);
        return launch_f32_mfma_act<0>(xf, ldx, wf, bf, rf, ldr, yf, ldy, T, K, N, s);
    }
    if (act == 1) hipLaunchKernelGGL(k_gemm_f32<1>, grid, dim3(256), 0, s, xf, ldx, wf, bf, rf, ldr, yf, ldy, T, K, N);
    else if (act == 2) hipLaunchKernelGGL(k_gemm_f32<2>, grid, dim3(256), 0, s, xf, ldx, wf, bf, rf, ldr, yf, ldy, T, K, N);
    else hipLaunchKernelGGL(k_gemm_f32<0>, grid, dim3(256), 0, s, xf, ldx, wf, bf, rf, ldr, yf, ldy, T, K, N);
    return hipGetLastError();
}

}  // namespace rag
