/*
 * ragged.h -- C interface of the ragged (minimally padded) transformer encoder
 * layer for AMD Instinct MI355X (gfx950).
 *
 * The method is the one evaluated in "The CoRa Tensor Compiler: Compilation
 * for Ragged Tensors with Minimal Padding" (Fegade, Chen, Gibbons, Mowry;
 * MLSys 2022): a batch of B variable-length sequences (lengths L_b) is stored
 * without padding, every operator runs on real tokens only, and all accesses
 * go through exclusive prefix sums of the lengths.
 *
 * Conventions for every entry point:
 *   - Pointers are DEVICE memory unless a comment says (host).  The caller owns
 *     every buffer; the library never allocates, frees or keeps device memory.
 *   - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL
 *     is the default stream).  Nothing synchronises unless the environment
 *     variable RAG_SYNC_CHECK=1 is set, in which case each call synchronises
 *     its stream and reports device-side errors and data errors (below).
 *   - Argument errors are detected on the host before anything is launched and
 *     returned as a negative rag_status; ragged_last_error() then describes
 *     the failure (a thread-local string).
 *   - Data errors that only the device can see (bad lengths, overflowing work
 *     lists or score buffers) set bits in the plan's status word; every later
 *     kernel that uses the plan then returns without touching its outputs.
 *   - Packed activations are row-major [T, width] with a leading dimension
 *     (row stride, in elements) `ld*`, T = sum of the lengths, sequences in
 *     caller order and tokens in position order.
 *   - dtype RAG_BF16: every tensor (activations, weights, biases, LayerNorm
 *     parameters, scores, probabilities) is bfloat16; products accumulate in
 *     fp32 and softmax / LayerNorm / GELU math is fp32; results are rounded to
 *     nearest even when stored.  dtype RAG_F32: every tensor is fp32 and no
 *     reduced-precision arithmetic is used.
 *   - bf16 operands that are read with 16-byte vector loads (Q, K, V, x, w,
 *     residual, y of packed_linear, x/y of the LayerNorm) must be 16-byte
 *     aligned with leading dimensions that are multiples of 8 elements.
 *   - All functions are reentrant; calls on different streams that share no
 *     output buffer may run concurrently.
 */
#ifndef RAGGED_H
#define RAGGED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t rag_status;
enum {
    RAG_OK = 0,
    RAG_ERR_ARG = -1,       /* null pointer, negative size, bad enum value      */
    RAG_ERR_DTYPE = -2,     /* unsupported dtype                                 */
    RAG_ERR_SHAPE = -3,     /* unsupported or inconsistent shape / alignment     */
    RAG_ERR_CAPACITY = -4,  /* a capacity is too small for the declared sizes    */
    RAG_ERR_WORKSPACE = -5, /* workspace too small                               */
    RAG_ERR_HIP = -6,       /* the HIP runtime reported an error                 */
    RAG_ERR_DATA = -7       /* (RAG_SYNC_CHECK only) the plan's status word is set */
};

enum { RAG_F32 = 0, RAG_BF16 = 1 };
enum { RAG_ACT_NONE = 0, RAG_ACT_GELU_ERF = 1, RAG_ACT_GELU_TANH = 2 };

/* Tile edge of the attention work lists (rows and columns of a score tile,
 * rows of an Attn.V block). */
#define RAG_TILE 64
/* Largest batch a plan accepts. */
#define RAG_MAX_BATCH 65536
/* The only head dimension the kernels are built for. */
#define RAG_HEAD_DIM 64

/* Bits of status[0]. */
enum {
    RAG_DATA_NEG_LENGTH = 1,    /* some L_b < 0                                  */
    RAG_DATA_LONG_LENGTH = 2,   /* some L_b > max_len                            */
    RAG_DATA_TOKEN_COUNT = 4,   /* sum of L_b != total_tokens                    */
    RAG_DATA_QKT_CAP = 8,       /* more score tiles than qkt_cap                 */
    RAG_DATA_AV_CAP = 16,       /* more row blocks than av_cap                   */
    RAG_DATA_SCORE_CAP = 32     /* H * sum L_b^2 exceeds a score buffer's capacity */
};

/*
 * The prelude's auxiliary arrays for one batch of lengths (the paper's
 * Section 2 pipeline: they depend only on the lengths, so one plan serves every
 * layer of a model).  The caller fills the host fields and allocates every
 * device array; ragged_offsets() fills the arrays.
 *
 *   tok_off[B+1]   exclusive prefix sum of the lengths: token t of sequence b
 *                  is row tok_off[b] + t of every packed tensor (Section 5.1,
 *                  fused loop over the batch and length loops; Appendix B,
 *                  prefix arrays A_d)
 *   att_off[B+1]   H times the exclusive prefix sum of L_b^2: score (b, i, h, j)
 *                  lives at att_off[b] + (i*H + h)*L_b + j (Section 5.3, the
 *                  4-D attention tensor X[b][i][h][j] with vdims i and j)
 *   order[B]       sequence indices sorted by length, longest first, ties by
 *                  lower index (Appendix D, load balancing)
 *   tok_seq[T]     sequence of every token (the fused loop's map from fused
 *                  index to outer index, Section 5.2)
 *   qkt_item_off[B+1], av_item_off[B+1]
 *                  exclusive prefix sums of the per-sequence item counts, in
 *                  `order` order
 *   qkt_items[4*n] (seq, head, ti, tj): the RAG_TILE x RAG_TILE score tile
 *                  (rows ti*64.., cols tj*64..) of one sequence and head;
 *                  n = sum_b H*ceil(L_b/64)^2
 *   av_items[3*n]  (seq, head, ti): rows ti*64.. of one sequence and head;
 *                  n = sum_b H*ceil(L_b/64)
 *                  Both lists visit sequences in `order`, and within a
 *                  sequence run head-major, then ti, then tj.  No tile ever
 *                  crosses a sequence boundary.
 *   status[4]      {data-error bits, number of qkt items, number of av items,
 *                  largest length}
 */
typedef struct rag_plan {
    int32_t batch;          /* (host) B, 1 <= B <= RAG_MAX_BATCH                 */
    int32_t total_tokens;   /* (host) T the caller expects, >= 0                 */
    int32_t max_len;        /* (host) upper bound on every L_b, >= 0             */
    int32_t heads;          /* (host) H >= 1                                     */
    int64_t qkt_cap;        /* (host) capacity of qkt_items, in items            */
    int64_t av_cap;         /* (host) capacity of av_items, in items             */
    const int32_t* lengths; /* [B]                                              */
    int32_t* tok_off;       /* [B+1]                                            */
    int64_t* att_off;       /* [B+1]                                            */
    int32_t* order;         /* [B]                                              */
    int32_t* tok_seq;       /* [T] (may be NULL when T == 0)                    */
    int32_t* qkt_item_off;  /* [B+1]                                            */
    int32_t* av_item_off;   /* [B+1]                                            */
    int32_t* qkt_items;     /* [4*qkt_cap]                                      */
    int32_t* av_items;      /* [3*av_cap]                                       */
    int32_t* status;        /* [4]                                              */
} rag_plan;

/* Weights of one encoder layer, each [out, in] row-major (y = x W^T + b) and
 * contiguous.  w_qkv is [3d, d] (rows 0..d-1 make Q, d..2d-1 K, 2d..3d-1 V; head
 * h uses columns h*dh..h*dh+dh-1 of each), w_o [d, d], w_ff1 [d_ff, d],
 * w_ff2 [d, d_ff]; biases and LayerNorm gamma/beta are vectors. */
typedef struct rag_layer_weights {
    const void *w_qkv, *b_qkv, *w_o, *b_o, *ln1_g, *ln1_b;
    const void *w_ff1, *b_ff1, *w_ff2, *b_ff2, *ln2_g, *ln2_b;
} rag_layer_weights;

/* Short name of a status code (static string). */
const char* ragged_status_string(rag_status s);

/* Description of the last error on the calling thread (static per thread). */
const char* ragged_last_error(void);

/*
 * (host only)  Capacities that always suffice for a batch with these host
 * values: av_cap = H * min(B*ceil(max_len/64), floor((T + 63B)/64)) and
 * qkt_cap = ceil(max_len/64) * av_cap.  Launches nothing.
 */
rag_status ragged_plan_capacity(int32_t batch, int32_t total_tokens, int32_t max_len,
                                int32_t heads, int64_t* qkt_cap /* (host) out */,
                                int64_t* av_cap /* (host) out */);

/*
 * Build the plan's device arrays from plan->lengths (the prelude; Section 2,
 * Section 5.3, Appendix B).  The status word is rewritten from scratch, so a
 * plan can be rebuilt for new lengths.  Host errors: RAG_ERR_ARG for null
 * pointers or out-of-range host fields, RAG_ERR_CAPACITY if a capacity exceeds
 * 2^31-1.  Data errors go to status[0].
 */
rag_status ragged_offsets(rag_plan* plan, void* stream);

/*
 * Ragged QK^T (the layer's QK^T operator): for every sequence b, head h and
 * positions i, j < L_b,
 *   scores[att_off[b] + (i*H + h)*L_b + j] = scale * sum_c q[(tok_off[b]+i)*ldq + h*hd + c]
 *                                                  * k[(tok_off[b]+j)*ldk + h*hd + c]
 * with hd = head_dim (must be RAG_HEAD_DIM), ldq, ldk >= H*hd.  `scores` holds
 * score_cap elements; if H * sum L_b^2 > score_cap nothing is written and
 * RAG_DATA_SCORE_CAP is set.
 */
rag_status ragged_qkt(const rag_plan* plan, const void* q, int32_t ldq, const void* k, int32_t ldk,
                      int32_t head_dim, float scale, void* scores, int64_t score_cap,
                      int32_t dtype, void* stream);

/*
 * Ragged row softmax (the layer's Softmax operator): each of the H*T rows
 * (b, i, h) holds L_b scores; probs_j = exp(s_j - max s) / sum exp(s - max s).
 * `probs` may equal `scores` (in place); otherwise the two must not overlap.
 */
rag_status ragged_softmax(const rag_plan* plan, const void* scores, void* probs, int64_t score_cap,
                          int32_t dtype, void* stream);

/*
 * Ragged Attn.V (the layer's AttnV operator, a reduction over the vloop j):
 *   out[(tok_off[b]+i)*ldo + h*hd + c] = sum_{j<L_b} probs[att_off[b] + (i*H+h)*L_b + j]
 *                                               * v[(tok_off[b]+j)*ldv + h*hd + c]
 */
rag_status ragged_attn_v(const rag_plan* plan, const void* probs, int64_t score_cap, const void* v,
                         int32_t ldv, int32_t head_dim, void* out, int32_t ldo, int32_t dtype,
                         void* stream);

/*
 * Fused ragged attention (bf16, any sequence length): the composition of
 * ragged_qkt, ragged_softmax and ragged_attn_v,
 *   out[t_i][h*hd + c] = sum_j softmax_j(scale * q_i . k_j) v[t_j][h*hd + c],
 * computed per (sequence, head) in one pass over the keys without storing
 * scores or probabilities: fp32 scores, an online softmax, bf16 unnormalised
 * exponentials as the operand of the P.V product and one division by the row
 * sum (so it differs from the three operators by rounding only).  The keys
 * stream through LDS in chunks, so no length limit applies beyond 32-bit byte
 * offsets within a sequence.  Same operand rules as the three operators;
 * RAG_ERR_DTYPE unless bf16, RAG_ERR_SHAPE if max_len * max(ldk, ldv) * 2
 * exceeds 2^31 - 1.
 */
rag_status ragged_attention(const rag_plan* plan, const void* q, int32_t ldq, const void* k, int32_t ldk,
                            const void* v, int32_t ldv, int32_t head_dim, float scale, void* out,
                            int32_t ldo, int32_t dtype, void* stream);

/*
 * Masked (causal) attention, the decoder's masked MHA (Section 7.2; Appendix D,
 * masked SDPA): position i attends to keys j <= i only, so each sequence's
 * attention matrix is lower triangular.  Same arguments, layout and errors as
 * the unmasked calls above, with these differences:
 *   ragged_qkt_causal      writes only the entries j <= i of each [L_b x L_b]
 *                          block (tiles above the diagonal are skipped; the
 *                          upper triangle of `scores` is left untouched);
 *   ragged_softmax_causal  row (b, i, h) covers its i + 1 scores j <= i, and
 *                          only those entries of `probs` are written;
 *   ragged_attn_v_causal   sums over j <= i (entries j > i of `probs` are not
 *                          read);
 *   ragged_attention_causal  the fused path, walking keys up to each query.
 */
rag_status ragged_qkt_causal(const rag_plan* plan, const void* q, int32_t ldq, const void* k, int32_t ldk,
                             int32_t head_dim, float scale, void* scores, int64_t score_cap,
                             int32_t dtype, void* stream);
rag_status ragged_softmax_causal(const rag_plan* plan, const void* scores, void* probs, int64_t score_cap,
                                 int32_t dtype, void* stream);
rag_status ragged_attn_v_causal(const rag_plan* plan, const void* probs, int64_t score_cap, const void* v,
                                int32_t ldv, int32_t head_dim, void* out, int32_t ldo, int32_t dtype,
                                void* stream);
rag_status ragged_attention_causal(const rag_plan* plan, const void* q, int32_t ldq, const void* k,
                                   int32_t ldk, const void* v, int32_t ldv, int32_t head_dim, float scale,
                                   void* out, int32_t ldo, int32_t dtype, void* stream);

/*
 * Packed-token linear operator (Proj1 / Proj2 / FF1 / FF2 of the layer, run
 * over the T real tokens only: Section 5.1 and Section 7.2):
 *   y[t][n] = act(sum_k x[t][k] * w[n][k] + bias[n]) + residual[t][n]
 * x [T, K] (ldx), w [N, K] contiguous, bias [N] or NULL, residual [T, N] (ldr)
 * or NULL, y [T, N] (ldy).  bf16 requires K % 64 == 0 and N % 64 == 0.
 * y must not overlap x or w; it may equal residual (same ld).  With T == 0
 * nothing is accessed and the data pointers may be NULL.
 */
rag_status packed_linear(const void* x, int32_t ldx, const void* w, const void* bias,
                         const void* residual, int32_t ldr, int32_t act, void* y, int32_t ldy,
                         int32_t T, int32_t K, int32_t N, int32_t dtype, void* stream);

/*
 * LayerNorm over the d features of each of T token rows (the layer's two
 * LayerNorm operators): y = gamma * (x - mean) / sqrt(var + eps) + beta with
 * the population variance.  bf16 requires d % 8 == 0 and d <= 4096.
 * y may equal x (same ld).  With T == 0 the data pointers may be NULL.
 */
rag_status packed_layernorm(const void* x, int32_t ldx, const void* gamma, const void* beta,
                            float eps, void* y, int32_t ldy, int32_t T, int32_t d, int32_t dtype,
                            void* stream);

/*
 * Variable-sized batched GEMM (vgemm; Section 7.1, the matrix-multiplication
 * experiments): a batch of B independent products with their own sizes,
 *   C_b[i][j] = sum_{l < k_b} A_b[i][l] * B_b[j][l],   i < m_b, j < n_b,
 * A_b [m_b, k_b], B_b [n_b, k_b] (both with the reduction dimension contiguous)
 * and C_b [m_b, n_b], all row-major.  The three operands of the whole batch are
 * stored packed, each problem right after the previous one with no padding:
 * A_b starts at element a_off[b] of `a`, B_b at b_off[b] of `b`, C_b at c_off[b]
 * of `c`.  The work is split into RAG_VGEMM_TILE_M x RAG_VGEMM_TILE_N tiles of
 * the outputs; tiles at a problem's edge are predicated, never padded in memory.
 */
#define RAG_VGEMM_TILE_M 128
#define RAG_VGEMM_TILE_N 256
/* Largest batch a vgemm plan accepts, and largest m, n or k of one problem. */
#define RAG_VGEMM_MAX_BATCH 4096
#define RAG_VGEMM_MAX_DIM 65536
/* Largest tile_cap a vgemm plan accepts. */
#define RAG_VGEMM_MAX_TILES (1 << 30)

/* Bits of a vgemm plan's status[0]. */
enum {
    RAG_VGEMM_NEG_SIZE = 1,     /* some m, n or k < 0                                */
    RAG_VGEMM_LARGE_SIZE = 2,   /* some m, n or k > RAG_VGEMM_MAX_DIM                */
    RAG_VGEMM_TILE_CAP = 4,     /* more output tiles than tile_cap                   */
    RAG_VGEMM_OPERAND_CAP = 8,  /* (set by ragged_vgemm) a, b or c smaller than the
                                   packed batch (a_off[B], b_off[B], c_off[B])       */
    RAG_VGEMM_BF16_SHAPE = 16   /* (set by ragged_vgemm with RAG_BF16) some k % 64 or
                                   n % 8 is not 0                                    */
};

/*
 * The vgemm prelude's auxiliary arrays (the same role as rag_plan: they depend
 * only on the sizes, so one plan serves every call on a batch of that shape).
 * The caller fills the host fields and allocates every device array;
 * vgemm_offsets() fills the arrays.
 *   a_off, b_off, c_off [B+1]  exclusive prefix sums of m_b k_b, n_b k_b, m_b n_b
 *   order[B]        problems by m_b n_b k_b (multiply-adds), largest first,
 *                   ties by lower index (thread remapping, Section 4 and
 *                   Appendix A.1: the largest work is scheduled first)
 *   tile_off[B+1]   exclusive prefix sum, in `order` order, of the tile counts
 *                   ceil(m_b / RAG_VGEMM_TILE_M) * ceil(n_b / RAG_VGEMM_TILE_N)
 *   tile_items[4*n] (problem, tile row, tile column, 0) for every output tile:
 *                   problems in `order`, tile rows fastest inside a problem;
 *                   n = tile_off[B]
 *   status[3]       {data-error bits, n, 1 if some problem breaks the bf16
 *                   shape rule of ragged_vgemm (k_b % 64 == 0, n_b % 8 == 0)}
 */
typedef struct rag_vgemm_plan {
    int32_t batch;          /* (host) B, 1 <= B <= RAG_VGEMM_MAX_BATCH           */
    int64_t tile_cap;       /* (host) capacity of tile_items, in tiles,
                               0 <= tile_cap <= RAG_VGEMM_MAX_TILES              */
    const int32_t* dims;    /* [3*B] (m_b, n_b, k_b)                             */
    int64_t* a_off;         /* [B+1]                                            */
    int64_t* b_off;         /* [B+1]                                            */
    int64_t* c_off;         /* [B+1]                                            */
    int32_t* order;         /* [B]                                              */
    int64_t* tile_off;      /* [B+1]                                            */
    int32_t* tile_items;    /* [4*tile_cap], 16-byte aligned                    */
    int32_t* status;        /* [3]                                              */
} rag_vgemm_plan;

/*
 * (host only)  A tile_cap that always suffices when every m_b <= max_m and
 * n_b <= max_n: batch * ceil(max_m / 128) * ceil(max_n / 256).  Launches
 * nothing.  ragged_vgemm launches one workgroup per tile of tile_cap, so a
 * capacity far above the real tile count costs idle workgroups.
 */
rag_status vgemm_plan_capacity(int32_t batch, int32_t max_m, int32_t max_n, int64_t* tile_cap /* (host) out */);

/*
 * (host only)  The exact number of output tiles of a batch whose sizes the
 * caller also holds on the host: dims (host) is [batch][3] of (m_b, n_b, k_b),
 * the same array plan->dims holds on the device, and *tiles receives
 * sum_b ceil(m_b / RAG_VGEMM_TILE_M) * ceil(n_b / RAG_VGEMM_TILE_N), the
 * smallest tile_cap that serves the batch.  RAG_ERR_ARG for a NULL pointer, a
 * batch outside [1, RAG_VGEMM_MAX_BATCH] or a size outside [0,
 * RAG_VGEMM_MAX_DIM].  Launches nothing.
 */
rag_status vgemm_tile_count(int32_t batch, const int32_t* dims /* (host) */, int64_t* tiles /* (host) out */);

/*
 * Build the vgemm plan's device arrays from plan->dims.  The status word is
 * rewritten from scratch.  Host errors: RAG_ERR_ARG for null or misaligned
 * arrays and out-of-range host fields, RAG_ERR_CAPACITY if tile_cap exceeds
 * RAG_VGEMM_MAX_TILES.
 * Data errors (negative or too large sizes, too many tiles) go to status[0]
 * and make ragged_vgemm return without writing.
 */
rag_status vgemm_offsets(rag_vgemm_plan* plan, void* stream);

/*
 * The vgemm itself over a plan built by vgemm_offsets(): every tile of every
 * problem, largest problems first.  a, b and c hold a_cap, b_cap and c_cap
 * elements; if the packed batch does not fit, nothing is written and
 * RAG_VGEMM_OPERAND_CAP is set (like every data-error bit it stays set until
 * vgemm_offsets() rebuilds the plan).  dtype RAG_BF16 (fp32 accumulation, products
 * rounded to nearest even when stored) needs every k_b % 64 == 0 and every
 * n_b % 8 == 0, else nothing is written and RAG_VGEMM_BF16_SHAPE is set; a,
 * b, c must then be 16-byte aligned.  dtype RAG_F32 takes any sizes.  A problem
 * with k_b == 0 gets C_b = 0.  c must not overlap a or b.
 */
rag_status ragged_vgemm(const rag_vgemm_plan* plan, const void* a, int64_t a_cap, const void* b,
                        int64_t b_cap, void* c, int64_t c_cap, int32_t dtype, void* stream);

/*
 * Triangular matrix multiplication (trmm; Section 7.1, the matrix-multiplication
 * experiments): a square lower-triangular L times a dense B,
 *   C[i][j] = sum_{k <= i} L[i][k] * B[k][j],   i < n, j < m,
 * L [n, n] (ldl >= n), B [n, m] (ldb >= m), C [n, m] (ldc >= m), all row-major.
 * Row i of L holds its nonzeros in columns 0..i, so the reduction is a
 * variable loop whose extent grows with the row; entries above the diagonal
 * never reach the result (they may hold anything, NaN included).  Output row
 * tiles with the most work run first.  dtype RAG_BF16 (fp32 accumulation,
 * rounded to nearest even when stored) needs m, ldl, ldb and ldc to be
 * multiples of 8, 16-byte aligned operands, (n + 64) * ldb < 2^30 and
 * ldl < 2^23; RAG_F32 takes
 * any sizes.  C must not overlap L or B.  With n == 0 or m == 0 nothing is
 * accessed.
 */
rag_status ragged_trmm(const void* l, int32_t ldl, const void* b, int32_t ldb, void* c, int32_t ldc, int32_t n,
                       int32_t m, int32_t dtype, void* stream);

/* encoder_layer flags */
enum {
    RAG_LAYER_UNFUSED_ATTENTION = 1, /* run ragged_qkt/softmax/attn_v with a
                                        materialised score buffer in the workspace */
    RAG_LAYER_CAUSAL = 2,            /* masked attention (position i sees keys j <= i):
                                        the decoder variant of the layer */
    RAG_LAYER_BUILD_PLAN = 4         /* build the plan first, exactly as ragged_offsets()
                                        would (bf16 batches of up to 256 sequences: inside
                                        the QKV projection's launch, which does not read it) */
};

/* Number of events encoder_layer records when `events` is not NULL. */
#define RAG_LAYER_EVENTS 10

/*
 * (host only)  Workspace bytes encoder_layer needs for these sizes.  With
 * RAG_LAYER_UNFUSED_ATTENTION, and always for RAG_F32 or max_len * 3 * d_model
 * * 2 > 2^31 - 1 (where the fused attention kernel does not apply), the score
 * buffer is sized for the worst case H * T * max_len.
 */
rag_status encoder_layer_workspace(int32_t total_tokens, int32_t max_len, int32_t d_model,
                                   int32_t heads, int32_t d_ff, int32_t dtype, int32_t flags,
                                   size_t* bytes /* (host) out */);

/*
 * One post-LayerNorm Transformer encoder layer over the packed real tokens
 * (the paper's nine-operator layer, Section 7.2 and Appendix D):
 *   QKV = x Wqkv^T + bqkv;  P = softmax(Q K^T / sqrt(dh)) per sequence and head;
 *   O = P V;  H1 = LN1(O Wo^T + bo + x);  y = LN2(act(H1 W1^T + b1) W2^T + b2 + H1)
 * `plan` must have been built by ragged_offsets() for the batch (it is then
 * only read), unless `flags` holds RAG_LAYER_BUILD_PLAN: the layer then fills
 * the plan's arrays itself before its attention stage, with the same results
 * and data-error reporting as ragged_offsets().  x, y are [T, d_model] contiguous and must not overlap.  `events`, if
 * not NULL, holds RAG_LAYER_EVENTS hipEvent_t handles created by the caller:
 * events[k] is recorded on `stream` before stage k and events[9] after stage
 * 8, with the stages 0 QKV projection, 1 QK^T, 2 softmax, 3 Attn.V, 4 output
 * projection, 5 LayerNorm 1, 6 FF1, 7 FF2, 8 LayerNorm 2.  With fused
 * attention (the default) stages 1 and 2 are empty and stage 3 holds the one
 * fused attention kernel.
 * After a data error (a bit set in the plan's status word, by this call's
 * own prelude or an earlier one) the attention stage writes nothing, while
 * the token-wise stages (projections, LayerNorms) still run over the T rows
 * the host declared: y then holds unspecified values and must be discarded.
 * RAG_SYNC_CHECK=1 reports the condition as RAG_ERR_DATA.
 */
rag_status encoder_layer(const rag_plan* plan, const void* x, void* y, int32_t d_model,
                         int32_t heads, int32_t head_dim, int32_t d_ff, float ln_eps, int32_t act,
                         int32_t flags, const rag_layer_weights* w, void* workspace,
                         size_t workspace_bytes, int32_t dtype, void* stream,
                         void* const* events);

/*
 * encoder_layer for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same layer, arguments, results and errors as encoder_layer with events ==
 * NULL, but its workspace is a fixed device array of RAG_NOALLOC_SCRATCH_BYTES
 * inside the library (each GPU the library runs on holds its own copy until the
 * process ends).  The call allocates nothing.  RAG_ERR_WORKSPACE if the layer
 * would need more than that (encoder_layer_workspace gives the size), checked
 * on the host before anything launches.  Every call on one GPU shares that
 * GPU's array, so calls that overlap in time on one GPU (different streams or
 * host threads without ordering between them) race and must not be issued;
 * calls ordered on one stream are fine.  The array needs no clearing: the layer
 * writes every intermediate element before reading it.
 */
#define RAG_NOALLOC_SCRATCH_BYTES (64u << 20)
rag_status encoder_layer_noalloc(const rag_plan* plan, const void* x, void* y, int32_t d_model,
                                 int32_t heads, int32_t head_dim, int32_t d_ff, float ln_eps, int32_t act,
                                 int32_t flags, const rag_layer_weights* w, int32_t dtype, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RAGGED_H */
