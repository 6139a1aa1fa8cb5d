/*
 * oracle.c -- CPU oracle for the ragged (minimally padded) transformer encoder
 * layer evaluated in "The CoRa Tensor Compiler: Compilation for Ragged Tensors
 * with Minimal Padding" (Fegade, Chen, Gibbons, Mowry; MLSys 2022).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file: only the tests, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no code, header or table with the GPU path.
 *
 * Everything here is the plain definition, evaluated sequence by sequence on
 * real tokens only (nothing padded is materialised):
 *   - sums and products are accumulated in double precision;
 *   - a value is rounded to the storage type (bf16 with round-to-nearest-even,
 *     or fp32) exactly where a tensor of the library interface is stored.
 * Ragged storage and the tiling of the work change no arithmetic, so the
 * method's result is the plain result (up to rounding order).
 *
 * Readings of points the paper leaves open (each also listed in the design
 * notes of the repository):
 *   - scores are scaled by a caller-given factor (1/sqrt(head_dim) in the
 *     layer) applied to the finished dot product;
 *   - softmax subtracts the row maximum before exponentiating;
 *   - post-LayerNorm layer: the output projection adds the layer input as the
 *     residual, FF2 adds the first LayerNorm's output;
 *   - LayerNorm uses the population variance and a caller-given epsilon;
 *   - the FF1 activation is GELU (erf form by default, tanh form optional);
 *   - work lists order sequences by length, longest first, ties by index.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_F32 = 0, OR_BF16 = 1 };
enum { OR_ACT_NONE = 0, OR_ACT_GELU_ERF = 1, OR_ACT_GELU_TANH = 2 };

/* ------------------------------------------------------------------------ */
/* Storage types                                                              */
/* ------------------------------------------------------------------------ */

/* Round a double to the nearest bfloat16 value (ties to even) and return it as a
 * double.  bfloat16 keeps 8 significant bits and float32's exponent range, so
 * the quantum of a normal value m*2^e (0.5 <= |m| < 1) is 2^(e-8), and the
 * subnormal quantum is 2^-133.  rint() rounds ties to even in the default
 * rounding mode. */
static double bf16_round(double v) {
    if (isnan(v)) return v;
    if (isinf(v) || v == 0.0) return v;
    int e;
    frexp(v, &e);
    int qexp = e - 8;
    if (qexp < -133) qexp = -133;
    double q = ldexp(rint(ldexp(v, -qexp)), qexp);
    const double bf16_max = ldexp(255.0, 120); /* (2 - 2^-7) * 2^127 */
    if (fabs(q) > bf16_max) return v > 0 ? INFINITY : -INFINITY;
    return q;
}

static uint16_t bf16_bits_of(double rounded) {
    if (isnan(rounded)) return 0x7FC0;
    float f = (float)rounded; /* exact: every bfloat16 value is a float32 value */
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

static double bf16_value(uint16_t bits) {
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* Element `i` of a stored tensor, widened exactly to double. */
static double load(const void* base, int dtype, int64_t i) {
    if (dtype == OR_F32) return (double)((const float*)base)[i];
    return bf16_value(((const uint16_t*)base)[i]);
}

/* Round `v` to the storage type and store it as element `i`. */
static void store(void* base, int dtype, int64_t i, double v) {
    if (dtype == OR_F32) ((float*)base)[i] = (float)v; /* C conversion rounds to nearest even */
    else ((uint16_t*)base)[i] = bf16_bits_of(bf16_round(v));
}

/* Exposed for the tests: round a double array to bf16 bits. */
void oracle_round_bf16(int64_t n, const double* in, uint16_t* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = bf16_bits_of(bf16_round(in[i]));
}

/* ------------------------------------------------------------------------ */
/* Offsets and work lists (the prelude's auxiliary arrays)                    */
/* ------------------------------------------------------------------------ */

/* Token offsets: the storage offset of the first token of sequence b in a
 * [batch, vdim len, d] tensor whose batch and length dims are fused (Section
 * 5.1, fused loop bound F = sum of s(o); Appendix B, the A_d prefix arrays).
 * tok_off[b] = sum_{b' < b} L_b'  (exclusive, B+1 entries). */
static void token_offsets(int32_t B, const int32_t* L, int64_t* tok_off) {
    tok_off[0] = 0;
    for (int32_t b = 0; b < B; ++b) tok_off[b + 1] = tok_off[b] + L[b];
}

/* Attention offsets: the 4-D attention tensor X[b][i][h][j] of Section 5.3 has
 * cdims batch and heads and two vdims of size L_b.  Its batch dimension's
 * prefix array is A_1[b] = sum_{b' < b} L_b'^2 (Appendix B), and the
 * offset of X[b][i][h][j] is H*A_1[b] + i*H*L_b + h*L_b + j.
 * att_off[b] = H * sum_{b' < b} L_b'^2  (exclusive, B+1 entries). */
static void attention_offsets(int32_t B, const int32_t* L, int32_t H, int64_t* att_off) {
    att_off[0] = 0;
    for (int32_t b = 0; b < B; ++b) att_off[b + 1] = att_off[b] + (int64_t)H * L[b] * L[b];
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

/*
 * The prelude's arrays for one batch (Section 2 pipeline; Section 5.3 and
 * Appendix B storage offsets; Appendix D, load balancing: the sequences are
 * ordered longest first so that the largest blocks of work start first).
 *
 *   tok_off[B+1], att_off[B+1]       exclusive prefix sums above
 *   order[B]                         stable sort of the sequence indices by
 *                                    length, descending (ties: lower index first)
 *   tok_seq[T]                       token -> sequence (the fused loop's map
 *                                    from fused index to outer index, Section 5.2)
 *   qkt_item_off[B+1], av_item_off[B+1]
 *                                    exclusive prefix sums, in `order` order, of
 *                                    the per-sequence item counts
 *   qkt_items[4*n]  (seq, head, ti, tj): one tile_m x tile_n tile of one
 *                   sequence's L x L score block of one head
 *   av_items[3*n]   (seq, head, ti): one tile_m row block of one head
 *   Within a sequence the items run head-major, then ti, then tj.
 *
 * counts[0] = number of qkt items, counts[1] = number of av items.
 * Returns 0, or 1 if a length is negative, 2 if a capacity is exceeded
 * (counts are still reported; nothing beyond a capacity is written).
 */
int oracle_offsets(int32_t B, const int32_t* L, int32_t H, int32_t tile_m, int32_t tile_n,
                   int64_t* tok_off, int64_t* att_off, int32_t* order, int32_t* tok_seq,
                   int64_t* qkt_item_off, int64_t* av_item_off,
                   int32_t* qkt_items, int64_t qkt_cap, int32_t* av_items, int64_t av_cap,
                   int64_t* counts) {
    for (int32_t b = 0; b < B; ++b)
        if (L[b] < 0) return 1;
    token_offsets(B, L, tok_off);
    attention_offsets(B, L, H, att_off);

    /* Stable descending sort by insertion: a later index never passes an
     * equal-length earlier one. */
    for (int32_t b = 0; b < B; ++b) order[b] = b;
    for (int32_t k = 1; k < B; ++k) {
        int32_t cur = order[k];
        int32_t p = k - 1;
        while (p >= 0 && L[order[p]] < L[cur]) {
            order[p + 1] = order[p];
            --p;
        }
        order[p + 1] = cur;
    }

    if (tok_seq)
        for (int32_t b = 0; b < B; ++b)
            for (int64_t t = tok_off[b]; t < tok_off[b + 1]; ++t) tok_seq[t] = b;

    int64_t nq = 0, na = 0;
    int rc = 0;
    qkt_item_off[0] = 0;
    av_item_off[0] = 0;
    for (int32_t k = 0; k < B; ++k) {
        int32_t b = order[k];
        int64_t nti = ceil_div(L[b], tile_m), ntj = ceil_div(L[b], tile_n);
        for (int32_t h = 0; h < H; ++h) {
            for (int64_t ti = 0; ti < nti; ++ti) {
                for (int64_t tj = 0; tj < ntj; ++tj) {
                    if (nq < qkt_cap) {
                        int32_t* it = qkt_items + 4 * nq;
                        it[0] = b; it[1] = h; it[2] = (int32_t)ti; it[3] = (int32_t)tj;
                    } else {
                        rc = 2;
                    }
                    ++nq;
                }
                if (na < av_cap) {
                    int32_t* it = av_items + 3 * na;
                    it[0] = b; it[1] = h; it[2] = (int32_t)ti;
                } else {
                    rc = 2;
                }
                ++na;
            }
        }
        qkt_item_off[k + 1] = nq;
        av_item_off[k + 1] = na;
    }
    counts[0] = nq;
    counts[1] = na;
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Scaled dot-product attention on ragged storage                             */
/* ------------------------------------------------------------------------ */

/*
 * Ragged QK^T (the QK^T operator of the layer; Appendix D, per-operator
 * breakdown table of the transformer-layer discussion): for every sequence b, head h and positions i, j < L_b,
 *   S[b][i][h][j] = rd(scale * sum_{c < dh} Q[t_i][h*dh + c] * K[t_j][h*dh + c])
 * with t_i = tok_off[b] + i, Q/K packed [T, >= H*dh] with row strides ldq/ldk,
 * and S in the X[b][i][h][j] layout of Section 5.3.
 * causal != 0 gives masked attention (the decoder's masked MHA, Section 7.2 and
 * Appendix D): position i sees keys j <= i only, so only the lower triangle
 * j <= i of each [L_b x L_b] block is computed and written; entries j > i are
 * left untouched.
 */
void oracle_qkt(int dtype, int32_t B, const int32_t* L, int32_t H, int32_t dh,
                const void* q, int64_t ldq, const void* k, int64_t ldk, double scale, int causal, void* S) {
    int64_t* tok_off = malloc(sizeof(int64_t) * (B + 1));
    int64_t* att_off = malloc(sizeof(int64_t) * (B + 1));
    token_offsets(B, L, tok_off);
    attention_offsets(B, L, H, att_off);
    for (int32_t b = 0; b < B; ++b) {
        int64_t n = L[b];
        for (int64_t i = 0; i < n; ++i)
            for (int32_t h = 0; h < H; ++h)
                for (int64_t j = 0; j < (causal ? i + 1 : n); ++j) {
                    double acc = 0.0;
                    for (int32_t c = 0; c < dh; ++c)
                        acc += load(q, dtype, (tok_off[b] + i) * ldq + (int64_t)h * dh + c) *
                               load(k, dtype, (tok_off[b] + j) * ldk + (int64_t)h * dh + c);
                    store(S, dtype, att_off[b] + (i * H + h) * n + j, scale * acc);
                }
    }
    free(tok_off);
    free(att_off);
}

/*
 * Ragged row softmax (the Softmax operator): every row (b, i, h) of S holds L_b
 * scores; P_j = rd(exp(S_j - m) / sum_k exp(S_k - m)), m = max_k S_k.
 * P may alias S.  With causal != 0 row (b, i, h) holds the i + 1 scores j <= i
 * (masked attention); entries j > i are neither read nor written.
 */
void oracle_softmax(int dtype, int32_t B, const int32_t* L, int32_t H, int causal, const void* S, void* P) {
    int64_t base = 0;
    double* e = NULL;
    int64_t ecap = 0;
    for (int32_t b = 0; b < B; ++b) {
        int64_t n = L[b];
        if (n > ecap) {
            free(e);
            e = malloc(sizeof(double) * n);
            ecap = n;
        }
        for (int64_t r = 0; r < n * H; ++r) {
            int64_t row = base + r * n;
            int64_t len = causal ? r / H + 1 : n;  /* row r is position i = r / H of head r % H */
            double m = -INFINITY;
            for (int64_t j = 0; j < len; ++j) {
                double s = load(S, dtype, row + j);
                if (s > m) m = s;
            }
            double sum = 0.0;
            for (int64_t j = 0; j < len; ++j) {
                e[j] = exp(load(S, dtype, row + j) - m);
                sum += e[j];
            }
            for (int64_t j = 0; j < len; ++j) store(P, dtype, row + j, e[j] / sum);
        }
        base += (int64_t)H * n * n;
    }
    free(e);
}

/*
 * Ragged Attn.V (the AttnV operator, a reduction over the vloop j):
 *   O[t_i][h*dh + c] = rd(sum_{j < L_b} P[b][i][h][j] * V[t_j][h*dh + c]).
 * O is packed [T, >= H*dh] with row stride ldo.  With causal != 0 the sum runs
 * over j <= i (masked attention).
 */
void oracle_attn_v(int dtype, int32_t B, const int32_t* L, int32_t H, int32_t dh, int causal,
                   const void* P, const void* v, int64_t ldv, void* O, int64_t ldo) {
    int64_t* tok_off = malloc(sizeof(int64_t) * (B + 1));
    int64_t* att_off = malloc(sizeof(int64_t) * (B + 1));
    token_offsets(B, L, tok_off);
    attention_offsets(B, L, H, att_off);
    for (int32_t b = 0; b < B; ++b) {
        int64_t n = L[b];
        for (int64_t i = 0; i < n; ++i)
            for (int32_t h = 0; h < H; ++h)
                for (int32_t c = 0; c < dh; ++c) {
                    double acc = 0.0;
                    for (int64_t j = 0; j < (causal ? i + 1 : n); ++j)
                        acc += load(P, dtype, att_off[b] + (i * H + h) * n + j) *
                               load(v, dtype, (tok_off[b] + j) * ldv + (int64_t)h * dh + c);
                    store(O, dtype, (tok_off[b] + i) * ldo + (int64_t)h * dh + c, acc);
                }
    }
    free(tok_off);
    free(att_off);
}

/* ------------------------------------------------------------------------ */
/* Token-wise operators (the fused-loop linear operators and LayerNorm)       */
/* ------------------------------------------------------------------------ */

static double activation(int act, double x) {
    if (act == OR_ACT_GELU_ERF) return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));
    if (act == OR_ACT_GELU_TANH) {
        const double c = sqrt(2.0 / M_PI);
        return 0.5 * x * (1.0 + tanh(c * (x + 0.044715 * x * x * x)));
    }
    return x;
}

/*
 * Packed-token linear operator (Proj1, Proj2, FF1, FF2 of the layer: Section
 * 7.2 runs them over the fused batch x length loop, i.e. over the T real
 * tokens only):
 *   Y[t][n] = rd(act(sum_k X[t][k] * W[n][k] + bias[n]) + R[t][n])
 * W is [N, K] row-major (y = x W^T + b).  bias and R may be NULL.
 */
void oracle_linear(int dtype, int64_t T, int32_t K, int32_t N, const void* x, int64_t ldx,
                   const void* w, const void* bias, const void* r, int64_t ldr, int act,
                   void* y, int64_t ldy) {
    double* wd = malloc(sizeof(double) * (size_t)N * K);
    double* xd = malloc(sizeof(double) * (size_t)K);
    for (int64_t i = 0; i < (int64_t)N * K; ++i) wd[i] = load(w, dtype, i);
    for (int64_t t = 0; t < T; ++t) {
        for (int32_t k = 0; k < K; ++k) xd[k] = load(x, dtype, t * ldx + k);
        for (int32_t n = 0; n < N; ++n) {
            double acc = 0.0;
            const double* wr = wd + (int64_t)n * K;
            for (int32_t k = 0; k < K; ++k) acc += xd[k] * wr[k];
            if (bias) acc += load(bias, dtype, n);
            acc = activation(act, acc);
            if (r) acc += load(r, dtype, t * ldr + n);
            store(y, dtype, t * ldy + n, acc);
        }
    }
    free(wd);
    free(xd);
}

/* LayerNorm over the d features of every token row: population mean and
 * variance, y = rd(gamma * (x - mean) / sqrt(var + eps) + beta). */
void oracle_layernorm(int dtype, int64_t T, int32_t d, const void* x, int64_t ldx,
                      const void* gamma, const void* beta, double eps, void* y, int64_t ldy) {
    for (int64_t t = 0; t < T; ++t) {
        double mean = 0.0;
        for (int32_t c = 0; c < d; ++c) mean += load(x, dtype, t * ldx + c);
        mean /= d;
        double var = 0.0;
        for (int32_t c = 0; c < d; ++c) {
            double u = load(x, dtype, t * ldx + c) - mean;
            var += u * u;
        }
        var /= d;
        double inv = 1.0 / sqrt(var + eps);
        for (int32_t c = 0; c < d; ++c) {
            double u = (load(x, dtype, t * ldx + c) - mean) * inv;
            store(y, dtype, t * ldy + c, load(gamma, dtype, c) * u + load(beta, dtype, c));
        }
    }
}

/* ------------------------------------------------------------------------ */
/* The encoder layer                                                          */
/* ------------------------------------------------------------------------ */

typedef struct {
    const void *w_qkv, *b_qkv, *w_o, *b_o, *ln1_g, *ln1_b;
    const void *w_ff1, *b_ff1, *w_ff2, *b_ff2, *ln2_g, *ln2_b;
} oracle_layer_weights;

static size_t elem_size(int dtype) { return dtype == OR_F32 ? 4 : 2; }

/*
 * One post-LayerNorm Transformer encoder layer over the packed real tokens,
 * chaining the nine operators of the paper's layer (Section 2, figure comparing
 * the FasterTransformer and CoRa layers; Appendix D, per-operator breakdown
 * table):
 *   QKV = X Wqkv^T + bqkv                     [T, 3d]  (Q | K | V column blocks)
 *   S   = QK^T / sqrt(dh)  per sequence/head  (X[b][i][h][j] layout)
 *   P   = softmax(S)
 *   O   = P V                                 [T, d]   (heads side by side)
 *   Y1  = O Wo^T + bo + X
 *   H1  = LayerNorm1(Y1)
 *   F   = act(H1 W1^T + b1)                   [T, d_ff]
 *   Y2  = F W2^T + b2 + H1
 *   out = LayerNorm2(Y2)
 * With causal != 0 the attention is masked (position i sees keys j <= i), the
 * decoder variant of the layer (Section 7.2; Appendix D, masked SDPA).
 * Every intermediate is rounded to the storage type.  Returns 0, or 1 on
 * allocation failure.
 */
int oracle_encoder_layer(int dtype, int32_t B, const int32_t* L, int32_t d, int32_t H, int32_t d_ff,
                         double ln_eps, int act, int causal, const oracle_layer_weights* w,
                         const void* x, void* out) {
    int64_t T = 0, S2 = 0;
    for (int32_t b = 0; b < B; ++b) {
        T += L[b];
        S2 += (int64_t)L[b] * L[b];
    }
    int32_t dh = d / H;
    size_t es = elem_size(dtype);
    char* qkv = malloc(es * (size_t)(T * 3 * d + 1));
    char* s = malloc(es * (size_t)(S2 * H + 1));
    char* o = malloc(es * (size_t)(T * d + 1));
    char* y1 = malloc(es * (size_t)(T * d + 1));
    char* h1 = malloc(es * (size_t)(T * d + 1));
    char* f = malloc(es * (size_t)(T * d_ff + 1));
    char* y2 = malloc(es * (size_t)(T * d + 1));
    int rc = 0;
    if (!qkv || !s || !o || !y1 || !h1 || !f || !y2) {
        rc = 1;
        goto done;
    }
    oracle_linear(dtype, T, d, 3 * d, x, d, w->w_qkv, w->b_qkv, NULL, 0, OR_ACT_NONE, qkv, 3 * d);
    oracle_qkt(dtype, B, L, H, dh, qkv, 3 * d, qkv + es * d, 3 * d, 1.0 / sqrt((double)dh), causal, s);
    oracle_softmax(dtype, B, L, H, causal, s, s);
    oracle_attn_v(dtype, B, L, H, dh, causal, s, qkv + es * 2 * d, 3 * d, o, d);
    oracle_linear(dtype, T, d, d, o, d, w->w_o, w->b_o, x, d, OR_ACT_NONE, y1, d);
    oracle_layernorm(dtype, T, d, y1, d, w->ln1_g, w->ln1_b, ln_eps, h1, d);
    oracle_linear(dtype, T, d, d_ff, h1, d, w->w_ff1, w->b_ff1, NULL, 0, act, f, d_ff);
    oracle_linear(dtype, T, d_ff, d, f, d_ff, w->w_ff2, w->b_ff2, h1, d, OR_ACT_NONE, y2, d);
    oracle_layernorm(dtype, T, d, y2, d, w->ln2_g, w->ln2_b, ln_eps, out, d);
done:
    free(qkv); free(s); free(o); free(y1); free(h1); free(f); free(y2);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Variable-sized batched GEMM (vgemm, Section 7.1)                           */
/* ------------------------------------------------------------------------ */

/*
 * vgemm: a batch of B independent GEMMs with their own sizes (m_b, n_b, k_b),
 * stored ragged: the problems' matrices are packed one after another, each
 * row-major, and located through exclusive prefix sums of their sizes (the
 * storage of a ragged dimension, Section 5.3 / Appendix B):
 *   a_off[b] = sum_{b' < b} m_b' * k_b'    A_b is [m_b, k_b]
 *   b_off[b] = sum_{b' < b} n_b' * k_b'    B_b is [n_b, k_b] (rows are the
 *                                          output columns, k contiguous)
 *   c_off[b] = sum_{b' < b} m_b' * n_b'    C_b is [m_b, n_b]
 * Work is ordered largest first (Appendix D, load balancing): order[] sorts
 * the problems by m*n*k descending, ties by lower index; tile_off[] is the
 * exclusive prefix sum, in that order, of each problem's
 * ceil(m/tile_m) * ceil(n/tile_n) output tiles.  dims holds (m, n, k) per
 * problem.  Returns 0, or 1 if a size is negative.
 */
int oracle_vgemm_offsets(int32_t B, const int32_t* dims, int32_t tile_m, int32_t tile_n, int64_t* a_off,
                         int64_t* b_off, int64_t* c_off, int32_t* order, int64_t* tile_off) {
    for (int32_t b = 0; b < B; ++b)
        if (dims[3 * b] < 0 || dims[3 * b + 1] < 0 || dims[3 * b + 2] < 0) return 1;
    a_off[0] = b_off[0] = c_off[0] = 0;
    for (int32_t b = 0; b < B; ++b) {
        int64_t m = dims[3 * b], n = dims[3 * b + 1], k = dims[3 * b + 2];
        a_off[b + 1] = a_off[b] + m * k;
        b_off[b + 1] = b_off[b] + n * k;
        c_off[b + 1] = c_off[b] + m * n;
    }
    for (int32_t b = 0; b < B; ++b) order[b] = b;
    for (int32_t i = 1; i < B; ++i) {  /* stable insertion sort, work descending */
        int32_t cur = order[i];
        int64_t wc = (int64_t)dims[3 * cur] * dims[3 * cur + 1] * dims[3 * cur + 2];
        int32_t p = i - 1;
        while (p >= 0 && (int64_t)dims[3 * order[p]] * dims[3 * order[p] + 1] * dims[3 * order[p] + 2] < wc) {
            order[p + 1] = order[p];
            --p;
        }
        order[p + 1] = cur;
    }
    tile_off[0] = 0;
    for (int32_t i = 0; i < B; ++i) {
        int32_t b = order[i];
        tile_off[i + 1] = tile_off[i] + ceil_div(dims[3 * b], tile_m) * ceil_div(dims[3 * b + 1], tile_n);
    }
    return 0;
}

/*
 * vgemm product: for every problem b, C_b[i][j] = rd(sum_k A_b[i][k] * B_b[j][k]),
 * i < m_b, j < n_b, on the packed storage above.
 */
void oracle_vgemm(int dtype, int32_t B, const int32_t* dims, const void* a, const void* bm, void* c) {
    int64_t ao = 0, bo = 0, co = 0;
    for (int32_t p = 0; p < B; ++p) {
        int64_t m = dims[3 * p], n = dims[3 * p + 1], k = dims[3 * p + 2];
        for (int64_t i = 0; i < m; ++i)
            for (int64_t j = 0; j < n; ++j) {
                double acc = 0.0;
                for (int64_t t = 0; t < k; ++t) acc += load(a, dtype, ao + i * k + t) * load(bm, dtype, bo + j * k + t);
                store(c, dtype, co + i * n + j, acc);
            }
        ao += m * k;
        bo += n * k;
        co += m * n;
    }
}

/* ------------------------------------------------------------------------ */
/* Triangular matrix multiplication (trmm, Section 7.1)                      */
/* ------------------------------------------------------------------------ */

/*
 * trmm: a square lower-triangular matrix L (n x n) times a dense matrix B
 * (n x m).  Row i of a triangular matrix holds its nonzeros in columns 0..i,
 * so the reduction over k is a variable loop whose extent depends on the
 * output row (the paper's vloop):
 *   C[i][j] = rd(sum_{k <= i} L[i][k] * B[k][j]),   i < n, j < m.
 * Entries of L above the diagonal are never read.  All three are row-major
 * with leading dimensions ldl, ldb, ldc.
 */
void oracle_trmm(int dtype, int32_t n, int32_t m, const void* l, int64_t ldl, const void* b, int64_t ldb, void* c,
                 int64_t ldc) {
    for (int64_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < m; ++j) {
            double acc = 0.0;
            for (int64_t k = 0; k <= i; ++k) acc += load(l, dtype, i * ldl + k) * load(b, dtype, k * ldb + j);
            store(c, dtype, i * ldc + j, acc);
        }
}

/* The same definition for selected output rows only: row rows[r] of C goes to
 * row r of c (for spot checks of large products). */
void oracle_trmm_rows(int dtype, int32_t m, const void* l, int64_t ldl, const void* b, int64_t ldb,
                      const int32_t* rows, int32_t nrows, void* c, int64_t ldc) {
    for (int32_t r = 0; r < nrows; ++r) {
        const int64_t i = rows[r];
        for (int64_t j = 0; j < m; ++j) {
            double acc = 0.0;
            for (int64_t k = 0; k <= i; ++k) acc += load(l, dtype, i * ldl + k) * load(b, dtype, k * ldb + j);
            store(c, dtype, r * ldc + j, acc);
        }
    }
}
