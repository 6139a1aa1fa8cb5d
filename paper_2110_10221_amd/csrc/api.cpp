// C entry points: host-side argument validation, then kernel launches.
// Nothing here allocates device memory; every buffer comes from the caller.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "../../include/ragged.h"
#include "launch.h"

namespace {

thread_local char g_last_error[512] = "";

rag_status fail(rag_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return s;
}

bool sync_check_enabled() {
    static const bool on = [] {
        const char* v = getenv("RAG_SYNC_CHECK");
        return v && v[0] && strcmp(v, "0") != 0;
    }();
    return on;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t elem_size(int32_t dtype) { return dtype == RAG_F32 ? 4 : 2; }

rag_status check_dtype(int32_t dtype, const char* fn) {
    if (dtype != RAG_F32 && dtype != RAG_BF16) return fail(RAG_ERR_DTYPE, "%s: dtype %d is not RAG_F32 or RAG_BF16", fn, dtype);
    return RAG_OK;
}

// After enqueueing: report a launch error; with RAG_SYNC_CHECK also wait and
// report execution errors and the plan's data-error bits.
rag_status finish(hipError_t launch_err, hipStream_t s, const int32_t* status, const char* fn) {
    if (launch_err != hipSuccess)
        return fail(RAG_ERR_HIP, "%s: launch failed: %s", fn, hipGetErrorString(launch_err));
    if (!sync_check_enabled()) return RAG_OK;
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(RAG_ERR_HIP, "%s: execution failed: %s", fn, hipGetErrorString(e));
    if (status) {
        int32_t flags = 0;
        e = hipMemcpy(&flags, status, sizeof(flags), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return fail(RAG_ERR_HIP, "%s: status read failed: %s", fn, hipGetErrorString(e));
        if (flags) return fail(RAG_ERR_DATA, "%s: plan status word reports data errors 0x%x", fn, flags);
    }
    return RAG_OK;
}

// The fused attention kernel addresses a sequence's K and V rows with 32-bit
// byte offsets from the sequence's first row.
bool fused_fits(int64_t max_len, int64_t ld) { return max_len * ld * 2 <= INT32_MAX; }

// The bf16 attention operators address one item's scores (64 query rows of
// heads * max_len values) with 32-bit byte offsets.
bool op_item_fits(int64_t heads, int64_t max_len) { return 64 * heads * max_len * 2 + 64 <= INT32_MAX; }

rag_status view_plan(const rag_plan* p, rag::PlanView& v, const char* fn) {
    if (!p) return fail(RAG_ERR_ARG, "%s: plan is NULL", fn);
    if (p->batch < 1 || p->batch > RAG_MAX_BATCH)
        return fail(RAG_ERR_ARG, "%s: batch %d outside [1, %d]", fn, p->batch, RAG_MAX_BATCH);
    if (p->total_tokens < 0 || p->max_len < 0 || p->heads < 1)
        return fail(RAG_ERR_ARG, "%s: total_tokens %d, max_len %d, heads %d out of range", fn, p->total_tokens,
                    p->max_len, p->heads);
    if (p->qkt_cap < 0 || p->av_cap < 0) return fail(RAG_ERR_ARG, "%s: negative capacity", fn);
    if (p->qkt_cap > INT32_MAX || p->av_cap > INT32_MAX)
        return fail(RAG_ERR_CAPACITY, "%s: work-list capacities must stay below 2^31", fn);
    // H * max_len^2 * batch bounds every attention offset; keep it below 2^62
    if ((double)p->heads * p->max_len * p->max_len * p->batch > 4.0e18)
        return fail(RAG_ERR_SHAPE, "%s: heads * max_len^2 * batch overflows 64-bit offsets", fn);
    if (!p->lengths || !p->tok_off || !p->att_off || !p->order || !p->qkt_item_off || !p->av_item_off ||
        !p->status)
        return fail(RAG_ERR_ARG, "%s: a plan array is NULL", fn);
    if (p->total_tokens > 0 && !p->tok_seq) return fail(RAG_ERR_ARG, "%s: tok_seq is NULL", fn);
    if (p->qkt_cap > 0 && (!p->qkt_items || !aligned(p->qkt_items, 16)))
        return fail(RAG_ERR_ARG, "%s: qkt_items must be non-NULL and 16-byte aligned", fn);
    if (p->av_cap > 0 && !p->av_items) return fail(RAG_ERR_ARG, "%s: av_items is NULL", fn);
    if (!aligned(p->att_off, 8) || !aligned(p->lengths, 4) || !aligned(p->status, 4))
        return fail(RAG_ERR_ARG, "%s: misaligned plan array", fn);
    v = rag::PlanView{p->batch, p->total_tokens, p->max_len, p->heads, p->qkt_cap, p->av_cap,
                      p->lengths, p->tok_off, p->att_off, p->order, p->tok_seq, p->qkt_item_off,
                      p->av_item_off, p->qkt_items, p->av_items, p->status};
    return RAG_OK;
}

// A packed [rows, width] operand with leading dimension ld.
rag_status check_operand(const void* ptr, int64_t ld, int64_t width, int32_t dtype, size_t vec_align,
                         const char* name, const char* fn) {
    if (!ptr) return fail(RAG_ERR_ARG, "%s: %s is NULL", fn, name);
    if (ld < width) return fail(RAG_ERR_SHAPE, "%s: leading dimension of %s (%lld) < width %lld", fn, name,
                                (long long)ld, (long long)width);
    if (dtype == RAG_BF16) {
        if (!aligned(ptr, vec_align) || (ld * 2) % vec_align != 0)
            return fail(RAG_ERR_SHAPE, "%s: %s must be %zu-byte aligned with a leading dimension that keeps rows aligned",
                        fn, name, vec_align);
    } else if (!aligned(ptr, 4)) {
        return fail(RAG_ERR_SHAPE, "%s: %s must be 4-byte aligned", fn, name);
    }
    return RAG_OK;
}

bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
    return na && nb && pa < pb + nb && pb < pa + na;
}

size_t span_bytes(int64_t rows, int64_t ld, int64_t width, int32_t dtype) {
    return rows > 0 ? (size_t)((rows - 1) * ld + width) * elem_size(dtype) : 0;
}

int g_cu_cache[64];

}  // namespace

namespace rag {

rag_status report(rag_status status, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return status;
}

int device_cu_count() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
    if (dev < 64 && g_cu_cache[dev] > 0) return g_cu_cache[dev];
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    if (dev < 64) g_cu_cache[dev] = n;
    return n;
}

}  // namespace rag

extern "C" {

const char* ragged_status_string(rag_status s) {
    switch (s) {
        case RAG_OK: return "RAG_OK";
        case RAG_ERR_ARG: return "RAG_ERR_ARG";
        case RAG_ERR_DTYPE: return "RAG_ERR_DTYPE";
        case RAG_ERR_SHAPE: return "RAG_ERR_SHAPE";
        case RAG_ERR_CAPACITY: return "RAG_ERR_CAPACITY";
        case RAG_ERR_WORKSPACE: return "RAG_ERR_WORKSPACE";
        case RAG_ERR_HIP: return "RAG_ERR_HIP";
        case RAG_ERR_DATA: return "RAG_ERR_DATA";
        default: return "RAG_ERR_UNKNOWN";
    }
}

const char* ragged_last_error(void) { return g_last_error; }

rag_status ragged_plan_capacity(int32_t batch, int32_t total_tokens, int32_t max_len, int32_t heads,
                                int64_t* qkt_cap, int64_t* av_cap) {
    const char* fn = "ragged_plan_capacity";
    if (!qkt_cap || !av_cap) return fail(RAG_ERR_ARG, "%s: output pointer is NULL", fn);
    if (batch < 1 || batch > RAG_MAX_BATCH || total_tokens < 0 || max_len < 0 || heads < 1)
        return fail(RAG_ERR_ARG, "%s: sizes out of range", fn);
    const int64_t nt_max = ((int64_t)max_len + RAG_TILE - 1) / RAG_TILE;
    const int64_t by_len = (int64_t)batch * nt_max;
    const int64_t by_tok = ((int64_t)total_tokens + (int64_t)(RAG_TILE - 1) * batch) / RAG_TILE;
    const int64_t av = (int64_t)heads * (by_len < by_tok ? by_len : by_tok);
    *av_cap = av;
    *qkt_cap = nt_max * av;
    return RAG_OK;
}

rag_status ragged_offsets(rag_plan* plan, void* stream) {
    const char* fn = "ragged_offsets";
    rag::PlanView v;
    rag_status st = view_plan(plan, v, fn);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_offsets(v, s), s, plan->status, fn);
}

namespace {

rag_status qkt_impl(const rag_plan* plan, const void* q, int32_t ldq, const void* k, int32_t ldk, int32_t head_dim,
                    float scale, void* scores, int64_t score_cap, int32_t dtype, void* stream, bool causal,
                    const char* fn) {
    rag::PlanView v;
    rag_status st;
    if ((st = view_plan(plan, v, fn)) || (st = check_dtype(dtype, fn))) return st;
    if (head_dim != RAG_HEAD_DIM) return fail(RAG_ERR_SHAPE, "%s: head_dim %d unsupported (only %d)", fn, head_dim, RAG_HEAD_DIM);
    const int64_t width = (int64_t)plan->heads * head_dim;
    if ((st = check_operand(q, ldq, width, dtype, 16, "q", fn)) || (st = check_operand(k, ldk, width, dtype, 16, "k", fn)))
        return st;
    if (!std::isfinite(scale)) return fail(RAG_ERR_ARG, "%s: scale is not finite", fn);
    if (!scores || score_cap < 0) return fail(RAG_ERR_ARG, "%s: scores is NULL or score_cap < 0", fn);
    if (dtype == RAG_BF16 && !op_item_fits(plan->heads, plan->max_len))
        return fail(RAG_ERR_SHAPE, "%s: 64 * heads * max_len * 2 bytes exceeds 32-bit item offsets", fn);
    if (!aligned(scores, elem_size(dtype))) return fail(RAG_ERR_ARG, "%s: scores misaligned", fn);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_qkt(v, dtype, q, ldq, k, ldk, scale, scores, score_cap, causal, s), s, plan->status, fn);
}

rag_status softmax_impl(const rag_plan* plan, const void* scores, void* probs, int64_t score_cap, int32_t dtype,
                        void* stream, bool causal, const char* fn) {
    rag::PlanView v;
    rag_status st;
    if ((st = view_plan(plan, v, fn)) || (st = check_dtype(dtype, fn))) return st;
    if (!scores || !probs || score_cap < 0) return fail(RAG_ERR_ARG, "%s: scores/probs NULL or score_cap < 0", fn);
    if (dtype == RAG_BF16 && (int64_t)plan->heads * plan->max_len * 2 + 64 > INT32_MAX)
        return fail(RAG_ERR_SHAPE, "%s: heads * max_len * 2 bytes exceeds 32-bit row offsets", fn);
    if (!aligned(scores, elem_size(dtype)) || !aligned(probs, elem_size(dtype)))
        return fail(RAG_ERR_ARG, "%s: scores/probs misaligned", fn);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_softmax(v, dtype, scores, probs, score_cap, causal, s), s, plan->status, fn);
}

rag_status attn_v_impl(const rag_plan* plan, const void* probs, int64_t score_cap, const void* vv, int32_t ldv,
                       int32_t head_dim, void* out, int32_t ldo, int32_t dtype, void* stream, bool causal,
                       const char* fn) {
    rag::PlanView v;
    rag_status st;
    if ((st = view_plan(plan, v, fn)) || (st = check_dtype(dtype, fn))) return st;
    if (head_dim != RAG_HEAD_DIM) return fail(RAG_ERR_SHAPE, "%s: head_dim %d unsupported (only %d)", fn, head_dim, RAG_HEAD_DIM);
    const int64_t width = (int64_t)plan->heads * head_dim;
    if ((st = check_operand(vv, ldv, width, dtype, 16, "v", fn)) || (st = check_operand(out, ldo, width, dtype, 16, "out", fn)))
        return st;
    if (!probs || score_cap < 0) return fail(RAG_ERR_ARG, "%s: probs is NULL or score_cap < 0", fn);
    if (!aligned(probs, elem_size(dtype))) return fail(RAG_ERR_ARG, "%s: probs misaligned", fn);
    if (dtype == RAG_BF16 && !op_item_fits(plan->heads, plan->max_len))
        return fail(RAG_ERR_SHAPE, "%s: 64 * heads * max_len * 2 bytes exceeds 32-bit item offsets", fn);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_attn_v(v, dtype, probs, score_cap, vv, ldv, out, ldo, causal, s), s, plan->status, fn);
}

rag_status attention_impl(const rag_plan* plan, const void* q, int32_t ldq, const void* k, int32_t ldk,
                          const void* vv, int32_t ldv, int32_t head_dim, float scale, void* out, int32_t ldo,
                          int32_t dtype, void* stream, bool causal, const char* fn) {
    rag::PlanView v;
    rag_status st;
    if ((st = view_plan(plan, v, fn)) || (st = check_dtype(dtype, fn))) return st;
    if (dtype != RAG_BF16) return fail(RAG_ERR_DTYPE, "%s: the fused kernel is bf16 only", fn);
    if (head_dim != RAG_HEAD_DIM) return fail(RAG_ERR_SHAPE, "%s: head_dim %d unsupported (only %d)", fn, head_dim, RAG_HEAD_DIM);
    const int64_t width = (int64_t)plan->heads * head_dim;
    if ((st = check_operand(q, ldq, width, dtype, 16, "q", fn)) || (st = check_operand(k, ldk, width, dtype, 16, "k", fn)) ||
        (st = check_operand(vv, ldv, width, dtype, 16, "v", fn)) || (st = check_operand(out, ldo, width, dtype, 16, "out", fn)))
        return st;
    if (!std::isfinite(scale)) return fail(RAG_ERR_ARG, "%s: scale is not finite", fn);
    if (!fused_fits(plan->max_len, ldk > ldv ? ldk : ldv))
        return fail(RAG_ERR_SHAPE, "%s: max_len %d rows of leading dimension %d exceed the kernel's 32-bit offsets", fn,
                    plan->max_len, ldk > ldv ? ldk : ldv);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_fused_attention(v, dtype, q, ldq, k, ldk, vv, ldv, scale, out, ldo, causal, s), s,
                  plan->status, fn);
}

}  // namespace

rag_status ragged_qkt(const rag_plan* plan, const void* q, int32_t ldq, const void* k, int32_t ldk,
                      int32_t head_dim, float scale, void* scores, int64_t score_cap, int32_t dtype,
                      void* stream) {
    return qkt_impl(plan, q, ldq, k, ldk, head_dim, scale, scores, score_cap, dtype, stream, false, "ragged_qkt");
}

rag_status ragged_qkt_causal(const rag_plan* plan, const void* q, int32_t ldq, const void* k, int32_t ldk,
                             int32_t head_dim, float scale, void* scores, int64_t score_cap, int32_t dtype,
                             void* stream) {
    return qkt_impl(plan, q, ldq, k, ldk, head_dim, scale, scores, score_cap, dtype, stream, true,
                    "ragged_qkt_causal");
}

rag_status ragged_softmax(const rag_plan* plan, const void* scores, void* probs, int64_t score_cap, int32_t dtype,
                          void* stream) {
    return softmax_impl(plan, scores, probs, score_cap, dtype, stream, false, "ragged_softmax");
}

rag_status ragged_softmax_causal(const rag_plan* plan, const void* scores, void* probs, int64_t score_cap,
                                 int32_t dtype, void* stream) {
    return softmax_impl(plan, scores, probs, score_cap, dtype, stream, true, "ragged_softmax_causal");
}

rag_status ragged_attn_v(const rag_plan* plan, const void* probs, int64_t score_cap, const void* vv, int32_t ldv,
                         int32_t head_dim, void* out, int32_t ldo, int32_t dtype, void* stream) {
    return attn_v_impl(plan, probs, score_cap, vv, ldv, head_dim, out, ldo, dtype, stream, false, "ragged_attn_v");
}

rag_status ragged_attn_v_causal(const rag_plan* plan, const void* probs, int64_t score_cap, const void* vv,
                                int32_t ldv, int32_t head_dim, void* out, int32_t ldo, int32_t dtype,
                                void* stream) {
    return attn_v_impl(plan, probs, score_cap, vv, ldv, head_dim, out, ldo, dtype, stream, true,
                       "ragged_attn_v_causal");
}

rag_status ragged_attention(const rag_plan* plan, const void* q, int32_t ldq, const void* k, int32_t ldk,
                            const void* vv, int32_t ldv, int32_t head_dim, float scale, void* out, int32_t ldo,
                            int32_t dtype, void* stream) {
    return attention_impl(plan, q, ldq, k, ldk, vv, ldv, head_dim, scale, out, ldo, dtype, stream, false,
                          "ragged_attention");
}

rag_status ragged_attention_causal(const rag_plan* plan, const void* q, int32_t ldq, const void* k, int32_t ldk,
                                   const void* vv, int32_t ldv, int32_t head_dim, float scale, void* out,
                                   int32_t ldo, int32_t dtype, void* stream) {
    return attention_impl(plan, q, ldq, k, ldk, vv, ldv, head_dim, scale, out, ldo, dtype, stream, true,
                          "ragged_attention_causal");
}

namespace {

rag_status check_linear(const void* x, int32_t ldx, const void* w, const void* bias, const void* residual,
                        int32_t ldr, int32_t act, const void* y, int32_t ldy, int32_t T, int32_t K, int32_t N,
                        int32_t dtype, const char* fn) {
    rag_status st;
    if ((st = check_dtype(dtype, fn))) return st;
    if (T < 0 || K < 1 || N < 1) return fail(RAG_ERR_ARG, "%s: T %d, K %d, N %d out of range", fn, T, K, N);
    if (act < RAG_ACT_NONE || act > RAG_ACT_GELU_TANH) return fail(RAG_ERR_ARG, "%s: bad activation %d", fn, act);
    if (dtype == RAG_BF16 && (K % 64 != 0 || N % 64 != 0))
        return fail(RAG_ERR_SHAPE, "%s: bf16 needs K %% 64 == 0 and N %% 64 == 0 (K %d, N %d)", fn, K, N);
    if (T == 0) return RAG_OK;  // nothing is read or written
    if ((st = check_operand(x, ldx, K, dtype, 16, "x", fn)) || (st = check_operand(w, K, K, dtype, 16, "w", fn)) ||
        (st = check_operand(y, ldy, N, dtype, 16, "y", fn)))
        return st;
    if (residual && (st = check_operand(residual, ldr, N, dtype, 16, "residual", fn))) return st;
    if (bias && !aligned(bias, dtype == RAG_BF16 ? 8 : 4)) return fail(RAG_ERR_SHAPE, "%s: bias misaligned", fn);
    const size_t ys = span_bytes(T, ldy, N, dtype);
    if (ranges_overlap(y, ys, x, span_bytes(T, ldx, K, dtype)) ||
        ranges_overlap(y, ys, w, span_bytes(N, K, K, dtype)))
        return fail(RAG_ERR_ARG, "%s: y overlaps x or w", fn);
    if (residual && residual != y && ranges_overlap(y, ys, residual, span_bytes(T, ldr, N, dtype)))
        return fail(RAG_ERR_ARG, "%s: residual partially overlaps y", fn);
    if (residual == y && ldr != ldy) return fail(RAG_ERR_ARG, "%s: in-place residual needs ldr == ldy", fn);
    return RAG_OK;
}

rag_status check_layernorm(const void* x, int32_t ldx, const void* g, const void* b, const void* y, int32_t ldy,
                           int32_t T, int32_t d, int32_t dtype, const char* fn) {
    rag_status st;
    if ((st = check_dtype(dtype, fn))) return st;
    if (T < 0 || d < 1) return fail(RAG_ERR_ARG, "%s: T %d, d %d out of range", fn, T, d);
    const int per = dtype == RAG_BF16 ? 8 : 4;
    if (d % per != 0 || d > 4096) return fail(RAG_ERR_SHAPE, "%s: d %d must be a multiple of %d and <= 4096", fn, d, per);
    if (T == 0) return RAG_OK;  // nothing is read or written
    if ((st = check_operand(x, ldx, d, dtype, 16, "x", fn)) || (st = check_operand(y, ldy, d, dtype, 16, "y", fn)))
        return st;
    if (dtype == RAG_F32 && (!aligned(x, 16) || !aligned(y, 16) || ldx % 4 || ldy % 4))
        return fail(RAG_ERR_SHAPE, "%s: fp32 rows must be 16-byte aligned", fn);
    if (!g || !b || !aligned(g, 16) || !aligned(b, 16)) return fail(RAG_ERR_ARG, "%s: gamma/beta NULL or misaligned", fn);
    if (x != y && ranges_overlap(y, span_bytes(T, ldy, d, dtype), x, span_bytes(T, ldx, d, dtype)))
        return fail(RAG_ERR_ARG, "%s: y partially overlaps x", fn);
    if (x == y && ldx != ldy) return fail(RAG_ERR_ARG, "%s: in-place use needs ldx == ldy", fn);
    return RAG_OK;
}

}  // namespace

rag_status packed_linear(const void* x, int32_t ldx, const void* w, const void* bias, const void* residual,
                         int32_t ldr, int32_t act, void* y, int32_t ldy, int32_t T, int32_t K, int32_t N,
                         int32_t dtype, void* stream) {
    const char* fn = "packed_linear";
    rag_status st = check_linear(x, ldx, w, bias, residual, ldr, act, y, ldy, T, K, N, dtype, fn);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_linear(dtype, x, ldx, w, bias, residual, ldr, act, y, ldy, T, K, N, s), s, nullptr, fn);
}

rag_status packed_layernorm(const void* x, int32_t ldx, const void* gamma, const void* beta, float eps, void* y,
                            int32_t ldy, int32_t T, int32_t d, int32_t dtype, void* stream) {
    const char* fn = "packed_layernorm";
    rag_status st = check_layernorm(x, ldx, gamma, beta, y, ldy, T, d, dtype, fn);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_layernorm(dtype, x, ldx, gamma, beta, eps, y, ldy, T, d, s), s, nullptr, fn);
}

namespace {

constexpr size_t kAlign = 256;
size_t round_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// The fused attention kernel exists for bf16 (and sequences whose K / V rows its
// 32-bit offsets reach); other layers run the three attention operators over a
// materialised score buffer.  The layer's Q, K and V are column blocks of one
// [T, 3d] buffer.
bool unfused_attention(int32_t dtype, int32_t flags, int64_t max_len, int64_t d) {
    return (flags & RAG_LAYER_UNFUSED_ATTENTION) || dtype == RAG_F32 || !fused_fits(max_len, 3 * d);
}

struct LayerBuffers {
    size_t qkvf, act_a, h1o, scores, total;
};

LayerBuffers layer_buffers(int64_t T, int64_t max_len, int64_t d, int64_t H, int64_t d_ff, int32_t dtype,
                           int32_t flags) {
    const size_t es = elem_size(dtype);
    LayerBuffers lb{};
    lb.qkvf = round_up((size_t)T * (size_t)(3 * d > d_ff ? 3 * d : d_ff) * es);  // QKV, later FF1 output
    lb.act_a = round_up((size_t)T * d * es);                                     // Y1, later Y2
    lb.h1o = round_up((size_t)T * d * es);                                       // attention output, later H1
    lb.scores = unfused_attention(dtype, flags, max_len, d) ? round_up((size_t)H * T * max_len * es) : 0;
    lb.total = lb.qkvf + lb.act_a + lb.h1o + lb.scores;
    return lb;
}

}  // namespace

rag_status encoder_layer_workspace(int32_t total_tokens, int32_t max_len, int32_t d_model, int32_t heads,
                                   int32_t d_ff, int32_t dtype, int32_t flags, size_t* bytes) {
    const char* fn = "encoder_layer_workspace";
    rag_status st;
    if ((st = check_dtype(dtype, fn))) return st;
    if (!bytes) return fail(RAG_ERR_ARG, "%s: bytes is NULL", fn);
    if (total_tokens < 0 || max_len < 0 || d_model < 1 || heads < 1 || d_ff < 1)
        return fail(RAG_ERR_ARG, "%s: sizes out of range", fn);
    *bytes = layer_buffers(total_tokens, max_len, d_model, heads, d_ff, dtype, flags).total;
    return RAG_OK;
}

rag_status encoder_layer(const rag_plan* plan, const void* x, void* y, int32_t d_model, int32_t heads,
                         int32_t head_dim, int32_t d_ff, float ln_eps, int32_t act, int32_t flags,
                         const rag_layer_weights* w, void* workspace, size_t workspace_bytes, int32_t dtype,
                         void* stream, void* const* events) {
    const char* fn = "encoder_layer";
    rag::PlanView v;
    rag_status st;
    if ((st = view_plan(plan, v, fn)) || (st = check_dtype(dtype, fn))) return st;
    if (!w) return fail(RAG_ERR_ARG, "%s: weights is NULL", fn);
    if (heads != plan->heads) return fail(RAG_ERR_SHAPE, "%s: heads %d differs from the plan's %d", fn, heads, plan->heads);
    if (head_dim != RAG_HEAD_DIM) return fail(RAG_ERR_SHAPE, "%s: head_dim %d unsupported (only %d)", fn, head_dim, RAG_HEAD_DIM);
    if (d_model != heads * head_dim) return fail(RAG_ERR_SHAPE, "%s: d_model %d != heads * head_dim", fn, d_model);
    if (flags & ~(RAG_LAYER_UNFUSED_ATTENTION | RAG_LAYER_CAUSAL | RAG_LAYER_BUILD_PLAN))
        return fail(RAG_ERR_ARG, "%s: unknown flags 0x%x", fn, flags);
    const int T = plan->total_tokens, d = d_model;
    if (dtype == RAG_BF16 && unfused_attention(dtype, flags, plan->max_len, d) && !op_item_fits(heads, plan->max_len))
        return fail(RAG_ERR_SHAPE, "%s: 64 * heads * max_len * 2 bytes exceeds 32-bit item offsets", fn);
    const LayerBuffers lb = layer_buffers(T, plan->max_len, d, heads, d_ff, dtype, flags);
    if (!workspace || workspace_bytes < lb.total)
        return fail(RAG_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", fn, workspace_bytes, lb.total);
    if (!aligned(workspace, kAlign)) return fail(RAG_ERR_WORKSPACE, "%s: workspace must be %zu-byte aligned", fn, kAlign);
    char* ws = static_cast<char*>(workspace);
    void* qkv = ws;                      // [T, 3d], later F [T, d_ff]
    void* act_a = ws + lb.qkvf;          // Y1, later Y2
    void* h1o = ws + lb.qkvf + lb.act_a;  // attention output O, later H1
    void* scores = ws + lb.qkvf + lb.act_a + lb.h1o;
    const size_t es = elem_size(dtype);
    const char* qkvc = static_cast<const char*>(qkv);
    // every token-wise step is validated up front, so nothing is launched unless all are valid
    if ((st = check_linear(x, d, w->w_qkv, w->b_qkv, nullptr, 0, RAG_ACT_NONE, qkv, 3 * d, T, d, 3 * d, dtype, fn)) ||
        (st = check_linear(h1o, d, w->w_o, w->b_o, x, d, RAG_ACT_NONE, act_a, d, T, d, d, dtype, fn)) ||
        (st = check_layernorm(act_a, d, w->ln1_g, w->ln1_b, h1o, d, T, d, dtype, fn)) ||
        (st = check_linear(h1o, d, w->w_ff1, w->b_ff1, nullptr, 0, act, qkv, d_ff, T, d, d_ff, dtype, fn)) ||
        (st = check_linear(qkv, d_ff, w->w_ff2, w->b_ff2, h1o, d, RAG_ACT_NONE, act_a, d, T, d_ff, d, dtype, fn)) ||
        (st = check_layernorm(act_a, d, w->ln2_g, w->ln2_b, y, d, T, d, dtype, fn)))
        return st;
    if (ranges_overlap(x, span_bytes(T, d, d, dtype), y, span_bytes(T, d, d, dtype)))
        return fail(RAG_ERR_ARG, "%s: x and y overlap", fn);
    if (ranges_overlap(ws, lb.total, x, span_bytes(T, d, d, dtype)) ||
        ranges_overlap(ws, lb.total, y, span_bytes(T, d, d, dtype)))
        return fail(RAG_ERR_ARG, "%s: workspace overlaps x or y", fn);

    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipSuccess;
    auto mark = [&](int k) {
        if (events && e == hipSuccess) e = hipEventRecord(static_cast<hipEvent_t>(events[k]), s);
    };
    auto run = [&](hipError_t r) {
        if (e == hipSuccess) e = r;
    };
    const float scale = 1.0f / sqrtf((float)head_dim);
    const bool causal = (flags & RAG_LAYER_CAUSAL) != 0;
    mark(0);
    run(rag::launch_linear(dtype, x, d, w->w_qkv, w->b_qkv, nullptr, 0, RAG_ACT_NONE, qkv, 3 * d, T, d, 3 * d, s,
                           (flags & RAG_LAYER_BUILD_PLAN) ? &v : nullptr));
    mark(1);
    if (unfused_attention(dtype, flags, plan->max_len, d)) {
        const int64_t cap = (int64_t)(lb.scores / es);
        run(rag::launch_qkt(v, dtype, qkvc, 3 * d, qkvc + es * d, 3 * d, scale, scores, cap, causal, s));
        mark(2);
        run(rag::launch_softmax(v, dtype, scores, scores, cap, causal, s));
        mark(3);
        run(rag::launch_attn_v(v, dtype, scores, cap, qkvc + 2 * es * d, 3 * d, h1o, d, causal, s));
    } else {
        mark(2);
        mark(3);
        run(rag::launch_fused_attention(v, dtype, qkvc, 3 * d, qkvc + es * d, 3 * d, qkvc + 2 * es * d, 3 * d, scale,
                                        h1o, d, causal, s));
    }
    mark(4);
    run(rag::launch_linear(dtype, h1o, d, w->w_o, w->b_o, x, d, RAG_ACT_NONE, act_a, d, T, d, d, s));
    mark(5);
    run(rag::launch_layernorm(dtype, act_a, d, w->ln1_g, w->ln1_b, ln_eps, h1o, d, T, d, s));
    mark(6);
    run(rag::launch_linear(dtype, h1o, d, w->w_ff1, w->b_ff1, nullptr, 0, act, qkv, d_ff, T, d, d_ff, s));
    mark(7);
    run(rag::launch_linear(dtype, qkv, d_ff, w->w_ff2, w->b_ff2, h1o, d, RAG_ACT_NONE, act_a, d, T, d_ff, d, s));
    mark(8);
    run(rag::launch_layernorm(dtype, act_a, d, w->ln2_g, w->ln2_b, ln_eps, y, d, T, d, s));
    mark(9);
    return finish(e, s, plan->status, fn);
}

namespace {

rag_status view_vgemm_plan(const rag_vgemm_plan* p, rag::VgemmView& v, const char* fn) {
    if (!p) return fail(RAG_ERR_ARG, "%s: plan is NULL", fn);
    if (p->batch < 1 || p->batch > RAG_VGEMM_MAX_BATCH)
        return fail(RAG_ERR_ARG, "%s: batch %d outside [1, %d]", fn, p->batch, RAG_VGEMM_MAX_BATCH);
    if (p->tile_cap < 0) return fail(RAG_ERR_ARG, "%s: negative tile_cap", fn);
    if (p->tile_cap > RAG_VGEMM_MAX_TILES)
        return fail(RAG_ERR_CAPACITY, "%s: tile_cap %lld exceeds %d", fn, (long long)p->tile_cap, RAG_VGEMM_MAX_TILES);
    if (!p->dims || !p->a_off || !p->b_off || !p->c_off || !p->order || !p->tile_off || !p->status)
        return fail(RAG_ERR_ARG, "%s: a plan array is NULL", fn);
    if (p->tile_cap > 0 && (!p->tile_items || !aligned(p->tile_items, 16)))
        return fail(RAG_ERR_ARG, "%s: tile_items must be non-NULL and 16-byte aligned", fn);
    if (!aligned(p->dims, 4) || !aligned(p->a_off, 8) || !aligned(p->b_off, 8) || !aligned(p->c_off, 8) ||
        !aligned(p->order, 4) || !aligned(p->tile_off, 8) || !aligned(p->status, 4))
        return fail(RAG_ERR_ARG, "%s: misaligned plan array", fn);
    v = rag::VgemmView{p->batch, p->tile_cap, p->dims, p->a_off, p->b_off, p->c_off, p->order,
                       p->tile_off, p->tile_items, p->status};
    return RAG_OK;
}

}  // namespace

rag_status vgemm_plan_capacity(int32_t batch, int32_t max_m, int32_t max_n, int64_t* tile_cap) {
    const char* fn = "vgemm_plan_capacity";
    if (!tile_cap) return fail(RAG_ERR_ARG, "%s: output pointer is NULL", fn);
    if (batch < 1 || batch > RAG_VGEMM_MAX_BATCH || max_m < 0 || max_n < 0 || max_m > RAG_VGEMM_MAX_DIM ||
        max_n > RAG_VGEMM_MAX_DIM)
        return fail(RAG_ERR_ARG, "%s: sizes out of range", fn);
    *tile_cap = (int64_t)batch * ((max_m + RAG_VGEMM_TILE_M - 1) / RAG_VGEMM_TILE_M) *
                ((max_n + RAG_VGEMM_TILE_N - 1) / RAG_VGEMM_TILE_N);
    return RAG_OK;
}

rag_status vgemm_tile_count(int32_t batch, const int32_t* dims, int64_t* tiles) {
    const char* fn = "vgemm_tile_count";
    if (!dims || !tiles) return fail(RAG_ERR_ARG, "%s: dims or tiles is NULL", fn);
    if (batch < 1 || batch > RAG_VGEMM_MAX_BATCH)
        return fail(RAG_ERR_ARG, "%s: batch %d outside [1, %d]", fn, batch, RAG_VGEMM_MAX_BATCH);
    int64_t n = 0;
    for (int32_t p = 0; p < batch; ++p) {
        const int32_t m = dims[3 * p], nn = dims[3 * p + 1], k = dims[3 * p + 2];
        if (m < 0 || nn < 0 || k < 0 || m > RAG_VGEMM_MAX_DIM || nn > RAG_VGEMM_MAX_DIM || k > RAG_VGEMM_MAX_DIM)
            return fail(RAG_ERR_ARG, "%s: problem %d has sizes (%d, %d, %d) outside [0, %d]", fn, p, m, nn, k,
                        RAG_VGEMM_MAX_DIM);
        n += (int64_t)((m + RAG_VGEMM_TILE_M - 1) / RAG_VGEMM_TILE_M) * ((nn + RAG_VGEMM_TILE_N - 1) / RAG_VGEMM_TILE_N);
    }
    *tiles = n;
    return RAG_OK;
}

rag_status vgemm_offsets(rag_vgemm_plan* plan, void* stream) {
    const char* fn = "vgemm_offsets";
    rag::VgemmView v;
    rag_status st = view_vgemm_plan(plan, v, fn);
    if (st) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_vgemm_offsets(v, s), s, plan->status, fn);
}

rag_status ragged_vgemm(const rag_vgemm_plan* plan, const void* a, int64_t a_cap, const void* b, int64_t b_cap,
                        void* c, int64_t c_cap, int32_t dtype, void* stream) {
    const char* fn = "ragged_vgemm";
    rag::VgemmView v;
    rag_status st;
    if ((st = view_vgemm_plan(plan, v, fn)) || (st = check_dtype(dtype, fn))) return st;
    if (a_cap < 0 || b_cap < 0 || c_cap < 0) return fail(RAG_ERR_ARG, "%s: negative operand capacity", fn);
    if ((a_cap && !a) || (b_cap && !b) || (c_cap && !c)) return fail(RAG_ERR_ARG, "%s: a, b or c is NULL", fn);
    const size_t align = dtype == RAG_BF16 ? 16 : 4;
    if (!aligned(a, align) || !aligned(b, align) || !aligned(c, align))
        return fail(RAG_ERR_SHAPE, "%s: a, b and c must be %zu-byte aligned", fn, align);
    const size_t es = elem_size(dtype);
    if (ranges_overlap(c, c_cap * es, a, a_cap * es) || ranges_overlap(c, c_cap * es, b, b_cap * es))
        return fail(RAG_ERR_ARG, "%s: c overlaps a or b", fn);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_vgemm(v, dtype, a, a_cap, b, b_cap, c, c_cap, s), s, plan->status, fn);
}

rag_status ragged_trmm(const void* l, int32_t ldl, const void* b, int32_t ldb, void* c, int32_t ldc, int32_t n,
                       int32_t m, int32_t dtype, void* stream) {
    const char* fn = "ragged_trmm";
    rag_status st;
    if ((st = check_dtype(dtype, fn))) return st;
    if (n < 0 || m < 0) return fail(RAG_ERR_ARG, "%s: negative size (n %d, m %d)", fn, n, m);
    if (n == 0 || m == 0) return RAG_OK;
    if ((st = check_operand(l, ldl, n, dtype, 16, "L", fn)) || (st = check_operand(b, ldb, m, dtype, 16, "B", fn)) ||
        (st = check_operand(c, ldc, m, dtype, 16, "C", fn)))
        return st;
    if (dtype == RAG_BF16) {
        if (m % 8 != 0) return fail(RAG_ERR_SHAPE, "%s: bf16 needs m %% 8 == 0 (m = %d)", fn, m);
        // 32-bit buffer offsets: B rows up to n rounded to 64, 128-row panels of L
        if ((int64_t)(n + 64) * ldb >= (int64_t)1 << 30 || ldl >= 1 << 23)
            return fail(RAG_ERR_SHAPE, "%s: bf16 needs (n + 64) * ldb < 2^30 and ldl < 2^23", fn);
    }
    const size_t lc = span_bytes(n, ldc, m, dtype);
    if (ranges_overlap(c, lc, l, span_bytes(n, ldl, n, dtype)) || ranges_overlap(c, lc, b, span_bytes(n, ldb, m, dtype)))
        return fail(RAG_ERR_ARG, "%s: C overlaps L or B", fn);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return finish(rag::launch_trmm(dtype, l, ldl, b, ldb, c, ldc, n, m, s), s, nullptr, fn);
}

}  // extern "C"
