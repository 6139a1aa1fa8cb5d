// Host-side launchers of the HIP kernels.  Each .hip file defines its kernels
// and the launchers below; api.cpp validates arguments and calls them.  Every
// launcher enqueues work on `stream` and returns the launch error (if any).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ragged.h"

namespace rag {

struct PlanView {
    int32_t batch, total_tokens, max_len, heads;
    int64_t qkt_cap, av_cap;
    const int32_t* lengths;
    int32_t* tok_off;
    int64_t* att_off;
    int32_t* order;
    int32_t* tok_seq;
    int32_t* qkt_item_off;
    int32_t* av_item_off;
    int32_t* qkt_items;
    int32_t* av_items;
    int32_t* status;
};

// Number of compute units of the current device (cached per device).
int device_cu_count();

// Record a formatted message as the thread's last error and return `status`.
rag_status report(rag_status status, const char* fmt, ...);

hipError_t launch_offsets(const PlanView& p, hipStream_t s);

// Attention operators; dtype 0 = fp32, 1 = bf16.  Persistent grids sized from the
// host-side capacities; item counts are read on the device.
// `causal` selects masked attention (position i sees keys j <= i).
hipError_t launch_qkt(const PlanView& p, int dtype, const void* q, int ldq, const void* k, int ldk,
                      float scale, void* scores, int64_t score_cap, bool causal, hipStream_t s);
hipError_t launch_softmax(const PlanView& p, int dtype, const void* scores, void* probs,
                          int64_t score_cap, bool causal, hipStream_t s);
hipError_t launch_attn_v(const PlanView& p, int dtype, const void* probs, int64_t score_cap,
                         const void* v, int ldv, void* out, int ldo, bool causal, hipStream_t s);
hipError_t launch_fused_attention(const PlanView& p, int dtype, const void* q, int ldq, const void* k,
                                  int ldk, const void* v, int ldv, float scale, void* out, int ldo,
                                  bool causal, hipStream_t s);

// With `plan`, the launch also builds that batch's plan (as launch_offsets does):
// bf16 projections of batches up to 256 sequences carry the prelude's
// workgroups behind their tiles, other cases launch the prelude first.
hipError_t launch_linear(int dtype, const void* x, int ldx, const void* w, const void* bias,
                         const void* residual, int ldr, int act, void* y, int ldy, int T, int K, int N,
                         hipStream_t s, const PlanView* plan = nullptr);

// Variable-sized batched GEMM.  VgemmView mirrors rag_vgemm_plan.
struct VgemmView {
    int32_t batch;
    int64_t tile_cap;
    const int32_t* dims;
    int64_t* a_off;
    int64_t* b_off;
    int64_t* c_off;
    int32_t* order;
    int64_t* tile_off;
    int32_t* tile_items;
    int32_t* status;
};

hipError_t launch_vgemm_offsets(const VgemmView& p, hipStream_t s);
hipError_t launch_vgemm(const VgemmView& p, int dtype, const void* a, int64_t a_cap, const void* b, int64_t b_cap,
                        void* c, int64_t c_cap, hipStream_t s);

// C = tril(L) B: L [n, n] (ldl), B and C [n, m] (ldb, ldc).
hipError_t launch_trmm(int dtype, const void* l, int ldl, const void* b, int ldb, void* c, int ldc, int n, int m,
                       hipStream_t s);

hipError_t launch_layernorm(int dtype, const void* x, int ldx, const void* gamma, const void* beta,
                            float eps, void* y, int ldy, int T, int d, hipStream_t s);

}  // namespace rag
