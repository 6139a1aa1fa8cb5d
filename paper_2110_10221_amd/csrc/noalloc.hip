// encoder_layer without a caller-provided workspace, for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid allocation).  The layer's intermediate tensors (QKV /
// FF1 output, Y1 / Y2, attention output / H1, and the score buffer of the
// unfused path) live in one file-scope device array of fixed size instead;
// every kernel is the one encoder_layer runs.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/ragged.h"
#include "launch.h"

namespace {

// Each device the library runs on holds its own copy until the process ends.
static __device__ __align__(256) unsigned char scratch[RAG_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices];
std::once_flag g_scratch_once[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// The array's device address on the current device.  In host code `scratch`
// names a host-side stand-in, never a device address, so the address is taken
// once per device (with that device current) and kept.
hipError_t scratch_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::call_once(g_scratch_once[dev], [dev] {
        void* p = nullptr;
        g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch[dev] = g_scratch_err[dev] == hipSuccess ? p : nullptr;
    });
    if (g_scratch_err[dev] != hipSuccess) return g_scratch_err[dev];
    *out = g_scratch[dev];
    return *out ? hipSuccess : hipErrorInvalidSymbol;
}

}  // namespace

extern "C" rag_status encoder_layer_noalloc(const rag_plan* plan, const void* x, void* y, int32_t d_model,
                                            int32_t heads, int32_t head_dim, int32_t d_ff, float ln_eps,
                                            int32_t act, int32_t flags, const rag_layer_weights* w, int32_t dtype,
                                            void* stream) {
    const char* fn = "encoder_layer_noalloc";
    if (!plan) return rag::report(RAG_ERR_ARG, "%s: plan is NULL", fn);
    size_t need = 0;
    const rag_status st =
        encoder_layer_workspace(plan->total_tokens, plan->max_len, d_model, heads, d_ff, dtype, flags, &need);
    if (st != RAG_OK) return st;
    if (need > (size_t)RAG_NOALLOC_SCRATCH_BYTES)
        return rag::report(RAG_ERR_WORKSPACE, "%s: the layer needs %zu bytes of scratch, above the fixed %zu",
                           fn, need, (size_t)RAG_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    const hipError_t e = scratch_address(&ws);
    if (e != hipSuccess)
        return rag::report(RAG_ERR_HIP, "%s: scratch address: %s", fn, hipGetErrorString(e));
    return encoder_layer(plan, x, y, d_model, heads, head_dim, d_ff, ln_eps, act, flags, w, ws,
                         (size_t)RAG_NOALLOC_SCRATCH_BYTES, dtype, stream, nullptr);
}
