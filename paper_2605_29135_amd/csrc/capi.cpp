// capi.cpp -- C entry points for routing, the expert FFN and combine; error and
// device-flag handling shared by the whole library.
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>

#include "internal.h"
#include "../../include/moe_budget.h"

namespace moe {

namespace {
thread_local std::string g_error;

constexpr int kMaxDevices = 64;
std::mutex g_dev_mu;
int *g_flags[kMaxDevices] = {};
}  // namespace

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
    return code;
}

int fail_hip(hipError_t e, const char *what) {
    return fail(MOE_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), int(e));
}

void clear_error() { g_error.clear(); }

int *device_error_flags() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_dev_mu);
    if (!g_flags[dev]) {
        int *p = nullptr;
        if (hipMalloc(&p, 256) != hipSuccess) return nullptr;
        if (hipMemset(p, 0, 256) != hipSuccess) {
            (void)hipFree(p);
            return nullptr;
        }
        g_flags[dev] = p;
    }
    return g_flags[dev];
}

int *device_error_flags_ready() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_dev_mu);
    return g_flags[dev];
}

}  // namespace moe

using moe::fail;
using moe::fail_hip;

namespace {

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int finish_launch(hipError_t e, const char *what) {
    if (e != hipSuccess) return fail_hip(e, what);
    moe::clear_error();
    return MOE_OK;
}

}  // namespace

extern "C" {

int moe_init(int device) {
    hipError_t e = hipSetDevice(device);
    if (e != hipSuccess) return fail_hip(e, "hipSetDevice");
    if (!moe::device_error_flags()) return fail(MOE_ERR_HIP, "allocating device error flags failed");
    const int st = moe::noalloc_scratch_setup();
    if (st != MOE_OK) return st;
    moe::clear_error();
    return MOE_OK;
}

const char *moe_last_error(void) { return moe::g_error.c_str(); }

int moe_sync_check(void *stream) {
    hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
    int *flags = moe::device_error_flags();
    if (!flags) return fail(MOE_ERR_HIP, "device error flags unavailable");
    int v = 0;
    if ((e = hipMemcpy(&v, flags, sizeof v, hipMemcpyDeviceToHost)) != hipSuccess)
        return fail_hip(e, "reading device error flags");
    if (v) {
        if ((e = hipMemset(flags, 0, sizeof v)) != hipSuccess) return fail_hip(e, "clearing device error flags");
        if (v & moe::kErrRange) return fail(MOE_ERR_RANGE, "an expert id was outside [0, E)");
        if (v & moe::kErrNonfinite) return fail(MOE_ERR_NONFINITE, "a router logit was NaN or infinite");
        if (v & moe::kErrNotResident) return fail(MOE_ERR_NOT_RESIDENT, "an expert had no slot");
        if (v & moe::kErrBudget) return fail(MOE_ERR_BUDGET, "a device lookup needed more experts than slots");
    }
    moe::clear_error();
    return MOE_OK;
}

int moe_route_topk(const float *x, const void *w_router, int w_dtype, int T, int H, int E, int k,
                   const float *logit_bias, float *logits, int32_t *ids, float *weights, int flags,
                   float *x_norm, void *stream) {
    if (T < 0 || E < 1 || E > MOE_MAX_EXPERTS || k < 1 || k > E || k > MOE_MAX_TOPK)
        return fail(MOE_ERR_INVALID_ARG, "route: need T >= 0, 1 <= k <= min(E, %d), E <= %d (T=%d E=%d k=%d)",
                    MOE_MAX_TOPK, MOE_MAX_EXPERTS, T, E, k);
    if (T == 0) return MOE_OK;
    if (!logits || !ids || !weights) return fail(MOE_ERR_INVALID_ARG, "route: NULL output");
    if (x) {
        if (!w_router) return fail(MOE_ERR_INVALID_ARG, "route: NULL router weights");
        if (!moe::router_shape_supported(H, w_dtype))
            return fail(MOE_ERR_INVALID_ARG, "route: unsupported H=%d / dtype %d (H %% 128 == 0, f32 or bf16)",
                        H, w_dtype);
        if (!aligned16(x) || !aligned16(w_router) || (x_norm && !aligned16(x_norm)))
            return fail(MOE_ERR_INVALID_ARG, "route: x, w_router and x_norm must be 16-byte aligned");
    } else if (!logit_bias) {
        return fail(MOE_ERR_INVALID_ARG, "route: x and logit_bias are both NULL");
    }
    int *eflags = moe::device_error_flags();
    if (!eflags) return fail(MOE_ERR_HIP, "device error flags unavailable");
    auto s = static_cast<hipStream_t>(stream);
    const bool norm = flags & MOE_ROUTE_RMSNORM;
    hipError_t e = moe::launch_router_logits(x, w_router, w_dtype, T, H, E, logit_bias, logits, norm,
                                             norm ? x_norm : nullptr, s);
    if (e != hipSuccess) return fail_hip(e, "route: router logits launch");
    return finish_launch(moe::launch_topk_softmax(logits, T, E, k, ids, weights, eflags, s), "route: top-k launch");
}

size_t moe_ffn_workspace_bytes(int T, int k, int I) {
    if (T < 0 || k < 0 || I < 0) return 0;
    return moe::ffn_workspace_bytes(T, k, I);
}

int moe_expert_ffn_grouped(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                           const float *weights, const int32_t *slot_of, const void *pool,
                           size_t expert_bytes, int w_dtype, const void *shared_w, float *y_out,
                           void *workspace, size_t workspace_bytes, int flags, void *stream) {
    if (T < 0 || T > MOE_MAX_DECODE_TOKENS)
        return fail(MOE_ERR_INVALID_ARG, "ffn: T=%d outside [0, %d]", T, MOE_MAX_DECODE_TOKENS);
    if (k < 1 || k > MOE_MAX_TOPK || E < 1 || k > E)
        return fail(MOE_ERR_INVALID_ARG, "ffn: need 1 <= k <= min(E, %d) (E=%d k=%d)", MOE_MAX_TOPK, E, k);
    if (!moe::ffn_shape_supported(H, I, w_dtype))
        return fail(MOE_ERR_INVALID_ARG, "ffn: unsupported H=%d I=%d dtype=%d (multiples of 128; f32, bf16, int4g128)",
                    H, I, w_dtype);
    if (expert_bytes < moe::expert_blob_bytes(H, I, w_dtype) || expert_bytes % 256)
        return fail(MOE_ERR_INVALID_ARG, "ffn: expert_bytes %zu must be >= %zu and a multiple of 256",
                    expert_bytes, moe::expert_blob_bytes(H, I, w_dtype));
    if (T == 0) return MOE_OK;
    if (!x || !ids || !weights || !pool || !y_out || !workspace)
        return fail(MOE_ERR_INVALID_ARG, "ffn: NULL pointer argument");
    if (!aligned16(x) || !aligned16(pool) || (shared_w && !aligned16(shared_w)) || !aligned16(workspace))
        return fail(MOE_ERR_INVALID_ARG, "ffn: x, pool, shared_w and workspace must be 16-byte aligned");
    if (workspace_bytes < moe::ffn_workspace_bytes(T, k, I))
        return fail(MOE_ERR_INVALID_ARG, "ffn: workspace of %zu bytes, need %zu", workspace_bytes,
                    moe::ffn_workspace_bytes(T, k, I));
    int *eflags = moe::device_error_flags();
    if (!eflags) return fail(MOE_ERR_HIP, "device error flags unavailable");
    const moe::FfnWorkspace ws = moe::ffn_workspace(workspace, T, k, I);
    return finish_launch(moe::launch_expert_ffn(x, T, H, I, E, k, ids, weights, slot_of, pool, expert_bytes,
                                                w_dtype, shared_w, y_out, flags & MOE_ACCUMULATE, ws, eflags,
                                                static_cast<hipStream_t>(stream)),
                         "ffn launch");
}

int moe_expert_ffn_grouped_noalloc(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                                   const float *weights, const int32_t *slot_of, const void *pool, size_t expert_bytes,
                                   int w_dtype, const void *shared_w, float *y_out, int flags, void *stream) {
    // Nothing here allocates: the error flags and the scratch address come from moe_init's set-up.
    int *eflags = moe::device_error_flags_ready();
    void *ws = moe::noalloc_scratch();
    if (!eflags || !ws)
        return fail(MOE_ERR_INVALID_ARG, "ffn (no allocation): call moe_init on this device first");
    if (T < 0 || T > MOE_MAX_DECODE_TOKENS || k < 1 || k > MOE_MAX_TOPK || I < 0)
        return fail(MOE_ERR_INVALID_ARG, "ffn (no allocation): T=%d or k=%d out of range", T, k);
    const size_t need = moe::ffn_workspace_bytes(T, k, I);
    if (need > size_t(MOE_NOALLOC_SCRATCH_BYTES))
        return fail(MOE_ERR_INVALID_ARG,
                    "ffn (no allocation): T=%d k=%d I=%d needs %zu bytes of workspace, the fixed scratch holds %d",
                    T, k, I, need, MOE_NOALLOC_SCRATCH_BYTES);
    return moe_expert_ffn_grouped(x, T, H, I, E, k, ids, weights, slot_of, pool, expert_bytes, w_dtype, shared_w,
                                  y_out, ws, size_t(MOE_NOALLOC_SCRATCH_BYTES), flags, stream);
}

size_t moe_prefill_workspace_bytes(int T, int k, int E, int H, int I) {
    if (T < 0 || k < 1 || E < 1 || H < 1 || I < 1) return 0;
    return moe::prefill_workspace_bytes(T, k, E, H, I);
}

int moe_prefill_grouped(const float *x, int T, int H, int I, int E, int k, const int32_t *ids, const float *weights,
                        const int32_t *slot_of, const void *pool, size_t expert_bytes, int w_dtype,
                        const void *shared_w, float *y_out, void *workspace, size_t workspace_bytes, int flags,
                        void *stream) {
    if (T < 0 || k < 1 || k > MOE_MAX_TOPK || E < 1 || E > MOE_MAX_EXPERTS || k > E)
        return fail(MOE_ERR_INVALID_ARG, "prefill: need T >= 0, 1 <= k <= min(E, %d), E <= %d (T=%d E=%d k=%d)",
                    MOE_MAX_TOPK, MOE_MAX_EXPERTS, T, E, k);
    if (!moe::ffn_shape_supported(H, I, w_dtype))
        return fail(MOE_ERR_INVALID_ARG, "prefill: unsupported H=%d I=%d dtype=%d", H, I, w_dtype);
    if (!moe::prefill_dtype_supported(w_dtype))
        return fail(MOE_ERR_INVALID_ARG, "prefill: weights must be MOE_BF16 or MOE_INT4G128 (dtype=%d)", w_dtype);
    if (expert_bytes < moe::expert_blob_bytes(H, I, w_dtype) || expert_bytes % 256)
        return fail(MOE_ERR_INVALID_ARG, "prefill: expert_bytes %zu must be >= %zu and a multiple of 256", expert_bytes,
                    moe::expert_blob_bytes(H, I, w_dtype));
    if (T == 0) return MOE_OK;
    if (size_t(T) * k > size_t(INT32_MAX) / 2) return fail(MOE_ERR_INVALID_ARG, "prefill: T*k too large");
    if (!x || !ids || !weights || !pool || !y_out || !workspace)
        return fail(MOE_ERR_INVALID_ARG, "prefill: NULL pointer argument");
    if (!aligned16(x) || !aligned16(pool) || (shared_w && !aligned16(shared_w)) || !aligned16(workspace))
        return fail(MOE_ERR_INVALID_ARG, "prefill: x, pool, shared_w and workspace must be 16-byte aligned");
    if (workspace_bytes < moe::prefill_workspace_bytes(T, k, E, H, I))
        return fail(MOE_ERR_INVALID_ARG, "prefill: workspace of %zu bytes, need %zu", workspace_bytes,
                    moe::prefill_workspace_bytes(T, k, E, H, I));
    int *eflags = moe::device_error_flags();
    if (!eflags) return fail(MOE_ERR_HIP, "device error flags unavailable");
    const moe::PrefillWorkspace ws = moe::prefill_workspace(workspace, T, k, E, H, I);
    return finish_launch(moe::launch_prefill_ffn(x, T, H, I, E, k, ids, weights, slot_of, pool, expert_bytes, w_dtype,
                                                 shared_w, y_out, flags & MOE_ACCUMULATE, ws, eflags,
                                                 static_cast<hipStream_t>(stream)),
                         "prefill launch");
}

int moe_combine(const float *y_partial, const float *weights, const float *y_shared, int T, int k,
                int H, float *y_out, int flags, void *stream) {
    if (T < 0 || k < 0 || H < 0) return fail(MOE_ERR_INVALID_ARG, "combine: negative size");
    if (size_t(T) * H == 0) return MOE_OK;
    if ((k > 0 && (!y_partial || !weights)) || !y_out) return fail(MOE_ERR_INVALID_ARG, "combine: NULL pointer");
    return finish_launch(moe::launch_combine(y_partial, weights, y_shared, T, k, H, y_out, flags & MOE_ACCUMULATE,
                                             static_cast<hipStream_t>(stream)),
                         "combine launch");
}

size_t moe_attention_workspace_bytes(int n_heads, int n_kv, int head_dim, int max_pos) {
    if (n_heads < 1 || n_kv < 1 || head_dim < 1 || max_pos < 1) return 0;
    return moe::attention_workspace_bytes(n_heads, n_kv, head_dim, max_pos);
}

int moe_attention_decode(float *x, int H, int n_heads, int n_kv, int head_dim, const void *w_qkv, const void *w_o,
                         void *k_cache, void *v_cache, int max_pos, int p, float theta, void *workspace,
                         size_t workspace_bytes, void *stream) {
    if (!x || !w_qkv || !w_o || !k_cache || !v_cache || !workspace)
        return fail(MOE_ERR_INVALID_ARG, "attention: NULL pointer");
    if (!moe::attention_shape_supported(H, n_heads, n_kv, head_dim, max_pos))
        return fail(MOE_ERR_INVALID_ARG, "attention: unsupported shape (H %d, heads %d/%d, head_dim %d, max_pos %d)", H,
                    n_heads, n_kv, head_dim, max_pos);
    if (p < 0 || p >= max_pos) return fail(MOE_ERR_INVALID_ARG, "attention: position %d outside [0, %d)", p, max_pos);
    if (!(theta > 1.f)) return fail(MOE_ERR_INVALID_ARG, "attention: rotary base must exceed 1");
    if (!aligned16(x) || !aligned16(w_qkv) || !aligned16(w_o) || !aligned16(k_cache) || !aligned16(v_cache) ||
        !aligned16(workspace))
        return fail(MOE_ERR_INVALID_ARG, "attention: buffers must be 16-byte aligned");
    if (workspace_bytes < moe::attention_workspace_bytes(n_heads, n_kv, head_dim, max_pos))
        return fail(MOE_ERR_INVALID_ARG, "attention: workspace of %zu bytes, need %zu", workspace_bytes,
                    moe::attention_workspace_bytes(n_heads, n_kv, head_dim, max_pos));
    return finish_launch(moe::launch_attention_decode(x, H, n_heads, n_kv, head_dim, w_qkv, w_o,
                                                      static_cast<uint16_t *>(k_cache), static_cast<uint16_t *>(v_cache),
                                                      max_pos, p, theta, workspace, static_cast<hipStream_t>(stream)),
                         "attention launch");
}

int moe_hbm_read_probe(const void *buf, size_t bytes, float *sink, void *stream) {
    if (!buf || !sink) return fail(MOE_ERR_INVALID_ARG, "hbm read probe: NULL pointer");
    if (bytes % 16 || reinterpret_cast<uintptr_t>(buf) % 16)
        return fail(MOE_ERR_INVALID_ARG, "hbm read probe: buffer and size must be multiples of 16 bytes");
    if (bytes / 16 / (4 * 256) >= (size_t(1) << 31))
        return fail(MOE_ERR_INVALID_ARG, "hbm read probe: buffer too large for one launch");
    return finish_launch(moe::launch_hbm_read(buf, bytes, sink, static_cast<hipStream_t>(stream)), "read probe launch");
}

}  // extern "C"
