// stack.cpp -- decode step over a stack of MoE layers: x <- x + MoE_l(rmsnorm(x)),
// l = 0..L-1 (attention is the identity; the pre-norm is fused into the router).  Under a budget each layer brings its ids to
// the host, runs the slot lookup, then enqueues the expert FFN and releases
// the slots; with every expert resident the whole step stays on the device.
#include <string.h>

#include <vector>

#include "internal.h"
#include "../../include/moe_budget.h"

namespace {

// Device time of consecutive spans on one stream: each entry is N+1 events
// (span i runs from event i to event i+1) taken from a ring; an entry's spans
// are folded into running sums when the entry is reused or on read-out.
template <int N>
class SpanTimer {
  public:
    static constexpr int kEntries = 1024;
    hipError_t init() {
        for (auto &en : entries_)
            for (auto &ev : en.ev) {
                hipError_t e = hipEventCreate(&ev);
                if (e != hipSuccess) return e;
            }
        return hipSuccess;
    }
    void destroy() {
        for (auto &en : entries_)
            for (auto &ev : en.ev)
                if (ev) (void)hipEventDestroy(ev);
    }
    // Events of the next entry, or nullptr if folding its old spans failed.
    hipEvent_t *next() {
        Entry &en = entries_[next_];
        next_ = (next_ + 1) % kEntries;
        if (en.used && !fold(en)) return nullptr;
        en.used = true;
        return en.ev;
    }
    bool flush() {
        for (auto &en : entries_)
            if (en.used && !fold(en)) return false;
        return true;
    }
    void read(int span, double *mean_ms, uint64_t *count) {
        *mean_ms = n_[span] ? sum_ms_[span] / double(n_[span]) : 0.0;
        *count = n_[span];
        sum_ms_[span] = 0.0;
        n_[span] = 0;
    }

  private:
    struct Entry {
        hipEvent_t ev[N + 1] = {};
        bool used = false;
    };
    bool fold(Entry &en) {
        if (hipEventSynchronize(en.ev[N]) != hipSuccess) return false;
        for (int i = 0; i < N; ++i) {
            float ms = 0.f;
            if (hipEventElapsedTime(&ms, en.ev[i], en.ev[i + 1]) != hipSuccess) return false;
            sum_ms_[i] += ms;
            ++n_[i];
        }
        en.used = false;
        return true;
    }
    Entry entries_[kEntries];
    int next_ = 0;
    double sum_ms_[N] = {};
    uint64_t n_[N] = {};
};

}  // namespace

struct moe_stack {
    moe_stack_desc d{};
    std::vector<const void *> router_w, shared_w;
    const int32_t *slot_table = nullptr;
    const void *pool = nullptr;
    bool budgeted = false;
    size_t expert_bytes = 0;
    float *logits = nullptr;    // device [Tmax x E]
    float *h = nullptr;         // device [Tmax x H]: RMS-normalised input of the current layer
    int32_t *ids = nullptr;     // device [Tmax x k]
    float *weights = nullptr;   // device [Tmax x k]
    int32_t *ids_host = nullptr;  // pinned [Tmax x k]
    void *ws = nullptr;
    size_t ws_bytes = 0;
    hipEvent_t ids_ready = nullptr;
    bool timing = false;
    SpanTimer<1> route_timer;   // router logits + top-k
    SpanTimer<2> ffn_timer;     // span 0: gate/up + SwiGLU, span 1: down + combine
};

extern "C" {

int moe_stack_destroy(moe_stack *s) {
    if (!s) return MOE_OK;
    (void)hipDeviceSynchronize();
    if (s->logits) (void)hipFree(s->logits);
    if (s->h) (void)hipFree(s->h);
    if (s->ids) (void)hipFree(s->ids);
    if (s->weights) (void)hipFree(s->weights);
    if (s->ids_host) (void)hipHostFree(s->ids_host);
    if (s->ws) (void)hipFree(s->ws);
    if (s->ids_ready) (void)hipEventDestroy(s->ids_ready);
    s->route_timer.destroy();
    s->ffn_timer.destroy();
    delete s;
    return MOE_OK;
}

int moe_stack_create(const moe_stack_desc *d, moe_stack **out) {
    if (!d || !out) return moe::fail(MOE_ERR_INVALID_ARG, "NULL descriptor or output");
    *out = nullptr;
    if (d->n_layers < 1 || d->E < 1 || d->k < 1 || d->k > d->E || d->k > MOE_MAX_TOPK || d->E > MOE_MAX_EXPERTS)
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: bad L/E/k (%d/%d/%d)", d->n_layers, d->E, d->k);
    if (d->max_tokens < 1 || d->max_tokens > MOE_MAX_DECODE_TOKENS)
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: max_tokens must be in [1, %d]", MOE_MAX_DECODE_TOKENS);
    if (!moe::ffn_shape_supported(d->H, d->I, d->w_dtype) || !moe::router_shape_supported(d->H, d->router_dtype))
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: unsupported H/I/dtype");
    if (!d->router_w || !d->cache) return moe::fail(MOE_ERR_INVALID_ARG, "stack: router weights and cache required");
    moe_cache_stats cs;
    int st = expert_cache_stats(d->cache, &cs);
    if (st != MOE_OK) return st;

    auto *s = new moe_stack();
    s->d = *d;
    s->router_w.assign(d->router_w, d->router_w + d->n_layers);
    if (d->shared_w) s->shared_w.assign(d->shared_w, d->shared_w + d->n_layers);
    s->d.router_w = nullptr;
    s->d.shared_w = nullptr;
    expert_cache_slot_table(d->cache, &s->slot_table, &s->pool);
    s->budgeted = cs.capacity < d->n_layers * d->E;
    s->expert_bytes = moe::cache_expert_bytes(d->cache);
    if (s->expert_bytes < moe::expert_blob_bytes(d->H, d->I, d->w_dtype)) {
        delete s;
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: cache slots are smaller than one expert blob");
    }
    const int T = d->max_tokens;
    hipError_t e;
    auto bail = [&](hipError_t err, const char *what) {
        int code = moe::fail_hip(err, what);
        moe_stack_destroy(s);
        return code;
    };
    if ((e = hipMalloc(&s->logits, sizeof(float) * T * d->E)) != hipSuccess) return bail(e, "stack buffers");
    if ((e = hipMalloc(&s->h, sizeof(float) * T * d->H)) != hipSuccess) return bail(e, "stack buffers");
    if ((e = hipMalloc(&s->ids, sizeof(int32_t) * T * d->k)) != hipSuccess) return bail(e, "stack buffers");
    if ((e = hipMalloc(&s->weights, sizeof(float) * T * d->k)) != hipSuccess) return bail(e, "stack buffers");
    if ((e = hipHostMalloc(&s->ids_host, sizeof(int32_t) * T * d->k, 0)) != hipSuccess) return bail(e, "stack buffers");
    s->ws_bytes = moe::ffn_workspace_bytes(T, d->k, d->I);
    if ((e = hipMalloc(&s->ws, s->ws_bytes)) != hipSuccess) return bail(e, "stack workspace");
    if ((e = hipEventCreateWithFlags(&s->ids_ready, hipEventDisableTiming)) != hipSuccess)
        return bail(e, "stack event");
    if ((e = s->route_timer.init()) != hipSuccess || (e = s->ffn_timer.init()) != hipSuccess)
        return bail(e, "stack timing events");
    *out = s;
    moe::clear_error();
    return MOE_OK;
}

int moe_stack_decode_step(moe_stack *s, int step, float *x, int T, const float *logit_bias,
                          int32_t *ids_out, float *weights_out, void *stream) {
    if (!s || !x) return moe::fail(MOE_ERR_INVALID_ARG, "stack step: NULL argument");
    if (T < 1 || T > s->d.max_tokens)
        return moe::fail(MOE_ERR_INVALID_ARG, "stack step: T=%d outside [1, %d]", T, s->d.max_tokens);
    auto strm = static_cast<hipStream_t>(stream);
    int *eflags = moe::device_error_flags();
    if (!eflags) return moe::fail(MOE_ERR_HIP, "device error flags unavailable");
    const auto &d = s->d;
    const moe::FfnWorkspace ws = moe::ffn_workspace(s->ws, T, d.k, d.I);
    for (int l = 0; l < d.n_layers; ++l) {
        int32_t *ids = ids_out ? ids_out + size_t(l) * T * d.k : s->ids;
        float *w = weights_out ? weights_out + size_t(l) * T * d.k : s->weights;
        const float *bias = logit_bias ? logit_bias + size_t(l) * T * d.E : nullptr;
        hipEvent_t *rt = s->timing ? s->route_timer.next() : nullptr;
        if (rt) (void)hipEventRecord(rt[0], strm);
        hipError_t e = moe::launch_router_logits(x, s->router_w[l], d.router_dtype, T, d.H, d.E, bias, s->logits,
                                                 true, s->h, strm);
        if (e == hipSuccess) e = moe::launch_topk_softmax(s->logits, T, d.E, d.k, ids, w, eflags, strm);
        if (e != hipSuccess) return moe::fail_hip(e, "stack step: routing");
        if (rt) (void)hipEventRecord(rt[1], strm);
        if (s->budgeted) {
            e = hipMemcpyAsync(s->ids_host, ids, sizeof(int32_t) * T * d.k, hipMemcpyDeviceToHost, strm);
            if (e == hipSuccess) e = hipEventRecord(s->ids_ready, strm);
            if (e == hipSuccess) e = hipEventSynchronize(s->ids_ready);
            if (e != hipSuccess) return moe::fail_hip(e, "stack step: ids to host");
            int st = expert_cache_lookup(d.cache, step, l, s->ids_host, T * d.k, nullptr, nullptr, strm);
            if (st != MOE_OK) return st;
        }
        moe::FfnEvents fe{}, *fep = nullptr;
        if (hipEvent_t *ft = s->timing ? s->ffn_timer.next() : nullptr) {
            fe = {ft[0], ft[1], ft[2]};
            fep = &fe;
        }
        e = moe::launch_expert_ffn(s->h, T, d.H, d.I, d.E, d.k, ids, w, s->slot_table + size_t(l) * d.E, s->pool,
                                   s->expert_bytes, d.w_dtype, s->shared_w.empty() ? nullptr : s->shared_w[l], x,
                                   true, ws, eflags, strm, fep);
        if (e != hipSuccess) return moe::fail_hip(e, "stack step: expert FFN");
        if (s->budgeted) {
            int st = expert_cache_release(d.cache, strm);
            if (st != MOE_OK) return st;
        }
    }
    moe::clear_error();
    return MOE_OK;
}

int moe_stack_set_timing(moe_stack *s, int on) {
    if (!s) return moe::fail(MOE_ERR_INVALID_ARG, "stack is NULL");
    s->timing = on != 0;
    return MOE_OK;
}

int moe_stack_kernel_time(moe_stack *s, int which, double *mean_ms, uint64_t *count) {
    if (!s || !mean_ms || !count || which < 0 || which > 2)
        return moe::fail(MOE_ERR_INVALID_ARG, "kernel_time: bad argument");
    bool ok = which == 0 ? s->route_timer.flush() : s->ffn_timer.flush();
    if (!ok) return moe::fail(MOE_ERR_HIP, "kernel_time: reading events failed");
    if (which == 0)
        s->route_timer.read(0, mean_ms, count);
    else
        s->ffn_timer.read(which - 1, mean_ms, count);
    return MOE_OK;
}

}  // extern "C"
