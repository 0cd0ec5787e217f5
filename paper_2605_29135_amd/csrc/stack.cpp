// stack.cpp -- decode step and prefill chunk over a stack of MoE layers:
// x <- x + MoE_l(rmsnorm(x)), l = 0..L-1 (attention is the identity; for a
// decode step the pre-norm is fused into the router).  Under a budget each
// layer brings its ids to the host, runs the slot lookup, then enqueues the
// expert FFN and releases the slots; with every expert resident the whole
// step stays on the device.
#include <string.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <vector>

#include "host_ffn.h"
#include "internal.h"
#include "../../include/moe_budget.h"

namespace {

// Arguments of the last layer's launches, for re-launching them in isolation.
// A past token remembered for reverse rotation: its layer-0 expert set (sorted,
// the context signature) and its expert set at every layer.
struct Snapshot {
    std::vector<int32_t> sig;   // [k] ascending
    std::vector<int32_t> sets;  // [L x k] in rank order
    uint64_t stamp = 0;         // token counter when stored
};

// The buffers a captured decode graph was recorded with (a replay needs the same ones).
struct GraphKey {
    const float *x = nullptr, *bias = nullptr;
    const int32_t *ids = nullptr;
    const float *w = nullptr, *logits = nullptr;
    bool operator==(const GraphKey &o) const {
        return x == o.x && bias == o.bias && ids == o.ids && w == o.w && logits == o.logits;
    }
};

struct LastLayer {
    bool valid = false;
    int T = 0, layer = 0;
    const int32_t *ids = nullptr;
    const float *weights = nullptr;
    const int32_t *slot_of = nullptr;
    const uint8_t *pool = nullptr;
    moe::FfnPlan plan;
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
    int32_t *slots_host = nullptr; // [Tmax x k] slot of each id after the lookup
    int32_t *dev_slots = nullptr;  // device [L x max_tokens x k]: slot of each id after each layer's device lookup
    int *dev_step = nullptr;       // device: step tag of a replayed decode graph's decisions
    int32_t *all_experts = nullptr;  // device [E]: 0..E-1, the prefill's prefetch of a whole layer
    bool attn = false;             // a self-attention block before each MoE block
    moe_attention_desc ad{};       // its shapes (the arrays below hold its per-layer buffers)
    std::vector<const void *> a_wqkv, a_wo;
    std::vector<void *> a_k, a_v;
    void *attn_ws = nullptr;
    int attn_pos = 0;              // position of the next decode step
    int last_attn_pos = -1;        // position of the last one
    hipGraphExec_t graph_exec = nullptr;  // one-token decode step captured for replay (device residency)
    GraphKey graph_key;
    void *ws = nullptr;
    size_t ws_bytes = 0;
    void *pws = nullptr;        // prefill workspace (max_prefill_tokens > 0)
    size_t pws_bytes = 0;
    int tcap = 0;               // rows of the per-token buffers: max(max_tokens, max_prefill_tokens)
    hipEvent_t ids_ready = nullptr;
    moe::IdsMailbox *mbox = nullptr;      // coherent pinned: one token's ids published by the top-k kernel
    moe::IdsMailbox *mbox_dev = nullptr;  // its device address
    uint32_t mbox_seq = 0;
    std::vector<uint32_t> demand;          // [L x E] demand lookups per expert (prefetch ranking)
    std::vector<Snapshot> snaps;           // reverse rotation: remembered tokens (<= d.recall)
    std::vector<int32_t> cur_sets;         // [L x k] the current token's expert sets
    int recalled = -1;                     // snapshot recalled for the current token, or -1
    uint64_t tokens = 0;                   // one-token decode steps so far (snapshot stamps)
    moe_host_tier *host = nullptr;  // the host tier, when the cache has one
    float *h_pub = nullptr;         // coherent pinned [H]: the layer's normalised input, published by the top-k
    float *h_pub_dev = nullptr;     // its device address
    float *y_pub = nullptr;         // coherent pinned [H]: the host tier's output for the layer
    float *y_pub_dev = nullptr;     // its device address
    std::vector<const void *> host_blobs;  // [k] blobs the host tier computes this layer
    std::vector<float> host_w;             // [k] their combine weights
    uint64_t host_calls = 0;               // layers whose experts the host tier computed (some or all)
    float *scratch_x = nullptr;  // device [Tmax x H] scratch input/output of kernel re-launches
    float *scratch_y = nullptr;  // device [Tmax x H]
    std::vector<LastLayer> last;  // per layer, arguments of the last decode step
};

namespace {

// Wait until the top-k kernel has published sequence number `seq`, then copy
// the ids.  A bounded spin: should the sequence number not appear, the stream
// is synchronised so that a failed kernel reports its error.
int wait_published_ids(moe_stack *s, uint32_t seq, hipStream_t strm) {
    volatile uint32_t *flag = &s->mbox->seq;
    const auto t0 = std::chrono::steady_clock::now();
    for (uint64_t spin = 0; *flag != seq; ++spin) {
        if ((spin & 4095) == 4095 && std::chrono::steady_clock::now() - t0 > std::chrono::seconds(10)) {
            hipError_t e = hipStreamSynchronize(strm);
            if (e != hipSuccess) return moe::fail_hip(e, "stack step: routing");
            if (*flag != seq) return moe::fail(MOE_ERR_HIP, "stack step: the routing kernel did not publish its ids");
            break;
        }
        __builtin_ia32_pause();
    }
    std::atomic_thread_fence(std::memory_order_acquire);
    const volatile int32_t *src = s->mbox->ids;
    for (int j = 0; j < s->d.k; ++j) s->ids_host[j] = src[j];
    if (s->host) {
        const volatile float *w = s->mbox->w;
        for (int j = 0; j < s->d.k; ++j) s->host_w[size_t(j)] = w[j];
    }
    return MOE_OK;
}

// Speculative prefetch after layer l of a one-token step: the next layer's (the
// next step's first layer after the last) most often demanded experts that are
// not resident, up to d.prefetch of them, ties to the lower id.
// The snapshot whose signature shares the most experts with `s0` (the token's
// layer-0 ids), at least the configured overlap; ties go to the most recent.
int find_recall(const moe_stack *s, const int32_t *s0) {
    const auto &d = s->d;
    const int need = d.recall_overlap > 0 ? d.recall_overlap : d.k;
    int best = -1, best_n = 0;
    for (size_t i = 0; i < s->snaps.size(); ++i) {
        const Snapshot &sn = s->snaps[i];
        int n = 0;
        for (int j = 0; j < d.k; ++j)
            n += std::binary_search(sn.sig.begin(), sn.sig.end(), s0[j]) ? 1 : 0;
        if (n < need) continue;
        if (best < 0 || n > best_n || (n == best_n && sn.stamp > s->snaps[best].stamp)) {
            best = int(i);
            best_n = n;
        }
    }
    return best;
}

// End of a one-token step: remember it, over a snapshot with the same signature, else the oldest.
void store_snapshot(moe_stack *s) {
    const auto &d = s->d;
    Snapshot sn;
    sn.sig.assign(s->cur_sets.begin(), s->cur_sets.begin() + d.k);
    std::sort(sn.sig.begin(), sn.sig.end());
    sn.sets = s->cur_sets;
    sn.stamp = ++s->tokens;
    for (Snapshot &o : s->snaps)
        if (o.sig == sn.sig) {
            o = std::move(sn);
            return;
        }
    if (int(s->snaps.size()) < d.recall) {
        s->snaps.push_back(std::move(sn));
        return;
    }
    size_t oldest = 0;
    for (size_t i = 1; i < s->snaps.size(); ++i)
        if (s->snaps[i].stamp < s->snaps[oldest].stamp) oldest = i;
    s->snaps[oldest] = std::move(sn);
}

int prefetch_next(moe_stack *s, int step, int l) {
    const auto &d = s->d;
    const int ln = (l + 1) % d.n_layers, sn = l + 1 == d.n_layers ? step + 1 : step;
    std::vector<std::pair<uint32_t, int32_t>> cand;
    cand.reserve(size_t(d.E));
    for (int e = 0; e < d.E; ++e)
        if (!moe::cache_resident(d.cache, ln, e)) cand.emplace_back(s->demand[size_t(ln) * d.E + e], e);
    const size_t n = std::min(cand.size(), size_t(d.prefetch));
    if (n == 0) return MOE_OK;
    std::partial_sort(cand.begin(), cand.begin() + n, cand.end(), [](const auto &a, const auto &b) {
        return a.first != b.first ? a.first > b.first : a.second < b.second;
    });
    int32_t ids[MOE_MAX_EXPERTS];
    for (size_t i = 0; i < n; ++i) ids[i] = cand[i].second;
    return expert_cache_prefetch(d.cache, sn, ln, ids, int(n));
}

}  // namespace

extern "C" {

int moe_stack_destroy(moe_stack *s) {
    if (!s) return MOE_OK;
    (void)hipDeviceSynchronize();
    if (s->logits) (void)hipFree(s->logits);
    if (s->h) (void)hipFree(s->h);
    if (s->ids) (void)hipFree(s->ids);
    if (s->weights) (void)hipFree(s->weights);
    if (s->ids_host) (void)hipHostFree(s->ids_host);
    delete[] s->slots_host;
    if (s->ws) (void)hipFree(s->ws);
    if (s->pws) (void)hipFree(s->pws);
    if (s->ids_ready) (void)hipEventDestroy(s->ids_ready);
    if (s->mbox) (void)hipHostFree(s->mbox);
    if (s->scratch_x) (void)hipFree(s->scratch_x);
    if (s->scratch_y) (void)hipFree(s->scratch_y);
    if (s->dev_slots) (void)hipFree(s->dev_slots);
    if (s->dev_step) (void)hipFree(s->dev_step);
    if (s->all_experts) (void)hipFree(s->all_experts);
    if (s->attn_ws) (void)hipFree(s->attn_ws);
    if (s->host) moe_host_tier_destroy(s->host);
    if (s->h_pub) (void)hipHostFree(s->h_pub);
    if (s->y_pub) (void)hipHostFree(s->y_pub);
    if (s->graph_exec) (void)hipGraphExecDestroy(s->graph_exec);
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
    if (d->max_prefill_tokens < 0 || d->max_prefill_tokens > (1 << 20))
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: max_prefill_tokens must be in [0, 2^20]");
    if (d->prefetch < 0 || d->prefetch > d->E)
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: prefetch must be in [0, E]");
    if (d->recall < 0 || d->recall > 4096 || d->recall_overlap < 0 || d->recall_overlap > d->k)
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: recall must be in [0, 4096], recall_overlap in [0, k]");
    if (d->cache && moe::cache_device(d->cache) && (d->prefetch > 0 || d->recall > 0))
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: prefetch and recall need host lookups (not MOE_CACHE_DEVICE)");
    if (const moe_attention_desc *a = d->attention) {
        if (!moe::attention_shape_supported(d->H, a->n_heads, a->n_kv, a->head_dim, a->max_pos) || !(a->theta > 1.f) ||
            a->start_pos < 0 || a->start_pos >= a->max_pos || !a->w_qkv || !a->w_o || !a->k_cache || !a->v_cache)
            return moe::fail(MOE_ERR_INVALID_ARG, "stack: unsupported attention block");
        for (int l = 0; l < d->n_layers; ++l)
            if (!a->w_qkv[l] || !a->w_o[l] || !a->k_cache[l] || !a->v_cache[l])
                return moe::fail(MOE_ERR_INVALID_ARG, "stack: attention buffers of layer %d missing", l);
        if (d->max_prefill_tokens > 0 || d->max_tokens != 1)
            return moe::fail(MOE_ERR_INVALID_ARG, "stack: an attention block decodes one token per step (no prefill)");
    }
    if (d->cache && moe::cache_host_tier(d->cache) &&
        (d->max_tokens != 1 || d->max_prefill_tokens > 0 || d->attention || d->prefetch > 0 || d->recall > 0))
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: a host-tier cache runs one-token decode steps only (max_tokens 1, "
                                              "no prefill, attention, prefetch or recall)");
    if (d->host_threads < 0) return moe::fail(MOE_ERR_INVALID_ARG, "stack: host_threads must be >= 0");
    if (d->max_prefill_tokens > 0 && !moe::prefill_dtype_supported(d->w_dtype))
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: prefill needs MOE_BF16 or MOE_INT4G128 experts");
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
    // a preloaded cache never misses: the step stays on the device; otherwise
    // every layer looks its experts up on the host
    s->budgeted = !moe::cache_preloaded(d->cache);
    s->expert_bytes = moe::cache_expert_bytes(d->cache);
    if (s->expert_bytes < moe::expert_blob_bytes(d->H, d->I, d->w_dtype)) {
        delete s;
        return moe::fail(MOE_ERR_INVALID_ARG, "stack: cache slots are smaller than one expert blob");
    }
    const int T = d->max_tokens > d->max_prefill_tokens ? d->max_tokens : d->max_prefill_tokens;
    s->tcap = T;
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
    s->slots_host = new int32_t[size_t(T) * d->k];
    if (moe::cache_device(d->cache) &&
        ((e = hipMalloc(&s->dev_slots, sizeof(int32_t) * size_t(d->n_layers) * d->max_tokens * d->k)) != hipSuccess ||
         (e = hipMalloc(&s->dev_step, sizeof(int))) != hipSuccess))
        return bail(e, "stack buffers");
    if (moe::cache_device(d->cache) && d->max_prefill_tokens > 0) {
        std::vector<int32_t> iota(size_t(d->E));
        for (int i = 0; i < d->E; ++i) iota[size_t(i)] = i;
        if ((e = hipMalloc(&s->all_experts, sizeof(int32_t) * size_t(d->E))) != hipSuccess ||
            (e = hipMemcpy(s->all_experts, iota.data(), sizeof(int32_t) * size_t(d->E), hipMemcpyHostToDevice)) !=
                hipSuccess)
            return bail(e, "stack buffers");
    }
    if (const moe_attention_desc *a = d->attention) {
        s->attn = true;
        s->ad = *a;
        for (int l = 0; l < d->n_layers; ++l) {
            s->a_wqkv.push_back(a->w_qkv[l]);
            s->a_wo.push_back(a->w_o[l]);
            s->a_k.push_back(a->k_cache[l]);
            s->a_v.push_back(a->v_cache[l]);
        }
        s->ad.w_qkv = s->ad.w_o = nullptr;
        s->ad.k_cache = s->ad.v_cache = nullptr;
        s->attn_pos = a->start_pos;
        if ((e = hipMalloc(&s->attn_ws, moe::attention_workspace_bytes(a->n_heads, a->n_kv, a->head_dim, a->max_pos))) !=
            hipSuccess)
            return bail(e, "stack attention workspace");
    }
    s->d.attention = nullptr;  // the caller's descriptor need not outlive the call
    s->last.assign(d->n_layers, LastLayer{});
    s->demand.assign(size_t(d->n_layers) * d->E, 0u);
    s->cur_sets.assign(size_t(d->n_layers) * d->k, 0);
    s->ws_bytes = moe::ffn_workspace_bytes(d->max_tokens, d->k, d->I);
    if ((e = hipMalloc(&s->ws, s->ws_bytes)) != hipSuccess) return bail(e, "stack workspace");
    if (d->max_prefill_tokens > 0) {
        s->pws_bytes = moe::prefill_workspace_bytes(d->max_prefill_tokens, d->k, d->E, d->H, d->I);
        if ((e = hipMalloc(&s->pws, s->pws_bytes)) != hipSuccess) return bail(e, "stack prefill workspace");
    }
    if ((e = hipEventCreateWithFlags(&s->ids_ready, hipEventDisableTiming)) != hipSuccess)
        return bail(e, "stack event");
    if ((e = hipHostMalloc(reinterpret_cast<void **>(&s->mbox), sizeof(moe::IdsMailbox),
                           hipHostMallocCoherent | hipHostMallocMapped)) != hipSuccess)
        return bail(e, "stack ids mailbox");
    memset(s->mbox, 0, sizeof(moe::IdsMailbox));
    if ((e = hipHostGetDevicePointer(reinterpret_cast<void **>(&s->mbox_dev), s->mbox, 0)) != hipSuccess)
        return bail(e, "stack ids mailbox");
    if (moe::cache_host_tier(d->cache)) {
        int st2 = moe_host_tier_create(d->host_threads, &s->host);
        if (st2 != MOE_OK) {
            moe_stack_destroy(s);
            return st2;
        }
        const unsigned fl = hipHostMallocCoherent | hipHostMallocMapped;
        if ((e = hipHostMalloc(reinterpret_cast<void **>(&s->h_pub), sizeof(float) * d->H, fl)) != hipSuccess ||
            (e = hipHostMalloc(reinterpret_cast<void **>(&s->y_pub), sizeof(float) * d->H, fl)) != hipSuccess ||
            (e = hipHostGetDevicePointer(reinterpret_cast<void **>(&s->h_pub_dev), s->h_pub, 0)) != hipSuccess ||
            (e = hipHostGetDevicePointer(reinterpret_cast<void **>(&s->y_pub_dev), s->y_pub, 0)) != hipSuccess)
            return bail(e, "stack host tier buffers");
        s->host_blobs.assign(size_t(d->k), nullptr);
        s->host_w.assign(size_t(d->k), 0.f);
    }
    const size_t Td = size_t(d->max_tokens);
    if ((e = hipMalloc(&s->scratch_x, sizeof(float) * Td * d->H)) != hipSuccess) return bail(e, "stack buffers");
    if ((e = hipMalloc(&s->scratch_y, sizeof(float) * Td * d->H)) != hipSuccess) return bail(e, "stack buffers");
    *out = s;
    moe::clear_error();
    return MOE_OK;
}

}  // extern "C"

namespace {
// The work of one decode step, enqueued on `strm`.  With step_dev (device-resident
// cache, one token: nothing waits for the host) the decisions take their step tag
// from device memory, so that the enqueued work can be captured once and replayed.
int enqueue_decode(moe_stack *s, int step, float *x, int T, const float *logit_bias, int32_t *ids_out,
                   float *weights_out, float *logits_out, hipStream_t strm, const int *step_dev) {
    int *eflags = moe::device_error_flags();
    if (!eflags) return moe::fail(MOE_ERR_HIP, "device error flags unavailable");
    const auto &d = s->d;
    const moe::FfnWorkspace ws = moe::ffn_workspace(s->ws, T, d.k, d.I);
    s->recalled = -1;
    if (s->attn && (T != 1 || s->attn_pos >= s->ad.max_pos))
        return moe::fail(MOE_ERR_INVALID_ARG, T != 1 ? "stack step: an attention block decodes one token per step"
                                                     : "stack step: the attention caches are full");
    for (int l = 0; l < d.n_layers; ++l) {
        if (s->attn) {
            hipError_t ea = moe::launch_attention_decode(x, d.H, s->ad.n_heads, s->ad.n_kv, s->ad.head_dim,
                                                         s->a_wqkv[l], s->a_wo[l], static_cast<uint16_t *>(s->a_k[l]),
                                                         static_cast<uint16_t *>(s->a_v[l]), s->ad.max_pos,
                                                         s->attn_pos, s->ad.theta, s->attn_ws, strm);
            if (ea != hipSuccess) return moe::fail_hip(ea, "stack step: attention");
        }
        int32_t *ids = ids_out ? ids_out + size_t(l) * T * d.k : s->ids;
        float *w = weights_out ? weights_out + size_t(l) * T * d.k : s->weights;
        float *lg = logits_out ? logits_out + size_t(l) * T * d.E : s->logits;
        const float *bias = logit_bias ? logit_bias + size_t(l) * T * d.E : nullptr;
        // lookups on the device need no ids on the host; otherwise one token under a budget has the
        // top-k kernel publish its ids straight to host memory
        const bool dev_lookup = s->budgeted && moe::cache_device(d.cache);
        const bool mailbox = s->budgeted && T == 1 && !dev_lookup;
        const uint32_t seq = mailbox ? ++s->mbox_seq : 0;
        hipError_t e = moe::launch_router_logits(x, s->router_w[l], d.router_dtype, T, d.H, d.E, bias, lg, true,
                                                 s->h, strm);
        const bool fused = dev_lookup && T == 1;  // one token: top-k and the lookup in one kernel
        // with a host tier the top-k also publishes the weights and h_l for the host's share of the layer
        if (e == hipSuccess && !fused)
            e = moe::launch_topk_softmax(lg, T, d.E, d.k, ids, w, eflags, strm, mailbox ? s->mbox_dev : nullptr, seq,
                                         s->h, mailbox ? s->h_pub_dev : nullptr, d.H);
        if (e != hipSuccess) return moe::fail_hip(e, "stack step: routing");
        if (fused) {
            int st = moe::cache_topk_lookup(d.cache, step, l, lg, d.k, ids, w,
                                            s->dev_slots + size_t(l) * d.max_tokens * d.k, eflags, strm, step_dev,
                                            true);
            if (st != MOE_OK) return st;
        } else if (dev_lookup) {
            int st = expert_cache_lookup_device(d.cache, step, l, ids, T * d.k,
                                                s->dev_slots + size_t(l) * d.max_tokens * d.k, strm);
            if (st != MOE_OK) return st;
        } else if (s->budgeted) {
            if (mailbox) {
                int st = wait_published_ids(s, seq, strm);
                if (st != MOE_OK) return st;
            } else {
                e = hipMemcpyAsync(s->ids_host, ids, sizeof(int32_t) * T * d.k, hipMemcpyDeviceToHost, strm);
                if (e == hipSuccess) e = hipEventRecord(s->ids_ready, strm);
                if (e == hipSuccess) e = hipEventSynchronize(s->ids_ready);
                if (e != hipSuccess) return moe::fail_hip(e, "stack step: ids to host");
            }
            int st = expert_cache_lookup(d.cache, step, l, s->ids_host, T * d.k, s->slots_host, nullptr, strm);
            if (st != MOE_OK) return st;
            for (int j = 0; j < T * d.k; ++j) ++s->demand[size_t(l) * d.E + s->ids_host[j]];
            if (d.recall > 0 && T == 1) {
                std::copy(s->ids_host, s->ids_host + d.k, s->cur_sets.begin() + size_t(l) * d.k);
                if (l == 0) s->recalled = find_recall(s, s->ids_host);
            }
        }
        // Where this layer's experts live: after a lookup the host knows every
        // slot (T == 1 passes them to the kernels directly); preloaded slots are
        // layer * E + expert, so the layer's pool starts at slot layer * E.
        moe::FfnPlan plan;
        const int32_t *slot_of = s->slot_table + size_t(l) * d.E;
        const uint8_t *pool = static_cast<const uint8_t *>(s->pool);
        int n_host = 0;
        if (s->budgeted && T == 1 && !dev_lookup) {
            plan.n = d.k;
            for (int j = 0; j < d.k; ++j) {
                if (s->slots_host[j] == MOE_SLOT_HOST) {  // computed by the host tier, skipped by the kernels
                    plan.off[j] = -1;
                    s->host_blobs[size_t(n_host)] = moe::cache_host_blob(d.cache, l, s->ids_host[j]);
                    s->host_w[size_t(n_host)] = s->host_w[size_t(j)];  // (n_host <= j: compacting in place)
                    ++n_host;
                } else {
                    plan.off[j] = (long long)s->slots_host[j] * (long long)s->expert_bytes;
                }
            }
        } else if (!s->budgeted) {
            pool += size_t(l) * d.E * s->expert_bytes;
            slot_of = nullptr;
        }
        // One token with device lookups: the gate/up launch streams the lookup's misses itself (their rows
        // from the host store while the resident experts' gate/up runs), so no fill launch precedes it.
        moe::FfnPlan fplan;
        if (fused) {
            fplan.fill = moe::cache_ffn_fill(d.cache, (long long)moe::down_offset(d.H, d.I, d.w_dtype));
            fplan.rank_slot = s->dev_slots + size_t(l) * d.max_tokens * d.k;  // as the fused lookup wrote them
        }
        // the host tier starts on its share at once; the GPU's share (every rank when no host tier, none when
        // the host computes them all and there is no shared expert) is enqueued meanwhile, so that it and the
        // fills run while the host computes
        if (n_host > 0) {
            int st = moe::host_ffn_begin(s->host, s->h_pub, d.H, d.I, d.w_dtype, n_host, s->host_blobs.data(),
                                         s->host_w.data(), s->y_pub);
            if (st != MOE_OK) return st;
        }
        if (n_host < d.k || !s->shared_w.empty())
            e = moe::launch_expert_ffn(s->h, T, d.H, d.I, d.E, d.k, ids, w, slot_of, pool, s->expert_bytes, d.w_dtype,
                                       s->shared_w.empty() ? nullptr : s->shared_w[l], x, true, ws, eflags, strm,
                                       fused ? &fplan : plan.n ? &plan : nullptr);
        s->last[l] = LastLayer{true, T, l, ids, w, slot_of, pool, plan};
        if (n_host > 0) {
            const int st = moe::host_ffn_finish(s->host);  // (also when the launch failed: the tier must end)
            if (e != hipSuccess) return moe::fail_hip(e, "stack step: expert FFN");
            if (st != MOE_OK) return st;
            // x += the host's share; the next layer's top-k, which rewrites h_pub, runs after this on the stream
            e = moe::launch_add(x, s->y_pub_dev, d.H, strm);
            if (e != hipSuccess) return moe::fail_hip(e, "stack step: adding the host tier's output");
            ++s->host_calls;
        }
        if (e != hipSuccess) return moe::fail_hip(e, "stack step: expert FFN");
        if (s->budgeted && !dev_lookup) {
            int st = expert_cache_release(d.cache, strm);
            if (st == MOE_OK && d.prefetch > 0 && T == 1) st = prefetch_next(s, step, l);  // after the release
            if (st == MOE_OK && s->recalled >= 0 && T == 1 && l + 1 < d.n_layers) {
                // reverse rotation: bring back the recalled token's next-layer set ahead of demand
                const Snapshot &sn = s->snaps[size_t(s->recalled)];
                st = expert_cache_prefetch(d.cache, step, l + 1, sn.sets.data() + size_t(l + 1) * d.k, d.k);
            }
            if (st != MOE_OK) return st;
        }
    }
    if (s->budgeted && d.recall > 0 && T == 1 && !moe::cache_device(d.cache)) {
        store_snapshot(s);
        s->recalled = -1;
    }
    if (s->attn) s->last_attn_pos = s->attn_pos++;
    moe::clear_error();
    return MOE_OK;
}

}  // namespace

extern "C" {

int moe_stack_decode_step(moe_stack *s, int step, float *x, int T, const float *logit_bias,
                          int32_t *ids_out, float *weights_out, float *logits_out, void *stream) {
    if (!s || !x) return moe::fail(MOE_ERR_INVALID_ARG, "stack step: NULL argument");
    if (T < 1 || T > s->d.max_tokens)
        return moe::fail(MOE_ERR_INVALID_ARG, "stack step: T=%d outside [1, %d]", T, s->d.max_tokens);
    return enqueue_decode(s, step, x, T, logit_bias, ids_out, weights_out, logits_out,
                          static_cast<hipStream_t>(stream), nullptr);
}

int moe_stack_decode_graph(moe_stack *s, int step, float *x, const float *logit_bias, int32_t *ids_out,
                           float *weights_out, float *logits_out, void *stream) {
    if (!s || !x) return moe::fail(MOE_ERR_INVALID_ARG, "stack step: NULL argument");
    auto strm = static_cast<hipStream_t>(stream);
    if (!s->budgeted || !moe::cache_device(s->d.cache) || s->attn)  // host waits, or a moving position: no graph
        return enqueue_decode(s, step, x, 1, logit_bias, ids_out, weights_out, logits_out, strm, nullptr);
    const GraphKey key{x, logit_bias, ids_out, weights_out, logits_out};
    hipError_t e = hipSuccess;
    if (!s->graph_exec || !(s->graph_key == key)) {
        if (s->graph_exec) (void)hipGraphExecDestroy(s->graph_exec);
        s->graph_exec = nullptr;
        // capture on a private stream ordered after the caller's work; nothing is executed while capturing
        hipStream_t cs = nullptr;
        hipEvent_t ev = nullptr;
        hipGraph_t g = nullptr;
        e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventRecord(ev, strm);
        if (e == hipSuccess) e = hipStreamWaitEvent(cs, ev, 0);
        int st = MOE_OK;
        if (e == hipSuccess) e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
        if (e == hipSuccess) {
            st = enqueue_decode(s, step, x, 1, logit_bias, ids_out, weights_out, logits_out, cs, s->dev_step);
            hipError_t e2 = hipStreamEndCapture(cs, &g);
            if (e == hipSuccess) e = e2;
        }
        if (e == hipSuccess && st == MOE_OK) e = hipGraphInstantiate(&s->graph_exec, g, nullptr, nullptr, 0);
        if (g) (void)hipGraphDestroy(g);
        if (ev) (void)hipEventDestroy(ev);
        if (cs) (void)hipStreamDestroy(cs);
        if (st != MOE_OK) return st;
        if (e != hipSuccess) {
            s->graph_exec = nullptr;
            return moe::fail_hip(e, "stack graph: capture");
        }
        s->graph_key = key;
    }
    e = moe::launch_set_int(s->dev_step, step, strm);
    if (e == hipSuccess) e = hipGraphLaunch(s->graph_exec, strm);
    if (e != hipSuccess) return moe::fail_hip(e, "stack graph: replay");
    moe::clear_error();
    return MOE_OK;
}

int moe_stack_prefill(moe_stack *s, int step, float *x, int T, int32_t *ids_out, float *weights_out,
                      float *logits_out, void *stream) {
    if (!s || !x) return moe::fail(MOE_ERR_INVALID_ARG, "stack prefill: NULL argument");
    if (s->d.max_prefill_tokens < 1) return moe::fail(MOE_ERR_INVALID_ARG, "stack prefill: created without prefill");
    if (T < 1 || T > s->d.max_prefill_tokens)
        return moe::fail(MOE_ERR_INVALID_ARG, "stack prefill: T=%d outside [1, %d]", T, s->d.max_prefill_tokens);
    auto strm = static_cast<hipStream_t>(stream);
    int *eflags = moe::device_error_flags();
    if (!eflags) return moe::fail(MOE_ERR_HIP, "device error flags unavailable");
    const auto &d = s->d;
    const moe::PrefillWorkspace ws = moe::prefill_workspace(s->pws, T, d.k, d.E, d.H, d.I);
    // Device LRU residency, a chunk long enough to use nearly every expert (T k >= 8 E) and room for two
    // whole layers: each layer's experts are prefetched (decisions on this stream, fills on the cache's copy
    // stream) right after the previous layer's lookup, so that they stream in while that layer's expert FFN
    // and the next routing run.  The previous layer's experts hold the most recent stamps, and with 2 E
    // slots or more at least E slots are older, so no prefetch victim is a slot that FFN still reads.  (A
    // rotary hand may stop at any slot outside the step: rotary stacks do not pipeline.)
    const bool dev_lookup = s->budgeted && moe::cache_device(d.cache);
    const bool pipe = dev_lookup && s->all_experts && moe::cache_capacity(d.cache) >= 2 * d.E &&
                      size_t(T) * d.k >= size_t(8) * d.E && !moe::cache_rotary(d.cache);
    if (pipe) {
        int st = moe::cache_prefetch_device(d.cache, step, 0, s->all_experts, d.E, strm);
        if (st != MOE_OK) return st;
    }
    for (int l = 0; l < d.n_layers; ++l) {
        int32_t *ids = ids_out ? ids_out + size_t(l) * T * d.k : s->ids;
        float *w = weights_out ? weights_out + size_t(l) * T * d.k : s->weights;
        float *lg = logits_out ? logits_out + size_t(l) * T * d.E : s->logits;
        hipError_t e = moe::launch_router_logits(x, s->router_w[l], d.router_dtype, T, d.H, d.E, nullptr, lg, true,
                                                 s->h, strm);
        if (e == hipSuccess) e = moe::launch_topk_softmax(lg, T, d.E, d.k, ids, w, eflags, strm);
        if (e != hipSuccess) return moe::fail_hip(e, "stack prefill: routing");
        const int32_t *slot_of = s->slot_table + size_t(l) * d.E;
        const uint8_t *pool = static_cast<const uint8_t *>(s->pool);
        if (dev_lookup) {
            int st = expert_cache_lookup_device(d.cache, step, l, ids, T * d.k, nullptr, strm);
            if (st == MOE_OK && pipe && l + 1 < d.n_layers)
                st = moe::cache_prefetch_device(d.cache, step, l + 1, s->all_experts, d.E, strm);
            if (st != MOE_OK) return st;
        } else if (s->budgeted) {
            e = hipMemcpyAsync(s->ids_host, ids, sizeof(int32_t) * T * d.k, hipMemcpyDeviceToHost, strm);
            if (e == hipSuccess) e = hipEventRecord(s->ids_ready, strm);
            if (e == hipSuccess) e = hipEventSynchronize(s->ids_ready);
            if (e != hipSuccess) return moe::fail_hip(e, "stack prefill: ids to host");
            int st = expert_cache_lookup(d.cache, step, l, s->ids_host, T * d.k, s->slots_host, nullptr, strm);
            if (st != MOE_OK) return st;
        } else {
            pool += size_t(l) * d.E * s->expert_bytes;  // preloaded: expert e of layer l sits at slot l * E + e
            slot_of = nullptr;
        }
        e = moe::launch_prefill_ffn(s->h, T, d.H, d.I, d.E, d.k, ids, w, slot_of, pool, s->expert_bytes, d.w_dtype,
                                    s->shared_w.empty() ? nullptr : s->shared_w[l], x, true, ws, eflags, strm);
        if (e != hipSuccess) return moe::fail_hip(e, "stack prefill: expert FFN");
        if (s->budgeted && !dev_lookup) {
            int st = expert_cache_release(d.cache, strm);
            if (st != MOE_OK) return st;
        }
    }
    moe::clear_error();
    return MOE_OK;
}

int moe_stack_kernel_time(moe_stack *s, int which, int n, void *stream, double *mean_ms) {
    const bool same_set = which >= 8;  // flag: a preloaded stack's repeats keep the step's own experts
    if (same_set) which -= 8;
    if (!s || !mean_ms || which < 0 || which > 4 || n < 1 || (same_set && (which < 1 || which > 3)))
        return moe::fail(MOE_ERR_INVALID_ARG, "kernel_time: bad argument");
    if (which == 4 && (!s->attn || s->last_attn_pos < 0))
        return moe::fail(MOE_ERR_INVALID_ARG, "kernel_time: no attention block, or no decode step yet");
    for (const LastLayer &ll : s->last)
        if (!ll.valid) return moe::fail(MOE_ERR_INVALID_ARG, "kernel_time: no decode step has run yet");
    auto strm = static_cast<hipStream_t>(stream);
    int *eflags = moe::device_error_flags();
    if (!eflags) return moe::fail(MOE_ERR_HIP, "device error flags unavailable");
    const auto &d = s->d;
    const int L = d.n_layers, T = s->last[0].T;
    const moe::FfnWorkspace ws = moe::ffn_workspace(s->ws, T, d.k, d.I);
    // One token with device lookups: each layer's slots, as its lookup left them, become that layer's
    // launch plan, so that every re-launch reads the slots the step read (later layers may have evicted
    // some of them since, which only changes the bytes read, not where or how many).
    std::vector<moe::FfnPlan> plans(static_cast<size_t>(L));
    for (int l = 0; l < L; ++l) plans[size_t(l)] = s->last[size_t(l)].plan;
    if (s->budgeted && moe::cache_device(d.cache) && T == 1) {
        std::vector<int32_t> slots(size_t(L) * d.max_tokens * d.k);
        hipError_t e0 = hipStreamSynchronize(strm);
        if (e0 == hipSuccess)
            e0 = hipMemcpy(slots.data(), s->dev_slots, sizeof(int32_t) * slots.size(), hipMemcpyDeviceToHost);
        if (e0 != hipSuccess) return moe::fail_hip(e0, "kernel_time: reading the step's slots");
        for (int l = 0; l < L; ++l) {
            moe::FfnPlan &pl = plans[size_t(l)];
            pl.n = d.k;
            for (int j = 0; j < d.k; ++j)
                pl.off[j] = (long long)slots[size_t(l) * d.max_tokens * d.k + j] * (long long)s->expert_bytes;
        }
    }
    // Every layer's launch of the last step, in step order, captured into one
    // graph on a private stream (so that host launch overhead does not starve
    // the device) and replayed n times.  The last layer's normalised input
    // feeds every launch; results go to scratch.
    // Multi-token steps under a budget read the device slot table, where an
    // earlier layer's experts may have been evicted since: replay only the
    // last layer then (T == 1 steps carry their slots with them).
    const int l0 = (s->budgeted && T > 1) ? L - 1 : 0;
    // A graph of a few launches would time the graph launch, not the kernels:
    // each layer's launch is repeated until the graph holds at least 32.  In a
    // preloaded stack every expert of a layer is resident, so repeat r of an
    // expert launch reads experts (e + r) mod E of the step's experts e: the
    // launches then stream an E-expert working set (beyond the last-level
    // cache for the large layers) instead of re-reading the same few experts.
    const int reps = (32 + (L - l0) - 1) / (L - l0);
    const bool rotate = !s->budgeted && !same_set && which >= 1 && which <= 3 && reps > 1;
    std::vector<int32_t> rot_host;
    int32_t *rot_dev = nullptr;
    hipError_t e = hipSuccess;
    if (rotate) {
        // [rep][layer][T * k]
        const size_t nid = size_t(T) * d.k, nl = size_t(L - l0);
        rot_host.resize(nid * nl * size_t(reps));
        e = hipStreamSynchronize(strm);
        for (size_t l = 0; l < nl && e == hipSuccess; ++l)
            e = hipMemcpy(rot_host.data() + l * nid, s->last[size_t(l0) + l].ids, sizeof(int32_t) * nid,
                          hipMemcpyDeviceToHost);
        for (int r = 1; r < reps && e == hipSuccess; ++r)
            for (size_t j = 0; j < nl * nid; ++j) {
                const int32_t id = rot_host[j];  // invalid ids (outside [0, E)) stay as they are
                rot_host[size_t(r) * nl * nid + j] = id >= 0 && id < d.E ? (id + r) % d.E : id;
            }
        if (e == hipSuccess) e = hipMalloc(&rot_dev, sizeof(int32_t) * rot_host.size());
        if (e == hipSuccess)
            e = hipMemcpy(rot_dev, rot_host.data(), sizeof(int32_t) * rot_host.size(), hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            if (rot_dev) (void)hipFree(rot_dev);
            return moe::fail_hip(e, "kernel_time: rotated expert sets");
        }
    }
    hipStream_t cs = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    hipEvent_t a = nullptr, b = nullptr;
    e = hipMemcpyAsync(s->scratch_x, s->h, sizeof(float) * T * d.H, hipMemcpyDeviceToDevice, strm);
    if (e == hipSuccess) e = hipEventCreate(&a);
    if (e == hipSuccess) e = hipEventCreate(&b);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventRecord(a, strm);
    if (e == hipSuccess) e = hipStreamWaitEvent(cs, a, 0);
    auto enqueue = [&](const LastLayer &ll, int r) -> hipError_t {
        const int l = ll.layer;
        if (which == 4)
            return moe::launch_attention_decode(s->scratch_x, d.H, s->ad.n_heads, s->ad.n_kv, s->ad.head_dim,
                                                s->a_wqkv[l], s->a_wo[l], static_cast<uint16_t *>(s->a_k[l]),
                                                static_cast<uint16_t *>(s->a_v[l]), s->ad.max_pos, s->last_attn_pos,
                                                s->ad.theta, s->attn_ws, cs);
        if (which == 0) {
            hipError_t r = moe::launch_router_logits(s->scratch_x, s->router_w[l], d.router_dtype, T, d.H, d.E, nullptr,
                                                     s->logits, true, s->scratch_y, cs);
            return r == hipSuccess ? moe::launch_topk_softmax(s->logits, T, d.E, d.k, s->ids, s->weights, eflags, cs)
                                   : r;
        }
        const int32_t *ids = rotate ? rot_dev + (size_t(r) * (L - l0) + size_t(l - l0)) * T * d.k : ll.ids;
        return moe::launch_expert_ffn(s->scratch_x, T, d.H, d.I, d.E, d.k, ids, ll.weights, ll.slot_of, ll.pool,
                                      s->expert_bytes, d.w_dtype, s->shared_w.empty() ? nullptr : s->shared_w[l],
                                      s->scratch_y, false, ws, eflags, cs,
                                      plans[size_t(l)].n ? &plans[size_t(l)] : nullptr,
                                      which == 1 ? moe::kFfnGateUp : which == 2 ? moe::kFfnDown : moe::kFfnBoth);
    };
    if (e == hipSuccess) e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
    if (e == hipSuccess) {
        for (int r = 0; r < reps && e == hipSuccess; ++r)
            for (int l = l0; l < L && e == hipSuccess; ++l) e = enqueue(s->last[l], r);
        hipError_t e2 = hipStreamEndCapture(cs, &graph);
        if (e == hipSuccess) e = e2;
    }
    if (e == hipSuccess) e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    if (e == hipSuccess) e = hipGraphLaunch(exec, cs);  // warm
    if (e == hipSuccess) e = hipEventRecord(a, cs);
    for (int i = 0; i < n && e == hipSuccess; ++i) e = hipGraphLaunch(exec, cs);
    if (e == hipSuccess) e = hipEventRecord(b, cs);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
    if (cs) (void)hipStreamSynchronize(cs);
    if (exec) (void)hipGraphExecDestroy(exec);
    if (graph) (void)hipGraphDestroy(graph);
    if (cs) (void)hipStreamDestroy(cs);
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
    if (rot_dev) (void)hipFree(rot_dev);
    if (e != hipSuccess) return moe::fail_hip(e, "kernel_time");
    *mean_ms = double(ms) / (double(n) * reps * (L - l0));
    moe::clear_error();
    return MOE_OK;
}

}  // extern "C"
