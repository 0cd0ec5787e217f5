// residency.cpp -- expert slot table in HBM, LRU or rotary replacement.
//
// The paper's residency picture (sec. 4, Fig. 1): every sub-module (expert)
// lives in the host tier; the accelerator holds a fixed group of slots; a
// lookup table maps sub-module id to slot; missing sub-modules are brought in
// by a selective load after an eviction makes room; the whole runs inside a
// memory budget (sec. 5).  Replacement is at step granularity: a step's
// ascending unique experts are looked up in turn, and a miss never evicts an
// expert the same step needs.  LRU: one recency stamp per lookup, the least
// recent slot is the victim.  Rotary (sec. 4, Fig. 2: the slot group advances
// around a cycle): the slots form a ring with a hand; demand hits charge their
// slot (saturating at charge_max); a miss turns the hand forward past the
// step's own slots and past charged slots (each losing one charge) to the first
// uncharged slot.  The charges are this library's reading of how the paper's
// rotation is steered, which it does not disclose.
//
// Device ordering (per cache):
//   demand lookup : on the compute stream, after any earlier prefetch's fills:
//                   [H2D fills] [slot-table update], then the caller's FFN, then
//                   release() records the slots' last-reader event.  The fills
//                   need no wait for a victim read on the same stream (stream
//                   order already puts it first); a victim read on another
//                   stream is waited for unless its event has completed.
//   prefetch      : the same on the copy stream (waiting for the victims' last
//                   readers), ending in an event the next demand lookup waits on.
// Events come from a ring; an entry is synchronised before it is re-recorded,
// so a slot whose reader entry was recycled has provably finished being read.
#include <stdarg.h>
#include <string.h>

#include <algorithm>
#include <functional>
#include <queue>
#include <vector>

#include "internal.h"
#include "../../include/moe_budget.h"

namespace {

struct EvRef {
    int idx = -1;
    uint64_t gen = 0;
};

class EventRing {
  public:
    explicit EventRing(int n = 512) : ev_(n), gen_(n, 0) {}
    hipError_t init() {
        for (auto &e : ev_) {
            hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableTiming);
            if (r != hipSuccess) return r;
        }
        return hipSuccess;
    }
    void destroy() {
        for (auto &e : ev_)
            if (e) (void)hipEventDestroy(e);
    }
    hipError_t record(hipStream_t s, EvRef *out) {
        const int i = next_;
        next_ = (next_ + 1) % int(ev_.size());
        if (gen_[i]) {
            hipError_t r = hipEventSynchronize(ev_[i]);  // the old record must be complete before reuse
            if (r != hipSuccess) return r;
        }
        ++gen_[i];
        out->idx = i;
        out->gen = gen_[i];
        return hipEventRecord(ev_[i], s);
    }
    // True while the referenced record may still be outstanding.
    bool live(const EvRef &r) const { return r.idx >= 0 && gen_[r.idx] == r.gen; }
    hipEvent_t event(const EvRef &r) const { return ev_[r.idx]; }

  private:
    std::vector<hipEvent_t> ev_;
    std::vector<uint64_t> gen_;
    int next_ = 0;
};

}  // namespace

struct moe_cache {
    moe_cache_desc d{};
    int L = 0, E = 0, C = 0;
    bool sim = false;

    std::vector<int32_t> key_of_slot;  // layer*E + expert, -1 = free
    std::vector<int32_t> slot_of_key;  // host mirror of the device table [L*E]
    std::vector<int32_t> prev, next;   // LRU: recency list over slots, head = least recent
    int head = -1, tail = -1;
    bool rotary = false;
    int charge_max = 0;
    std::vector<uint16_t> charge;      // rotary: charge of each slot
    int hand = 0;                      // rotary: ring position the next rotation starts from
    std::priority_queue<int, std::vector<int>, std::greater<int>> free_slots;
    std::vector<uint64_t> step_mark;   // == epoch while the key is in the current step's set
    uint64_t epoch = 0;

    uint8_t *pool = nullptr;            // device (or host under sim) slots
    const uint8_t *host_dev = nullptr;  // device-side address of the pinned host store (fill kernels read it)
    int32_t *dev_slot_of = nullptr;     // device (or host under sim) table [L*E]
    hipStream_t copy = nullptr;
    EventRing ring;
    std::vector<EvRef> reader;          // last recorded reader of each slot
    std::vector<hipStream_t> reader_stream;  // the stream that reader ran on
    std::vector<int> unreleased;        // slots handed out by the last lookup
    hipStream_t last_compute = nullptr;
    bool have_last_compute = false;
    EvRef prefetch_done;                // copy-stream point after the latest prefetch's fills
    std::vector<std::pair<const uint8_t *, uint8_t *>> pending;  // fills placed by the current lookup

    std::vector<moe_cache_event> log;
    moe_cache_stats st{};

    // host tier (moe_cache_desc.host_layers / host_quota)
    int host_layers = 0, host_quota = 0;
    std::vector<uint8_t> host_prev;  // [L*E]: 1 if the host served the key at its layer's last demand lookup

    bool dev_mode = false;   // MOE_CACHE_DEVICE: decisions and log on the device
    int clk_khz = 0;         // MOE_CACHE_DEVICE: rate of the device wall clock the fill clock counts in
    moe::DevResidency dr;
    // MOE_CACHE_DEVICE prefetch: its decisions on the caller's stream, its fills on the copy stream
    hipEvent_t pf_issued = nullptr, pf_done = nullptr;
    bool pf_pending = false;  // a prefetch's fills may still run: the next lookup waits for pf_done
};

namespace {

void unlink(moe_cache *c, int s) {
    const int p = c->prev[s], n = c->next[s];
    if (p >= 0) c->next[p] = n; else c->head = n;
    if (n >= 0) c->prev[n] = p; else c->tail = p;
    c->prev[s] = c->next[s] = -1;
}

void push_recent(moe_cache *c, int s) {
    c->prev[s] = c->tail;
    c->next[s] = -1;
    if (c->tail >= 0) c->next[c->tail] = s; else c->head = s;
    c->tail = s;
}

int check_ids(moe_cache *c, int layer, const int32_t *ids, int n, std::vector<int32_t> *R) {
    if (!c) return moe::fail(MOE_ERR_INVALID_ARG, "cache is NULL");
    if (layer < 0 || layer >= c->L) return moe::fail(MOE_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, c->L);
    if (n < 0 || (n > 0 && !ids)) return moe::fail(MOE_ERR_INVALID_ARG, "bad id list (n=%d)", n);
    for (int i = 0; i < n; ++i)
        if (ids[i] < 0 || ids[i] >= c->E)
            return moe::fail(MOE_ERR_RANGE, "expert id %d outside [0, %d)", ids[i], c->E);
    R->assign(ids, ids + n);
    std::sort(R->begin(), R->end());
    R->erase(std::unique(R->begin(), R->end()), R->end());
    if (int(R->size()) > c->C)
        return moe::fail(MOE_ERR_BUDGET, "step needs %zu experts but only %d slots fit the budget", R->size(), c->C);
    return MOE_OK;
}

// Records the pending last-reader event for slots of the previous lookup.
int release_pending(moe_cache *c, hipStream_t s) {
    if (c->unreleased.empty()) return MOE_OK;
    if (!c->sim) {
        EvRef r;
        hipError_t e = c->ring.record(s, &r);
        if (e != hipSuccess) return moe::fail_hip(e, "recording slot release");
        for (int slot : c->unreleased) {
            c->reader[slot] = r;
            c->reader_stream[slot] = s;
        }
    }
    c->unreleased.clear();
    return MOE_OK;
}

const uint8_t *host_blob(const moe_cache *c, int layer, int expert) {
    return static_cast<const uint8_t *>(c->d.host_base) + size_t(layer) * c->d.host_layer_stride +
           size_t(expert) * c->d.host_expert_stride;
}

// Insert (layer, e) at a free or victim slot and queue its fill.  Returns the
// slot, or -1 with the error recorded.
int place_and_fill(moe_cache *c, int layer, int e, int32_t *victim, std::vector<int32_t> *chg_idx,
                   std::vector<int32_t> *chg_val, int *status, hipStream_t fill) {
    int s;
    *victim = -1;
    if (!c->free_slots.empty()) {
        s = c->free_slots.top();
        c->free_slots.pop();
    } else {
        if (c->rotary) {
            // Some slot holds an expert outside the step (the key being placed is not resident and the
            // step has at most C experts), and every full turn takes a charge from each such slot, so the
            // hand stops within (charge_max + 1) turns.
            for (;;) {
                s = c->hand;
                c->hand = c->hand + 1 == c->C ? 0 : c->hand + 1;
                if (c->step_mark[c->key_of_slot[s]] == c->epoch) continue;
                if (c->charge[s] > 0) {
                    --c->charge[s];
                    continue;
                }
                break;
            }
        } else {
            s = c->head;
            while (s >= 0 && c->step_mark[c->key_of_slot[s]] == c->epoch) s = c->next[s];
            if (s < 0) {  // unreachable while |R| <= C
                *status = moe::fail(MOE_ERR_BUDGET, "no evictable slot");
                return -1;
            }
            unlink(c, s);
        }
        *victim = c->key_of_slot[s];
        c->slot_of_key[*victim] = -1;
        chg_idx->push_back(*victim);
        chg_val->push_back(-1);
        ++c->st.evictions;
    }
    const int32_t key = layer * c->E + e;
    uint8_t *dst = c->pool + size_t(s) * c->d.expert_bytes;
    const uint8_t *src = host_blob(c, layer, e);
    if (c->sim) {
        memcpy(dst, src, c->d.expert_bytes);
    } else {
        if (c->ring.live(c->reader[s]) && c->reader_stream[s] != fill) {
            const hipEvent_t ev = c->ring.event(c->reader[s]);
            if (hipEventQuery(ev) != hipSuccess) {
                hipError_t r = hipStreamWaitEvent(fill, ev, 0);
                if (r != hipSuccess) *status = moe::fail_hip(r, "ordering fill after last reader");
            }
        }
        // copied by the lookup's fill kernels, which read the store through its device-side address
        c->pending.emplace_back(c->host_dev + (src - static_cast<const uint8_t *>(c->d.host_base)), dst);
    }
    c->key_of_slot[s] = key;
    c->slot_of_key[key] = s;
    chg_idx->push_back(key);
    chg_val->push_back(s);
    if (c->rotary) c->charge[s] = 0;
    else push_recent(c, s);
    c->st.h2d_bytes += c->d.expert_bytes;
    return s;
}

// Enqueues the lookup's fills and slot-table changes (last value per entry
// wins) on `strm`: kernels that stream the blobs from host memory into their
// slots and write the table entries; with `done`, records the event marking
// the end of that work.  Under HOST_SIM the fills were done in place.
int publish(moe_cache *c, std::vector<int32_t> &idx, std::vector<int32_t> &val, hipStream_t strm, EvRef *done) {
    std::vector<int32_t> ui, uv;
    for (size_t i = 0; i < idx.size(); ++i) {
        bool later = false;
        for (size_t j = i + 1; j < idx.size(); ++j)
            if (idx[j] == idx[i]) later = true;
        if (!later) {
            ui.push_back(idx[i]);
            uv.push_back(val[i]);
        }
    }
    if (c->sim) {
        for (size_t i = 0; i < ui.size(); ++i) c->dev_slot_of[ui[i]] = uv[i];
        return MOE_OK;
    }
    const size_t nf = c->pending.size();
    const size_t nb = (nf + moe::kMaxFillBatch - 1) / moe::kMaxFillBatch;
    size_t t = 0;
    hipError_t e = hipSuccess;
    for (size_t b = 0; b < nb && e == hipSuccess; ++b) {
        moe::FillBatch fb;
        fb.bytes = (long long)c->d.expert_bytes;
        fb.table = c->dev_slot_of;
        for (size_t i = b * moe::kMaxFillBatch; i < nf && fb.n < moe::kMaxFillBatch; ++i, ++fb.n) {
            fb.src[fb.n] = c->pending[i].first;
            fb.dst[fb.n] = c->pending[i].second;
        }
        // table entries: an even share per batch, the rest with the last batch
        const size_t share = b + 1 == nb ? ui.size() - t : std::min(ui.size() - t, size_t(2 * moe::kMaxFillBatch));
        for (size_t j = 0; j < share && fb.n_tab < 2 * moe::kMaxFillBatch; ++j, ++t, ++fb.n_tab) {
            fb.tab_idx[fb.n_tab] = ui[t];
            fb.tab_val[fb.n_tab] = uv[t];
        }
        e = moe::launch_fill_slots(fb, strm);
    }
    if (e == hipSuccess && t < ui.size())  // more changes than the batches carry (not expected)
        e = moe::launch_slot_update(c->dev_slot_of, ui.data() + t, uv.data() + t, int(ui.size() - t), strm);
    c->pending.clear();
    if (e != hipSuccess) {
        // the lookup's placements stay unmapped, so that a retry misses again
        for (size_t i = 0; i < idx.size(); ++i) {
            if (val[i] < 0 || c->key_of_slot[val[i]] != idx[i]) continue;
            c->slot_of_key[idx[i]] = -1;
            c->key_of_slot[val[i]] = -1;
            unlink(c, val[i]);
            c->free_slots.push(val[i]);
        }
        return moe::fail(MOE_ERR_COPY, "expert fill launch failed: %s", hipGetErrorString(e));
    }
    if (done) {
        e = c->ring.record(strm, done);
        if (e != hipSuccess) return moe::fail_hip(e, "recording fill event");
    }
    return MOE_OK;
}

int lookup_impl(moe_cache *c, int step, int layer, const int32_t *ids, int n, bool prefetch,
                int32_t *slots_out, uint8_t *hit_out, hipStream_t compute) {
    std::vector<int32_t> R;
    int st = check_ids(c, layer, ids, n, &R);
    if (st != MOE_OK) return st;
    moe::clear_error();
    if (c->have_last_compute) {
        st = release_pending(c, c->last_compute);
        if (st != MOE_OK) return st;
    }
    const hipStream_t fill = prefetch ? c->copy : compute;
    if (!prefetch && !c->sim && c->ring.live(c->prefetch_done)) {
        // earlier prefetches' fills and table updates land before this lookup's fills and compute:
        // a hit may be one of them, and a victim may be a prefetched slot still being filled
        hipError_t e = hipStreamWaitEvent(compute, c->ring.event(c->prefetch_done), 0);
        if (e != hipSuccess) return moe::fail_hip(e, "ordering compute after prefetch");
        c->prefetch_done = EvRef{};
    }
    ++c->epoch;
    for (int e : R) c->step_mark[layer * c->E + e] = c->epoch;
    std::vector<int32_t> chg_idx, chg_val;
    std::vector<uint8_t> hit_of(R.size(), 0);
    // The host tier's share of a demand lookup: the whole step in a host layer; otherwise the non-resident
    // experts the host served at this layer's previous demand lookup, then more in ascending order while
    // fewer than host_quota are served.
    std::vector<uint8_t> to_host(R.size(), 0);
    if (!prefetch && (c->host_layers > 0 || c->host_quota > 0)) {
        uint8_t *prev = c->host_prev.data() + size_t(layer) * c->E;
        if (layer < c->host_layers) {
            std::fill(to_host.begin(), to_host.end(), uint8_t(1));
        } else {
            int served = 0;
            for (size_t r = 0; r < R.size(); ++r)
                if (c->slot_of_key[layer * c->E + R[r]] < 0 && prev[R[r]]) {
                    to_host[r] = 1;
                    ++served;
                }
            for (size_t r = 0; r < R.size() && served < c->host_quota; ++r)
                if (!to_host[r] && c->slot_of_key[layer * c->E + R[r]] < 0) {
                    to_host[r] = 1;
                    ++served;
                }
        }
        std::fill(prev, prev + c->E, uint8_t(0));
        for (size_t r = 0; r < R.size(); ++r) prev[R[r]] = to_host[r];
    }
    st = MOE_OK;
    for (size_t r = 0; r < R.size(); ++r) {
        const int e = R[r];
        const int32_t key = layer * c->E + e;
        if (to_host[r]) {
            ++c->st.host_computed;
            ++c->st.lookups;
            c->log.push_back({step, layer, e, MOE_EVENT_HOST, -1, -1});
            continue;
        }
        int s = c->slot_of_key[key];
        if (s >= 0) {
            if (prefetch) continue;  // a prefetch leaves resident experts untouched
            if (c->rotary) {
                if (c->charge[s] < c->charge_max) ++c->charge[s];
            } else {
                unlink(c, s);
                push_recent(c, s);
            }
            ++c->st.hits;
            ++c->st.lookups;
            hit_of[r] = 1;
            c->log.push_back({step, layer, e, MOE_EVENT_HIT, s, -1});
            continue;
        }
        int32_t victim;
        s = place_and_fill(c, layer, e, &victim, &chg_idx, &chg_val, &st, fill);
        if (s < 0) break;
        if (prefetch) {
            ++c->st.prefetches;
        } else {
            ++c->st.misses;
            ++c->st.lookups;
        }
        c->log.push_back({step, layer, e, prefetch ? MOE_EVENT_PREFETCH : MOE_EVENT_MISS, s, victim});
    }
    if (!chg_idx.empty()) {
        EvRef done;
        int pst = publish(c, chg_idx, chg_val, fill, prefetch ? &done : nullptr);
        if (pst != MOE_OK && st == MOE_OK) st = pst;
        if (!c->sim && pst == MOE_OK && prefetch) c->prefetch_done = done;
    }
    if (!prefetch) {
        for (int e : R) {
            const int s = c->slot_of_key[layer * c->E + e];
            if (s >= 0) c->unreleased.push_back(s);
        }
        c->last_compute = compute;
        c->have_last_compute = true;
        for (int i = 0; i < n; ++i) {
            const size_t r = size_t(std::lower_bound(R.begin(), R.end(), ids[i]) - R.begin());
            if (slots_out) slots_out[i] = to_host[r] ? MOE_SLOT_HOST : c->slot_of_key[layer * c->E + ids[i]];
            if (hit_out) hit_out[i] = hit_of[r];
        }
    }
    return st;
}

}  // namespace

size_t moe::cache_expert_bytes(const moe_cache *c) { return c->d.expert_bytes; }
bool moe::cache_preloaded(const moe_cache *c) { return c->d.flags & MOE_CACHE_PRELOAD; }
bool moe::cache_resident(const moe_cache *c, int layer, int expert) {
    return c->slot_of_key[size_t(layer) * c->E + expert] >= 0;
}
bool moe::cache_device(const moe_cache *c) { return c->dev_mode; }
int moe::cache_capacity(const moe_cache *c) { return c->C; }
bool moe::cache_rotary(const moe_cache *c) { return c->d.policy == MOE_POLICY_ROTARY; }
bool moe::cache_host_tier(const moe_cache *c) { return c->host_layers > 0 || c->host_quota > 0; }
const uint8_t *moe::cache_host_blob(const moe_cache *c, int layer, int expert) { return host_blob(c, layer, expert); }

namespace {
// A device lookup rewrites the fill list and may evict: an earlier device prefetch's fills come first.
hipError_t after_device_prefetch(moe_cache *c, hipStream_t s) {
    if (!c->pf_pending) return hipSuccess;
    c->pf_pending = false;
    return hipStreamWaitEvent(s, c->pf_done, 0);
}
}  // namespace

int moe::cache_prefetch_device(moe_cache *c, int step, int layer, const int32_t *ids_dev, int n, hipStream_t s) {
    if (!c || !c->dev_mode || layer < 0 || layer >= c->L || n < 0 || (n > 0 && !ids_dev))
        return moe::fail(MOE_ERR_INVALID_ARG, "device prefetch needs a MOE_CACHE_DEVICE cache, a valid layer and ids");
    if (n == 0) return MOE_OK;
    int *err = moe::device_error_flags();
    if (!err) return moe::fail(MOE_ERR_HIP, "device error flags unavailable");
    moe::DevLookup p{c->C, c->L, c->E, layer, step, c->d.policy == MOE_POLICY_ROTARY ? 1 : 0, c->charge_max,
                     (long long)c->d.host_layer_stride, (long long)c->d.host_expert_stride};
    p.prefetch = 1;
    hipError_t e = after_device_prefetch(c, s);
    if (e == hipSuccess) e = moe::launch_dev_lookup(c->dr, p, ids_dev, n, nullptr, err, s);
    // the fills go to the copy stream, so that work the caller queues next on `s` overlaps them
    if (e == hipSuccess) e = hipEventRecord(c->pf_issued, s);
    if (e == hipSuccess) e = hipStreamWaitEvent(c->copy, c->pf_issued, 0);
    if (e == hipSuccess)
        e = moe::launch_dev_fill(c->dr, c->host_dev, c->pool, (long long)c->d.expert_bytes, std::min(n, c->E),
                                 c->copy, false);
    if (e == hipSuccess) e = hipEventRecord(c->pf_done, c->copy);
    if (e != hipSuccess) return moe::fail_hip(e, "device prefetch");
    c->pf_pending = true;
    return MOE_OK;
}

moe::FfnFill moe::cache_ffn_fill(moe_cache *c, long long down_off) {
    moe::FfnFill f;
    f.clk = c->dr.clk;
    f.n = c->dr.n_fill;
    f.src = c->dr.fill_src;
    f.slot = c->dr.fill_slot;
    f.host = c->host_dev;
    f.pool = c->pool;
    f.doff = down_off;
    return f;
}

int moe::cache_topk_lookup(moe_cache *c, int step, int layer, const float *logits, int k, int32_t *ids,
                           float *weights, int32_t *slots_out, int *err_flags, hipStream_t s, const int *step_dev,
                           bool fill_in_ffn) {
    if (!c || !c->dev_mode || layer < 0 || layer >= c->L)
        return moe::fail(MOE_ERR_INVALID_ARG, "fused top-k lookup needs a MOE_CACHE_DEVICE cache and a valid layer");
    moe::DevLookup p{c->C, c->L, c->E, layer, step, c->d.policy == MOE_POLICY_ROTARY ? 1 : 0, c->charge_max,
                     (long long)c->d.host_layer_stride, (long long)c->d.host_expert_stride, step_dev};
    hipError_t e = after_device_prefetch(c, s);
    if (e == hipSuccess) e = moe::launch_topk_lookup(logits, c->E, k, ids, weights, err_flags, c->dr, p, slots_out, s);
    if (e == hipSuccess && !fill_in_ffn)
        e = moe::launch_dev_fill(c->dr, c->host_dev, c->pool, (long long)c->d.expert_bytes, std::min(k, c->E), s);
    return e == hipSuccess ? MOE_OK : moe::fail_hip(e, "fused top-k lookup");
}

namespace {
constexpr long long kDevEvents = 1 << 21;

// Device state of a MOE_CACHE_DEVICE cache, initialised like the host state.
int dev_state_create(moe_cache *c, bool preload) {
    moe::DevResidency &r = c->dr;
    const size_t C = size_t(c->C);
    hipError_t e = hipMalloc(&r.key_of_slot, sizeof(int32_t) * C);
    if (e == hipSuccess) e = hipMalloc(&r.stamp, sizeof(uint64_t) * C);
    if (e == hipSuccess) e = hipMalloc(&r.charge, sizeof(uint16_t) * C);
    if (e == hipSuccess) e = hipMalloc(&r.scal, sizeof(unsigned long long) * moe::kDevScalars);
    if (e == hipSuccess) e = hipMalloc(&r.events, sizeof(moe_cache_event) * size_t(kDevEvents));
    if (e == hipSuccess) e = hipMalloc(&r.fill_src, sizeof(long long) * size_t(c->E));
    if (e == hipSuccess) e = hipMalloc(&r.fill_slot, sizeof(int32_t) * size_t(c->E));
    if (e == hipSuccess) e = hipMalloc(&r.n_fill, sizeof(int32_t));
    // the fill clock costs its launches a few microseconds (stamps, atomics, the fold): only when asked for
    if (e == hipSuccess && (c->d.flags & MOE_CACHE_FILL_CLOCK))
        e = hipMalloc(&r.clk, sizeof(unsigned long long) * moe::kClkWords);
    if (e != hipSuccess) return moe::fail_hip(e, "allocating the device residency state");
    int dev = 0, khz = 0;
    if ((e = hipGetDevice(&dev)) == hipSuccess)
        e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (e != hipSuccess || khz <= 0) return moe::fail_hip(e, "reading the device wall-clock rate");
    c->clk_khz = khz;
    r.cap_events = kDevEvents;
    r.slot_of_key = c->dev_slot_of;
    std::vector<uint64_t> stamp(C, 0);
    std::vector<unsigned long long> scal(moe::kDevScalars, 0);
    if (preload) {
        for (size_t s = 0; s < C; ++s) stamp[s] = s + 1;  // preloaded in slot order, as the oracle's stamps
        scal[moe::kScalCtr] = C;
        scal[moe::kScalNextFree] = C;
    }
    std::vector<uint16_t> charge(C, 0);
    e = hipMemcpy(r.key_of_slot, c->key_of_slot.data(), sizeof(int32_t) * C, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(r.stamp, stamp.data(), sizeof(uint64_t) * C, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(r.charge, charge.data(), sizeof(uint16_t) * C, hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemcpy(r.scal, scal.data(), sizeof(unsigned long long) * scal.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(r.n_fill, 0, sizeof(int32_t));
    std::vector<unsigned long long> clk(moe::kClkWords, 0ull);
    for (int i = 0; i < moe::kClkLanes; ++i) clk[size_t(moe::kClkFillStart + i)] = ~0ull;
    if (e == hipSuccess && r.clk)
        e = hipMemcpy(r.clk, clk.data(), sizeof(unsigned long long) * clk.size(), hipMemcpyHostToDevice);
    return e == hipSuccess ? MOE_OK : moe::fail_hip(e, "initialising the device residency state");
}

void dev_state_destroy(moe_cache *c) {
    moe::DevResidency &r = c->dr;
    for (void *p : {static_cast<void *>(r.key_of_slot), static_cast<void *>(r.stamp), static_cast<void *>(r.charge),
                    static_cast<void *>(r.scal), static_cast<void *>(r.events), static_cast<void *>(r.fill_src),
                    static_cast<void *>(r.fill_slot), static_cast<void *>(r.n_fill), static_cast<void *>(r.clk)})
        if (p) (void)hipFree(p);
    r = moe::DevResidency{};
}
}  // namespace

extern "C" {

int expert_cache_create(const moe_cache_desc *d, moe_cache **out) {
    if (!d || !out) return moe::fail(MOE_ERR_INVALID_ARG, "NULL descriptor or output");
    *out = nullptr;
    if (d->n_layers < 1 || d->n_experts < 1 || d->expert_bytes == 0)
        return moe::fail(MOE_ERR_INVALID_ARG, "n_layers, n_experts and expert_bytes must be positive");
    if (d->expert_bytes % 256)
        return moe::fail(MOE_ERR_INVALID_ARG, "expert_bytes (%zu) must be a multiple of 256", d->expert_bytes);
    if (d->policy != MOE_POLICY_LRU && d->policy != MOE_POLICY_ROTARY)
        return moe::fail(MOE_ERR_INVALID_ARG, "unknown policy %d", d->policy);
    if (d->policy == MOE_POLICY_ROTARY && (d->charge_max < 0 || d->charge_max > 65535))
        return moe::fail(MOE_ERR_INVALID_ARG, "charge_max (%d) must be in [0, 65535]", d->charge_max);
    if (!d->host_base) return moe::fail(MOE_ERR_INVALID_ARG, "host_base is NULL");
    if (d->reserved_bytes > d->budget_bytes)
        return moe::fail(MOE_ERR_BUDGET, "reserved bytes exceed the budget");
    const size_t cap = (d->budget_bytes - d->reserved_bytes) / d->expert_bytes;
    const size_t keys = size_t(d->n_layers) * d->n_experts;
    if (cap < 1) return moe::fail(MOE_ERR_BUDGET, "budget holds no expert slot");
    const bool preload = d->flags & MOE_CACHE_PRELOAD;
    if (preload && cap < keys)
        return moe::fail(MOE_ERR_BUDGET, "preload needs %zu slots, the budget holds %zu", keys, cap);
    if (keys > size_t(INT32_MAX)) return moe::fail(MOE_ERR_INVALID_ARG, "too many experts");

    const bool dev_mode = d->flags & MOE_CACHE_DEVICE;
    const bool host_tier = d->host_layers != 0 || d->host_quota != 0;
    if (d->host_layers < 0 || d->host_layers > d->n_layers || d->host_quota < 0 || d->host_quota > d->n_experts)
        return moe::fail(MOE_ERR_INVALID_ARG, "host tier: host_layers %d / host_quota %d outside [0, L] / [0, E]",
                         d->host_layers, d->host_quota);
    if (host_tier && (d->flags & (MOE_CACHE_DEVICE | MOE_CACHE_PRELOAD)))
        return moe::fail(MOE_ERR_INVALID_ARG, "host tier: not with MOE_CACHE_DEVICE or MOE_CACHE_PRELOAD");
    if ((d->flags & MOE_CACHE_FILL_CLOCK) && !dev_mode)
        return moe::fail(MOE_ERR_INVALID_ARG, "MOE_CACHE_FILL_CLOCK needs MOE_CACHE_DEVICE");
    if (dev_mode && (d->flags & MOE_CACHE_HOST_SIM))
        return moe::fail(MOE_ERR_INVALID_ARG, "MOE_CACHE_DEVICE cannot be combined with MOE_CACHE_HOST_SIM");
    if (dev_mode && (std::min(cap, preload ? keys : cap) > size_t(moe::kDevMaxSlots) || d->n_experts > MOE_MAX_EXPERTS))
        return moe::fail(MOE_ERR_INVALID_ARG, "MOE_CACHE_DEVICE needs at most %d slots and %d experts per layer",
                         moe::kDevMaxSlots, MOE_MAX_EXPERTS);

    auto *c = new moe_cache();
    c->d = *d;
    c->dev_mode = dev_mode;
    c->L = d->n_layers;
    c->E = d->n_experts;
    c->C = int(std::min(cap, preload ? keys : cap));
    c->sim = d->flags & MOE_CACHE_HOST_SIM;
    c->key_of_slot.assign(c->C, -1);
    c->slot_of_key.assign(keys, -1);
    c->prev.assign(c->C, -1);
    c->next.assign(c->C, -1);
    c->step_mark.assign(keys, 0);
    c->reader.assign(c->C, EvRef{});
    c->reader_stream.assign(c->C, nullptr);
    c->st.capacity = c->C;
    c->rotary = d->policy == MOE_POLICY_ROTARY;
    c->charge_max = c->rotary ? d->charge_max : 0;
    c->charge.assign(c->C, 0);
    c->host_layers = d->host_layers;
    c->host_quota = d->host_quota;
    if (host_tier) c->host_prev.assign(keys, 0);

    auto cleanup = [&](int code) {
        expert_cache_destroy(c);
        return code;
    };
    const size_t pool_bytes = size_t(c->C) * d->expert_bytes;
    if (c->sim) {
        c->pool = static_cast<uint8_t *>(malloc(pool_bytes));
        c->dev_slot_of = static_cast<int32_t *>(malloc(sizeof(int32_t) * keys));
        if (!c->pool || !c->dev_slot_of) return cleanup(moe::fail(MOE_ERR_INVALID_ARG, "host allocation failed"));
        for (size_t i = 0; i < keys; ++i) c->dev_slot_of[i] = -1;
    } else {
        hipPointerAttribute_t attr;
        hipError_t e = hipPointerGetAttributes(&attr, d->host_base);
        if (e != hipSuccess || attr.type != hipMemoryTypeHost) {
            (void)hipGetLastError();
            delete c;
            return moe::fail(MOE_ERR_NOT_PINNED, "host store is not page-locked memory");
        }
        void *hd = nullptr;
        if ((e = hipHostGetDevicePointer(&hd, const_cast<void *>(d->host_base), 0)) != hipSuccess || !hd) {
            (void)hipGetLastError();
            delete c;
            return moe::fail(MOE_ERR_NOT_PINNED, "host store has no device mapping (allocate it with hipHostMalloc)");
        }
        c->host_dev = static_cast<const uint8_t *>(hd);
        if ((e = hipMalloc(&c->pool, pool_bytes)) != hipSuccess)
            return cleanup(moe::fail_hip(e, "allocating the slot pool"));
        if ((e = hipMalloc(&c->dev_slot_of, sizeof(int32_t) * keys)) != hipSuccess)
            return cleanup(moe::fail_hip(e, "allocating the slot table"));
        if ((e = hipMemset(c->dev_slot_of, 0xff, sizeof(int32_t) * keys)) != hipSuccess)
            return cleanup(moe::fail_hip(e, "clearing the slot table"));
        if ((e = hipStreamCreateWithFlags(&c->copy, hipStreamNonBlocking)) != hipSuccess)
            return cleanup(moe::fail_hip(e, "creating the copy stream"));
        if ((e = c->ring.init()) != hipSuccess) return cleanup(moe::fail_hip(e, "creating events"));
        if (dev_mode && ((e = hipEventCreateWithFlags(&c->pf_issued, hipEventDisableTiming)) != hipSuccess ||
                         (e = hipEventCreateWithFlags(&c->pf_done, hipEventDisableTiming)) != hipSuccess))
            return cleanup(moe::fail_hip(e, "creating events"));
    }
    if (preload) {
        for (int l = 0; l < c->L; ++l)
            for (int e = 0; e < c->E; ++e) {
                const int s = l * c->E + e;
                uint8_t *dst = c->pool + size_t(s) * d->expert_bytes;
                if (c->sim) {
                    memcpy(dst, host_blob(c, l, e), d->expert_bytes);
                } else {
                    hipError_t r = hipMemcpyAsync(dst, host_blob(c, l, e), d->expert_bytes,
                                                  hipMemcpyHostToDevice, c->copy);
                    if (r != hipSuccess) return cleanup(moe::fail_hip(r, "preloading experts"));
                }
                c->key_of_slot[s] = s;
                c->slot_of_key[s] = s;
                if (!c->rotary) push_recent(c, s);
            }
        if (c->sim) {
            for (size_t i = 0; i < keys; ++i) c->dev_slot_of[i] = int32_t(i);
        } else {
            hipError_t r = hipMemcpyAsync(c->dev_slot_of, c->slot_of_key.data(), sizeof(int32_t) * keys,
                                          hipMemcpyHostToDevice, c->copy);
            if (r == hipSuccess) r = hipStreamSynchronize(c->copy);
            if (r != hipSuccess) return cleanup(moe::fail_hip(r, "preloading experts"));
        }
    } else {
        for (int s = 0; s < c->C; ++s) c->free_slots.push(s);
    }
    if (c->dev_mode) {
        const int st = dev_state_create(c, preload);
        if (st != MOE_OK) return cleanup(st);
    }
    *out = c;
    return MOE_OK;
}

int expert_cache_destroy(moe_cache *c) {
    if (!c) return MOE_OK;
    if (c->sim) {
        free(c->pool);
        free(c->dev_slot_of);
    } else {
        if (c->copy) (void)hipStreamSynchronize(c->copy);
        if (c->have_last_compute) (void)hipStreamSynchronize(c->last_compute);
        c->ring.destroy();
        dev_state_destroy(c);
        if (c->pf_issued) (void)hipEventDestroy(c->pf_issued);
        if (c->pf_done) (void)hipEventDestroy(c->pf_done);
        if (c->copy) (void)hipStreamDestroy(c->copy);
        if (c->pool) (void)hipFree(c->pool);
        if (c->dev_slot_of) (void)hipFree(c->dev_slot_of);
    }
    delete c;
    return MOE_OK;
}

int expert_cache_lookup_device(moe_cache *c, int step, int layer, const int32_t *ids_dev, int n,
                               int32_t *slots_out_dev, void *stream) {
    if (!c) return moe::fail(MOE_ERR_INVALID_ARG, "cache is NULL");
    if (!c->dev_mode) return moe::fail(MOE_ERR_INVALID_ARG, "device lookups need a MOE_CACHE_DEVICE cache");
    if (layer < 0 || layer >= c->L) return moe::fail(MOE_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, c->L);
    if (n < 0 || (n > 0 && !ids_dev)) return moe::fail(MOE_ERR_INVALID_ARG, "bad ids");
    if (n == 0) return MOE_OK;
    int *err = moe::device_error_flags();
    if (!err) return moe::fail(MOE_ERR_HIP, "device error flags unavailable");
    moe::DevLookup p{c->C, c->L, c->E, layer, step, c->d.policy == MOE_POLICY_ROTARY ? 1 : 0, c->charge_max,
                     (long long)c->d.host_layer_stride, (long long)c->d.host_expert_stride};
    auto s = static_cast<hipStream_t>(stream);
    hipError_t e = after_device_prefetch(c, s);
    if (e == hipSuccess) e = moe::launch_dev_lookup(c->dr, p, ids_dev, n, slots_out_dev, err, s);
    if (e == hipSuccess)
        e = moe::launch_dev_fill(c->dr, c->host_dev, c->pool, (long long)c->d.expert_bytes, std::min(n, c->E), s);
    if (e != hipSuccess) return moe::fail_hip(e, "device lookup");
    moe::clear_error();
    return MOE_OK;
}

int expert_cache_prefetch_device(moe_cache *c, int step, int layer, const int32_t *ids_dev, int n, void *stream) {
    if (!c) return moe::fail(MOE_ERR_INVALID_ARG, "cache is NULL");
    if (!c->dev_mode) return moe::fail(MOE_ERR_INVALID_ARG, "device prefetches need a MOE_CACHE_DEVICE cache");
    if (layer < 0 || layer >= c->L) return moe::fail(MOE_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, c->L);
    if (n < 0 || (n > 0 && !ids_dev)) return moe::fail(MOE_ERR_INVALID_ARG, "bad ids");
    const int st = moe::cache_prefetch_device(c, step, layer, ids_dev, n, static_cast<hipStream_t>(stream));
    if (st == MOE_OK) moe::clear_error();
    return st;
}

int expert_cache_lookup(moe_cache *c, int step, int layer, const int32_t *ids_host, int n,
                        int32_t *slots_out, uint8_t *hit_out, void *compute_stream) {
    if (c && c->dev_mode) return moe::fail(MOE_ERR_INVALID_ARG, "a MOE_CACHE_DEVICE cache looks up on the device");
    return lookup_impl(c, step, layer, ids_host, n, false, slots_out, hit_out,
                       static_cast<hipStream_t>(compute_stream));
}

int expert_cache_prefetch(moe_cache *c, int step, int layer, const int32_t *ids_host, int n) {
    if (c && c->dev_mode) return moe::fail(MOE_ERR_INVALID_ARG, "a MOE_CACHE_DEVICE cache prefetches on the device (expert_cache_prefetch_device)");
    return lookup_impl(c, step, layer, ids_host, n, true, nullptr, nullptr, nullptr);
}

int expert_cache_release(moe_cache *c, void *compute_stream) {
    if (!c) return moe::fail(MOE_ERR_INVALID_ARG, "cache is NULL");
    if (c->dev_mode) return MOE_OK;  // one stream orders every fill after the earlier readers
    return release_pending(c, static_cast<hipStream_t>(compute_stream));
}

int expert_cache_slot_table(moe_cache *c, const int32_t **dev_slot_of, const void **pool) {
    if (!c) return moe::fail(MOE_ERR_INVALID_ARG, "cache is NULL");
    if (dev_slot_of) *dev_slot_of = c->dev_slot_of;
    if (pool) *pool = c->pool;
    return MOE_OK;
}

int expert_cache_stats(moe_cache *c, moe_cache_stats *out) {
    if (!c || !out) return moe::fail(MOE_ERR_INVALID_ARG, "NULL argument");
    if (c->dev_mode) {
        unsigned long long v[moe::kDevScalars];
        hipError_t e = hipDeviceSynchronize();
        if (e == hipSuccess) e = hipMemcpy(v, c->dr.scal, sizeof v, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return moe::fail_hip(e, "reading device residency counters");
        *out = moe_cache_stats{};
        out->hits = v[moe::kScalHits];
        out->misses = v[moe::kScalMisses];
        out->prefetches = v[moe::kScalPrefetches];
        out->lookups = out->hits + out->misses;
        out->evictions = v[moe::kScalEvictions];
        out->h2d_bytes = (out->misses + out->prefetches) * c->d.expert_bytes;
        out->capacity = c->C;
        out->occupancy = int32_t(std::min<unsigned long long>(v[moe::kScalNextFree], (unsigned long long)c->C));
        // fill clock: the folded totals plus the record of the last filling launch, not folded yet
        unsigned long long k[moe::kClkWords] = {};
        for (int i = 0; i < moe::kClkLanes; ++i) k[moe::kClkFillStart + i] = ~0ull;
        if (c->dr.clk && (e = hipMemcpy(k, c->dr.clk, sizeof k, hipMemcpyDeviceToHost)) != hipSuccess)
            return moe::fail_hip(e, "reading the fill clock");
        unsigned long long stall = k[moe::kClkStall], fill = k[moe::kClkFill];
        unsigned long long fs = ~0ull, fe = 0, ce = 0;
        for (int i = 0; i < moe::kClkLanes; ++i) {
            fs = std::min(fs, k[moe::kClkFillStart + i]);
            fe = std::max(fe, k[moe::kClkFillEnd + i]);
            ce = std::max(ce, k[moe::kClkComputeEnd + i]);
        }
        if (fe > 0 && fe > fs) {
            const unsigned long long from = std::max(fs, ce);
            if (fe > from) stall += fe - from;
            fill += fe - fs;
        }
        const double ns_per_tick = 1.0e6 / double(c->clk_khz);
        out->stall_ns = uint64_t(double(stall) * ns_per_tick + 0.5);
        out->fill_ns = uint64_t(double(fill) * ns_per_tick + 0.5);
        return MOE_OK;
    }
    *out = c->st;
    int occ = 0;
    for (int32_t k : c->key_of_slot) occ += k >= 0;
    out->occupancy = occ;
    return MOE_OK;
}

int expert_cache_trace(moe_cache *c, size_t first, moe_cache_event *buf, size_t cap, size_t *n_out) {
    if (!c || !n_out || (cap && !buf)) return moe::fail(MOE_ERR_INVALID_ARG, "NULL argument");
    if (c->dev_mode) {
        unsigned long long n_ev = 0;
        hipError_t e = hipDeviceSynchronize();
        if (e == hipSuccess)
            e = hipMemcpy(&n_ev, c->dr.scal + moe::kScalEvents, sizeof n_ev, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return moe::fail_hip(e, "reading the device decision log");
        if (n_ev > (unsigned long long)c->dr.cap_events)
            return moe::fail(MOE_ERR_INVALID_ARG, "the device decision log overflowed (%llu > %lld decisions)", n_ev,
                             c->dr.cap_events);
        size_t n = 0;
        if (first < n_ev) n = std::min<size_t>(cap, size_t(n_ev) - first);
        if (n && (e = hipMemcpy(buf, c->dr.events + first, n * sizeof(moe_cache_event), hipMemcpyDeviceToHost)) !=
                     hipSuccess)
            return moe::fail_hip(e, "reading the device decision log");
        *n_out = n;
        return MOE_OK;
    }
    size_t n = 0;
    if (first < c->log.size()) n = std::min(cap, c->log.size() - first);
    if (n) memcpy(buf, c->log.data() + first, n * sizeof(moe_cache_event));
    *n_out = n;
    return MOE_OK;
}

}  // extern "C"
