// Internal declarations shared by the library's translation units (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/moe_budget.h"

struct moe_cache;

namespace moe {

// Sticky device error bits (OR-ed by kernels into the per-device flag word).
enum : int { kErrRange = 1, kErrNonfinite = 2, kErrNotResident = 4, kErrBudget = 8 };

// Bytes of one expert blob and the byte offset of W_d inside it.
size_t expert_blob_bytes(int H, int I, int dtype);
size_t down_offset(int H, int I, int dtype);

// Workspace carve-up of moe_expert_ffn_grouped.
struct FfnWorkspace {
    float *act;       // [(T*k + T) x I] SwiGLU activations, one row per (token, rank) pair + shared
    int *groups;      // grouping table (T > 1 only)
};
size_t ffn_workspace_bytes(int T, int k, int I);
FfnWorkspace ffn_workspace(void *base, int T, int k, int I);

// Kernel launchers (all asynchronous on `s`).  Shapes are validated by the caller.
hipError_t launch_router_logits(const float *x, const void *w, int w_dtype, int T, int H, int E,
                                const float *bias, float *logits, bool norm, float *h_out, hipStream_t s);
// Host-visible mailbox for one token's ids (coherent pinned memory): the top-k
// kernel writes ids[0..k), then, after a system-scope fence, seq.
// With a host tier the wave also publishes the weights, and copies the token's normalised input h (H
// floats, from h_src in device memory) to h_pub (host memory), before the fence.
struct IdsMailbox {
    uint32_t seq;
    int32_t ids[MOE_MAX_TOPK];
    float w[MOE_MAX_TOPK];
};
hipError_t launch_topk_softmax(const float *logits, int T, int E, int k, int32_t *ids, float *weights,
                               int *err_flags, hipStream_t s, IdsMailbox *pub = nullptr, uint32_t seq = 0,
                               const float *h_src = nullptr, float *h_pub = nullptr, int H = 0);
// x[i] += y[i], i < n (y may be host memory: the host tier's output).
hipError_t launch_add(float *x, const float *y, int n, hipStream_t s);

// Which expert kernels launch_expert_ffn enqueues (grouping goes with gate/up).
enum : int { kFfnGateUp = 1, kFfnDown = 2, kFfnBoth = 3 };

// A single-token step's missing experts streamed in by its gate/up launch
// (device residency): the blocks of a rank whose slot is in the lookup's fill
// list read that expert's gate/up rows from the host store, use them and
// store them into the slot; one more row of blocks copies each missing blob's
// down part.  The host link then carries the misses while the resident
// experts' gate/up runs, and no separate fill launch sits on the step's path.
struct FfnFill {
    unsigned long long *clk = nullptr;  // device fill clock of the cache (DevResidency::clk), or nullptr
    const int32_t *n = nullptr;      // device: number of fills (nullptr: this launch fills nothing)
    const long long *src = nullptr;  // device [n]: byte offset of each blob in the host store
    const int32_t *slot = nullptr;   // device [n]: its slot
    const uint8_t *host = nullptr;   // device address of the host store
    uint8_t *pool = nullptr;         // the slot pool, written
    long long doff = 0;              // byte offset of the down part in a blob
    int blocks = 32;                 // blocks streaming one missing expert's gate/up rows
    int slices = 32;                 // pieces of one missing blob's down part (one block each)
};

// Slots of a single-token step known on the host (after a residency lookup):
// off[j] = byte offset from the pool of the expert of rank j, or -1 for a rank
// the host tier computes (the kernels skip it).  n = k when valid, 0 when the
// kernels must read ids and the slot table on the device -- or, with
// rank_slot, the slot of each rank as a device lookup wrote it (one read
// instead of two dependent ones; -1 for a rank the lookup did not place).
struct FfnPlan {
    int n = 0;
    long long off[16];
    FfnFill fill;  // one token, slots read on the device: the fills this launch performs
    const int32_t *rank_slot = nullptr;  // one token, n == 0: device [k] slots by rank
};

hipError_t launch_expert_ffn(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                             const float *weights, const int32_t *slot_of, const void *pool,
                             size_t expert_bytes, int dtype, const void *shared_w, float *y,
                             bool accumulate, const FfnWorkspace &ws, int *err_flags, hipStream_t s,
                             const FfnPlan *plan = nullptr, int parts = kFfnBoth);
hipError_t launch_combine(const float *y_partial, const float *weights, const float *y_shared, int T,
                          int k, int H, float *y, bool accumulate, hipStream_t s);
hipError_t launch_slot_update(int32_t *table, const int32_t *index, const int32_t *value, int n,
                              hipStream_t s);
// A batch of expert fills (host blob -> HBM slot, `bytes` each, a multiple of
// 16) and the slot-table changes that go with them, done by one kernel.
constexpr int kMaxFillBatch = 32;
struct FillBatch {
    int n = 0;            // fills
    int n_tab = 0;        // table entries
    long long bytes = 0;  // bytes per fill
    const uint8_t *src[kMaxFillBatch];  // pinned host memory, device-accessible
    uint8_t *dst[kMaxFillBatch];
    int32_t *table = nullptr;
    int32_t tab_idx[2 * kMaxFillBatch];
    int32_t tab_val[2 * kMaxFillBatch];
};
hipError_t launch_fill_slots(const FillBatch &b, hipStream_t s);

// Device-resident residency (MOE_CACHE_DEVICE): the whole decision state of the
// slot table lives in HBM and one kernel per lookup updates it, so a decode step
// needs no host round trip.  Decisions are those of the host runtime (LRU or
// rotary), event for event.
constexpr int kDevMaxSlots = 4096;
enum : int {
    kScalCtr, kScalHand, kScalNextFree, kScalHits, kScalMisses, kScalEvictions, kScalEvents, kScalPrefetches,
    kDevScalars
};
// Fill clock of a device-residency cache, in device wall-clock ticks: a launch that performs demand fills
// records when its filling blocks started (minimum) and ended (maximum) and when its other, computing blocks
// ended (maximum), each spread over kClkLanes words to keep the atomics apart; the cache's next lookup kernel
// folds the record into the stall and fill-time totals and clears it.  Stall = how long the fills outlasted
// both their own start and the launch's compute, i.e. the time they held up the step.
constexpr int kClkLanes = 8;
enum : int { kClkFillStart = 0, kClkFillEnd = kClkLanes, kClkComputeEnd = 2 * kClkLanes, kClkStall = 3 * kClkLanes,
             kClkFill, kClkFolds, kClkWords };
struct DevResidency {
    unsigned long long *clk = nullptr;   // [kClkWords] fill clock (above)
    int32_t *key_of_slot = nullptr;      // [C] layer*E + expert, -1 = free
    uint64_t *stamp = nullptr;           // [C] LRU: recency stamp
    uint16_t *charge = nullptr;          // [C] rotary: charge
    int32_t *slot_of_key = nullptr;      // [L*E] the device slot table
    unsigned long long *scal = nullptr;  // [kDevScalars]
    moe_cache_event *events = nullptr;   // [cap_events] decision log
    long long cap_events = 0;
    long long *fill_src = nullptr;       // [E] byte offset in the host store of each fill's blob
    int32_t *fill_slot = nullptr;        // [E] its slot
    int32_t *n_fill = nullptr;           // [1] fills of the last lookup
};
struct DevLookup {
    int C, L, E, layer, step, rotary, charge_max;
    long long layer_stride, expert_stride;
    const int *step_dev = nullptr;  // when set, the step tag of the decisions is read here instead of `step`
    int prefetch = 0;               // 1: insert the non-resident ids only, as expert_cache_prefetch does
};
// Sets *p = v on the stream (a one-lane kernel: a graph replay reads the step tag from device memory).
hipError_t launch_set_int(int *p, int v, hipStream_t s);
// slots_out (device, optional): slots_out[i] = slot of ids[i] after the lookup.
hipError_t launch_dev_lookup(const DevResidency &r, const DevLookup &p, const int32_t *ids, int n, int32_t *slots_out,
                             int *err, hipStream_t s);
// One token: top-k of its logits fused with the device lookup of the selected experts (one block).
hipError_t launch_topk_lookup(const float *logits, int E, int k, int32_t *ids, float *weights, int *err_flags,
                              const DevResidency &r, const DevLookup &p, int32_t *slots_out, hipStream_t s);
// Streams the last lookup's fills (at most max_fills) from the host store into their slots.  Demand fills
// (`demand`) record their span in the fill clock; a prefetch's fills, off the step's path, do not.
hipError_t launch_dev_fill(const DevResidency &r, const uint8_t *host_dev, uint8_t *pool, long long expert_bytes,
                           int max_fills, hipStream_t s, bool demand = true);
hipError_t launch_hbm_read(const void *buf, size_t bytes, float *sink, hipStream_t s);

// Prefill (any T): pairs grouped by expert, grouped bf16 MFMA GEMMs, rank-order combine.
struct PrefillWorkspace {
    int *hdr;           // [0] = tiles
    int *g_slot;        // [E + 1] slot of each group (-2 = shared expert)
    int *g_off;         // [E + 2] start of each group in `sorted`
    int *tile_g;        // [max tiles] group of each 64-row tile
    int *tile_r0;       // [max tiles] first row of each tile within its group
    int *sorted;        // [T*k + T] pair ids grouped by expert
    uint16_t *xb;       // [T x H] bf16 copy of x (int4: each 8-group in the order 0,4,1,5,2,6,3,7)
    uint16_t *act;      // [(T*k + T) x I] bf16 SwiGLU activations, rows in `sorted` order (same 8-group order)
    float *y_part;      // [T*k x H] expert outputs per routed pair
    float *y_shared;    // [T x H] shared expert outputs
    float *sx;          // int4: [T x H/128] sums of xb over each quantisation group
    float *sa;          // int4: [(T*k + T) x I/128] sums of act over each quantisation group
};
bool prefill_dtype_supported(int dtype);
size_t prefill_workspace_bytes(int T, int k, int E, int H, int I);
PrefillWorkspace prefill_workspace(void *base, int T, int k, int E, int H, int I);
hipError_t launch_prefill_ffn(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                              const float *weights, const int32_t *slot_of, const void *pool, size_t expert_bytes,
                              int dtype, const void *shared_w, float *y, bool accumulate, const PrefillWorkspace &ws,
                              int *err_flags, hipStream_t s);

// Decoder self-attention of one decode token (attention.hip).
bool attention_shape_supported(int H, int n_heads, int n_kv, int head_dim, int max_pos);
size_t attention_workspace_bytes(int n_heads, int n_kv, int head_dim, int max_pos);
hipError_t launch_attention_decode(float *x, int H, int n_heads, int n_kv, int head_dim, const void *w_qkv,
                                   const void *w_o, uint16_t *k_cache, uint16_t *v_cache, int max_pos, int p,
                                   float theta, void *workspace, hipStream_t s);

bool ffn_shape_supported(int H, int I, int dtype);
bool router_shape_supported(int H, int dtype);

// Error reporting across the C ABI: records a thread-local message, returns `code`.
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int fail_hip(hipError_t e, const char *what);
void clear_error();

// Slot stride of a cache's pool; whether it was preloaded (slot = layer * E + expert, never evicted).
size_t cache_expert_bytes(const struct ::moe_cache *c);
bool cache_preloaded(const struct ::moe_cache *c);
bool cache_resident(const struct ::moe_cache *c, int layer, int expert);  // host mirror
bool cache_device(const struct ::moe_cache *c);  // lookups run on the device (MOE_CACHE_DEVICE)
int cache_capacity(const struct ::moe_cache *c);  // slots
bool cache_rotary(const struct ::moe_cache *c);   // MOE_POLICY_ROTARY
bool cache_host_tier(const struct ::moe_cache *c);  // demand lookups may leave experts to the host tier
const uint8_t *cache_host_blob(const struct ::moe_cache *c, int layer, int expert);  // host address in the store
// MOE_CACHE_DEVICE: enqueue on `s` the prefetch of ids_dev[0..n) at `layer` (non-resident ones inserted, logged
// as prefetches; resident ones untouched), its fills on the cache's copy stream; the next device lookup waits
// for those fills.  Returns an MOE_ERR_* code.
int cache_prefetch_device(struct ::moe_cache *c, int step, int layer, const int32_t *ids_dev, int n, hipStream_t s);
// MOE_CACHE_DEVICE, one token: enqueue top-k of `logits` fused with the lookup of the chosen experts, then
// the fills of its misses, unless fill_in_ffn (the step's gate/up launch then performs them, see FfnFill).
// Returns an MOE_ERR_* code.
int cache_topk_lookup(struct ::moe_cache *c, int step, int layer, const float *logits, int k, int32_t *ids,
                      float *weights, int32_t *slots_out, int *err_flags, hipStream_t s,
                      const int *step_dev = nullptr, bool fill_in_ffn = false);
// The fill list of the cache's last device lookup, for a gate/up launch that performs its fills
// (cache_topk_lookup with fill_in_ffn; that launch must follow the lookup on its stream).
FfnFill cache_ffn_fill(struct ::moe_cache *c, long long down_off);

// Sticky error-flag word of the current device (set up on first use).
int *device_error_flags();
// The same, or nullptr when the current device has not been set up yet (allocates nothing).
int *device_error_flags_ready();

// Allocation-free FFN workspace (kernels.hip): noalloc_scratch_setup() looks up the current device's copy of
// the fixed array once (an MOE_* code); noalloc_scratch() returns its device address, or nullptr before set-up.
int noalloc_scratch_setup();
void *noalloc_scratch();

}  // namespace moe
