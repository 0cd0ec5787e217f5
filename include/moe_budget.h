/*
 * moe_budget.h -- C ABI of the MI355X (gfx950) library for one Mixture-of-Experts
 * decode step under a fixed HBM budget for expert weights.
 *
 * The step (paper sec. 4, Fig. 1): the routing result (hidden state h and the
 * routing vector r) picks a subset of experts (sec. 3); a lookup table maps
 * each sub-module (expert) id to a slot of a fixed-size slot group on the
 * accelerator; sub-modules missing from the slots are brought in from the
 * host tier ("selective load") after making room ("evict"); execution stays
 * within a memory budget (sec. 5, memory-constrained execution).  Residency
 * follows least-recently-used replacement, the conventional policy sec. 4
 * contrasts with its own rotation scheme (which the paper does not define).
 *
 * Conventions for every call:
 *  - Return value: MOE_OK (0) or a negative MOE_ERR_* code; moe_last_error()
 *    returns a thread-local message for the last failure of the calling
 *    thread.  Nothing aborts or throws across this boundary.
 *  - Pointers named "device" are HIP device memory of the current device, owned
 *    by the caller; "host" pointers are host memory owned by the caller.  The
 *    library owns only what it allocates itself (cache slot pools, its copy
 *    stream and events, per-device error flags, stack workspaces).
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Device
 *    work is enqueued asynchronously on it unless a call says otherwise.
 *  - Errors found on the device (expert id out of range, non-finite logits,
 *    expert not resident) are raised in per-device sticky flags; read and
 *    clear them with moe_sync_check().
 *
 * Expert blob layout (one contiguous blob per expert; the residency unit):
 *    W_gu [2I x H] row-major, rows interleaved: row 2i = gate row i,
 *                  row 2i+1 = up row i;
 *    W_d  [H x I]  row-major.
 *  MOE_INT4G128 stores each matrix as packed nibbles [rows x K/2] (even
 *  element in the low nibble, two's complement q in [-8, 7]) followed by its
 *  bf16 scales [rows x K/128]; the weight is scale * q.  The blob is
 *  [gu nibbles | gu scales | d nibbles | d scales].
 *  Bytes per expert: 3*H*I*4 (f32), 3*H*I*2 (bf16), 3*H*I/2 + 3*H*I/64 (int4).
 */
#ifndef MOE_BUDGET_H
#define MOE_BUDGET_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Exported entry points (the library is built with hidden default visibility). */
#define MOE_API __attribute__((visibility("default")))

/* ---- status codes ---- */
#define MOE_OK 0
#define MOE_ERR_INVALID_ARG (-1)  /* bad size, null pointer, unsupported shape */
#define MOE_ERR_RANGE (-2)        /* expert id outside [0, E) */
#define MOE_ERR_NONFINITE (-3)    /* NaN or +-inf router logit */
#define MOE_ERR_BUDGET (-4)       /* budget below one expert, or a step needs more experts than fit */
#define MOE_ERR_NOT_PINNED (-5)   /* host store is not page-locked (hipHostMalloc) memory */
#define MOE_ERR_HIP (-6)          /* a HIP runtime call failed */
#define MOE_ERR_COPY (-7)         /* a host-to-device fill failed; the slot stays unmapped */
#define MOE_ERR_NOT_RESIDENT (-8) /* the expert FFN found an expert with no slot */

/* ---- weight storage types ---- */
#define MOE_F32 0
#define MOE_BF16 1
#define MOE_INT4G128 2

/* ---- moe_route_topk flags ---- */
#define MOE_ROUTE_RMSNORM 1 /* route on the RMS-normalised input (pre-norm of the MoE block) */

/* ---- moe_expert_ffn_grouped flags ---- */
#define MOE_ACCUMULATE 1 /* y_out += MoE output (fused residual add) instead of y_out = output */

/* ---- residency ---- */
#define MOE_POLICY_LRU 0
#define MOE_POLICY_ROTARY 1 /* rotary slot group: a ring of slots swept by a hand (sec. 4, Fig. 2) */
#define MOE_CACHE_PRELOAD 1  /* start with every expert resident at slot layer*E + expert */
#define MOE_CACHE_HOST_SIM 2 /* no device: slots live in host memory and fills are memcpy */
#define MOE_CACHE_DEVICE 4   /* decisions on the device: lookups are kernels (expert_cache_lookup_device) */
#define MOE_CACHE_FILL_CLOCK 8 /* MOE_CACHE_DEVICE: time the demand fills on the device (stats stall_ns, fill_ns);
                                  the stamps add a few microseconds to each filling launch and lookup */

#define MOE_EVENT_HIT 0
#define MOE_EVENT_MISS 1
#define MOE_EVENT_PREFETCH 2
#define MOE_EVENT_HOST 3 /* served by the host tier: computed on host cores, not filled (slot -1) */

/* expert_cache_lookup's slots_out for an id the host tier serves */
#define MOE_SLOT_HOST (-2)

/* Limits of the decode kernels. */
#define MOE_MAX_EXPERTS 256   /* router top-k holds at most 4 logits per lane of a 64-wide wave */
#define MOE_MAX_TOPK 16
#define MOE_MAX_DECODE_TOKENS 16

/* ======================================================================= */
/* Library / device                                                        */
/* ======================================================================= */

/* Make `device` current for the calling thread and set up its error flags.
 * Other calls set up the current device on first use; calling this first
 * keeps that set-up out of timed regions. */
MOE_API int moe_init(int device);

/* Message of the calling thread's last failed call ("" if none). Owned by the
 * library; valid until the thread's next failing call. */
MOE_API const char *moe_last_error(void);

/* Synchronise `stream`, then read and clear the current device's sticky error
 * flags.  Returns MOE_ERR_RANGE, MOE_ERR_NONFINITE or MOE_ERR_NOT_RESIDENT
 * (first set, in that order) or MOE_OK. */
MOE_API int moe_sync_check(void *stream);

/* ======================================================================= */
/* Routing (paper sec. 3: tokens pass through a subset of experts; Fig. 1:   */
/* the routing result (h, r) drives the slot lookup)                         */
/* ======================================================================= */

/* Router logits and softmax-renormalised top-k for T tokens.
 *   x          device fp32 [T x H], or NULL to rank `logit_bias` alone
 *   w_router   device [E x H] row-major, w_dtype MOE_F32 or MOE_BF16
 *   logit_bias device fp32 [T x E] added to the router output, or NULL
 *   logits     device fp32 [T x E] out: z = W_r h (+ bias), fp32 accumulation,
 *              where h = x, or with MOE_ROUTE_RMSNORM h = x / sqrt(mean(x^2) + 1e-6)
 *   ids        device int32 [T x k] out: the k largest z of each token ranked by
 *              (z descending, expert id ascending)
 *   weights    device fp32 [T x k] out: exp(z_j - z_0) / sum_j' exp(z_j' - z_0)
 *   x_norm     device fp32 [T x H] out (MOE_ROUTE_RMSNORM only, may be NULL):
 *              the normalised h, the input of the block's experts
 * Limits: 1 <= k <= min(E, MOE_MAX_TOPK), E <= MOE_MAX_EXPERTS, H % 128 == 0.
 * A token with a non-finite logit gets ids -1 and weights 0 and raises
 * MOE_ERR_NONFINITE in the device flags.  T == 0 is a no-op. */
MOE_API int moe_route_topk(const float *x, const void *w_router, int w_dtype, int T, int H, int E, int k,
                           const float *logit_bias, float *logits, int32_t *ids, float *weights, int flags,
                           float *x_norm, void *stream);

/* ======================================================================= */
/* Expert FFN with weighted combine (north-star "fused SwiGLU expert FFN")   */
/* ======================================================================= */

/* Device workspace bytes moe_expert_ffn_grouped needs for T tokens. */
MOE_API size_t moe_ffn_workspace_bytes(int T, int k, int I);

/* y[t] = sum_j weights[t,j] * FFN_{ids[t,j]}(x[t]) + FFN_shared(x[t]), with
 * FFN(x) = W_d (silu(W_g x) * (W_u x)), fp32 accumulation, for T <= 16 tokens.
 *   x          device fp32 [T x H]
 *   ids        device int32 [T x k] (as written by moe_route_topk)
 *   weights    device fp32 [T x k]
 *   slot_of    device int32 [E]: slot of each expert of this layer (-1 = absent),
 *              or NULL for slot = expert id
 *   pool       device base of the slots; slot s starts at pool + s * expert_bytes
 *              (expert_bytes must be a multiple of 256)
 *   shared_w   device blob of the layer's shared expert (weight 1), or NULL
 *   y_out      device fp32 [T x H]; may alias x when flags has MOE_ACCUMULATE
 *   workspace  device, >= moe_ffn_workspace_bytes(T, k, I) bytes, 256-aligned
 * Each selected expert's weights are read once per call however many of the T
 * tokens chose it.  Ids out of range or without a slot raise MOE_ERR_RANGE /
 * MOE_ERR_NOT_RESIDENT in the device flags and contribute nothing. */
MOE_API int moe_expert_ffn_grouped(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                           const float *weights, const int32_t *slot_of, const void *pool,
                           size_t expert_bytes, int w_dtype, const void *shared_w, float *y_out,
                           void *workspace, size_t workspace_bytes, int flags, void *stream);

/* moe_expert_ffn_grouped without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the workspace is a fixed array of
 * MOE_NOALLOC_SCRATCH_BYTES in the library, one per device, held until the
 * process ends.  This call allocates nothing (no hipMalloc, no hipFree, no
 * allocating library routine); moe_init(device) must have run on the device
 * first (MOE_ERR_INVALID_ARG otherwise), since it looks up the array's address.
 * Needs moe_ffn_workspace_bytes(T, k, I) <= MOE_NOALLOC_SCRATCH_BYTES
 * (MOE_ERR_INVALID_ARG otherwise, with nothing enqueued); other arguments,
 * results and errors as for moe_expert_ffn_grouped.  Every call on a device
 * shares that device's array: calls whose work overlaps on one device (other
 * streams, other threads) race and must be serialised by the caller.  No part
 * of the array needs to start at zero (each call writes what it reads first). */
#define MOE_NOALLOC_SCRATCH_BYTES (4 << 20)
MOE_API int moe_expert_ffn_grouped_noalloc(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                                           const float *weights, const int32_t *slot_of, const void *pool,
                                           size_t expert_bytes, int w_dtype, const void *shared_w, float *y_out,
                                           int flags, void *stream);

/* Device workspace bytes moe_prefill_grouped needs. */
MOE_API size_t moe_prefill_workspace_bytes(int T, int k, int E, int H, int I);

/* Prompt evaluation (prefill; its rate is reported beside decode in the
 * table of sec. 8.1): the routed expert FFN of the sec. 4 step, over a whole
 * prompt chunk at once.
 * The expert FFN of moe_expert_ffn_grouped for a prefill chunk of any T, as
 * grouped GEMMs on the matrix cores: the T*k (token, rank) pairs are grouped by
 * expert on the device (the shared expert takes all T tokens), each group's
 * rows run through x W_gu^T -> SwiGLU -> W_d^T in 64-row tiles with bf16 MFMA
 * and fp32 accumulation, and each token's outputs are summed in rank order
 * with its weights (the moe_combine kernel).  x and the SwiGLU activations are
 * rounded to bf16 (round to nearest even) for the matrix cores, and int4
 * weights are dequantised to bf16 (scale * q, rounded once).
 * w_dtype MOE_BF16 or MOE_INT4G128 (MOE_ERR_INVALID_ARG otherwise); other
 * arguments as for moe_expert_ffn_grouped; H, I multiples of 128,
 * E <= MOE_MAX_EXPERTS; workspace >= moe_prefill_workspace_bytes(T, k, E, H, I).
 * Pairs with an id out of range or without a slot raise the device flag and
 * contribute nothing. */
MOE_API int moe_prefill_grouped(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                                const float *weights, const int32_t *slot_of, const void *pool,
                                size_t expert_bytes, int w_dtype, const void *shared_w, float *y_out,
                                void *workspace, size_t workspace_bytes, int flags, void *stream);

/* y_out[t,h] (+)= sum_j weights[t,j] * y_partial[t,j,h] (rank order) + y_shared[t,h].
 *   y_partial device fp32 [T x k x H]; y_shared device fp32 [T x H] or NULL;
 *   flags MOE_ACCUMULATE adds into y_out. */
MOE_API int moe_combine(const float *y_partial, const float *weights, const float *y_shared, int T, int k,
                int H, float *y_out, int flags, void *stream);

/* ======================================================================= */
/* Decoder self-attention of one decode token (the block before each MoE)   */
/* ======================================================================= */

/* Device workspace bytes moe_attention_decode needs. */
MOE_API size_t moe_attention_workspace_bytes(int n_heads, int n_kv, int head_dim, int max_pos);

/* x <- x + W_o Attn(rmsnorm(x)) for one token at position p, in place on x
 * (device fp32 [H]).  The paper runs its model with a 4096-token context and
 * attention on the accelerator (sec. 6) but describes no attention arithmetic;
 * this is a Qwen3-class reading: unit-gain RMS pre-norm (eps 1e-6);
 * [q; k; v] = W_qkv h with n_heads query heads and n_kv key/value heads of
 * head_dim each (query head j reads key/value head j / (n_heads / n_kv));
 * every query and key head RMS-normalised (unit gain, eps 1e-6), then rotated
 * by the rotary embedding of the rotate-half form (dims i and i + head_dim/2
 * turned by p * theta^(-2i/head_dim)); the key and value stored at position p
 * of the bf16 caches (round to nearest even); softmax(q . k / sqrt(head_dim))
 * over positions 0..p; the heads' outputs concatenated through W_o.
 *   w_qkv    device bf16 [(n_heads + 2 n_kv) head_dim x H]: query rows, key rows, value rows
 *   w_o      device bf16 [H x n_heads head_dim]
 *   k_cache  device bf16 [n_kv][head_dim / 8][max_pos][8] (8-dim pieces of each position's key, position-
 *            contiguous, so that 64 positions of a piece are one 1 KiB read)
 *   v_cache  device bf16 [n_kv][max_pos][head_dim]
 *            positions < p are read, position p is written
 *   workspace device, >= moe_attention_workspace_bytes(...), 16-byte aligned
 * Needs H a multiple of 128, n_heads * head_dim a multiple of 128, head_dim a
 * multiple of 8 up to 128, n_heads / n_kv one of 1, 2, 4, 8, 16, max_pos at most
 * 16384, 0 <= p < max_pos, theta > 1; MOE_ERR_INVALID_ARG otherwise.  Cache
 * content at positions above p is never used (it may be anything, NaN included). */
MOE_API int moe_attention_decode(float *x, int H, int n_heads, int n_kv, int head_dim, const void *w_qkv,
                                 const void *w_o, void *k_cache, void *v_cache, int max_pos, int p, float theta,
                                 void *workspace, size_t workspace_bytes, void *stream);


/* ======================================================================= */
/* Expert residency: slot table in HBM, misses filled from pinned host      */
/* memory (paper Fig. 1: host tier, slot group, lookup table sub-module id  */
/* -> slot, selective load, evict; sec. 4: LRU as the conventional policy,  */
/* and the rotary slot group whose residency advances around a ring).       */
/*                                                                         */
/* Replacement at step granularity: a lookup takes the step's ascending     */
/* unique experts; a miss takes the lowest free slot, else a victim whose   */
/* expert the same step does not need.                                      */
/*   MOE_POLICY_LRU: the least recently used slot (one stamp per lookup).   */
/*   MOE_POLICY_ROTARY: the slots form a ring with a hand; a demand hit     */
/*     raises its slot's charge by one (at most charge_max), a new entry    */
/*     starts uncharged; a miss rotates the hand forward, passing over the  */
/*     step's own slots, taking one charge from each charged slot it passes */
/*     and stopping at the first uncharged one, which is the victim; the    */
/*     hand then moves past it.  The paper does not disclose how its        */
/*     rotation is steered: the charges are this library's reading.         */
/* ======================================================================= */

typedef struct moe_cache moe_cache;

typedef struct {
    int n_layers;              /* L */
    int n_experts;             /* E routed experts per layer */
    size_t expert_bytes;       /* bytes of one expert blob; multiple of 256 */
    size_t budget_bytes;       /* HBM budget for expert weights */
    size_t reserved_bytes;     /* part of the budget held by always-resident weights (shared experts) */
    const void *host_base;     /* pinned host store, one hipHostMalloc allocation; expert (l, e) at
                                  host_base + l*host_layer_stride + e*host_expert_stride (blob size a multiple of 16) */
    size_t host_layer_stride;  /* 0 lets layers alias one host copy (keys stay distinct) */
    size_t host_expert_stride;
    int policy;                /* MOE_POLICY_LRU or MOE_POLICY_ROTARY */
    int flags;                 /* MOE_CACHE_PRELOAD | MOE_CACHE_HOST_SIM | MOE_CACHE_DEVICE | MOE_CACHE_FILL_CLOCK */
    int charge_max;            /* MOE_POLICY_ROTARY: most charge a slot holds, 0..65535 (0 = cyclic FIFO) */
    /* Host tier (the paper's run recipe keeps experts of some layers in host memory and computes them on
     * host cores, sec. 6 and Fig. 3): demand lookups may leave experts in the host store, to be computed there
     * (moe_host_expert_ffn) instead of filled over the link.  Both 0 = no host tier.  Not with
     * MOE_CACHE_DEVICE or MOE_CACHE_PRELOAD.  The rule, per demand lookup of layer l (prefetches ignore it):
     *   l < host_layers: every expert of the step is served by the host (no slot is touched);
     *   otherwise, of the step's non-resident experts, those the host served at layer l's previous demand
     *   lookup stay with the host, then further ones in ascending id order while the lookup's host count is
     *   below host_quota (the sticky ones count too, so a lookup serves at most max(host_quota, sticky) on
     *   the host, and by induction at most host_quota); the rest miss and are filled as usual.
     * Host-served experts log MOE_EVENT_HOST (slot -1, victim -1), take no recency stamp and no slot. */
    int host_layers;           /* 0..L */
    int host_quota;            /* 0..E */
} moe_cache_desc;

typedef struct {
    uint64_t lookups;     /* expert lookups (unique ids per call) */
    uint64_t hits;
    uint64_t misses;
    uint64_t prefetches;  /* speculative inserts */
    uint64_t evictions;
    uint64_t h2d_bytes;   /* bytes filled from the host store */
    int32_t capacity;     /* slots: floor((budget - reserved) / expert_bytes) */
    int32_t occupancy;    /* slots holding an expert */
    /* MOE_CACHE_DEVICE with MOE_CACHE_FILL_CLOCK (0 otherwise), device wall-clock time of the demand fills
     * (sec. 4's selective load on the step's path; a prefetch's fills are not counted):
     *   fill_ns:  per filling launch, from its first filling block's start to its last one's end, summed;
     *   stall_ns: per filling launch, how long its fills ran past both their start and the end of the
     *             launch's computing blocks (the resident experts' work), summed.  The fills' own traffic
     *             slows the computing blocks beside them, so this is a lower bound on what the misses add
     *             to the step. */
    uint64_t stall_ns;
    uint64_t fill_ns;
    uint64_t host_computed;  /* lookups served by the host tier (counted in lookups too) */
} moe_cache_stats;

/* One residency decision.  victim_key = layer * E + expert of the evicted
 * entry, or -1. */
typedef struct {
    int32_t step, layer, expert, kind, slot, victim_key;
} moe_cache_event;

/* Create a cache: allocates capacity * expert_bytes of HBM for the slots, a
 * copy stream and its events, and the device slot table int32 [L x E].
 * Fills (selective loads, sec. 4) are done by kernels that read the blobs from
 * the host store over PCIe, all of a lookup's fills and slot-table changes in
 * one launch (per 32 fills): a demand lookup enqueues them on its compute
 * stream, a prefetch on the cache's copy stream.
 * MOE_ERR_BUDGET if capacity < 1 (or < L*E with MOE_CACHE_PRELOAD);
 * MOE_ERR_NOT_PINNED if host_base is not hipHostMalloc memory.  PRELOAD fills
 * every slot synchronously before returning.  With MOE_CACHE_HOST_SIM no HIP
 * call is made: slots are host memory and `dev_slot_of` is a host array. */
MOE_API int expert_cache_create(const moe_cache_desc *desc, moe_cache **out);

/* MOE_CACHE_DEVICE: the slot table's decision state (slot keys, LRU stamps or
 * rotary charges, counters, a log of up to 2^21 decisions and a fill list;
 * about 50 MB of HBM besides the slots) lives on the device, and a lookup is a
 * kernel that takes the same decisions as expert_cache_lookup, followed by a
 * kernel that streams the misses from the host store: a decode step needs no
 * host round trip.  Needs capacity <= 4096 and n_experts <= 256; cannot be
 * combined with MOE_CACHE_HOST_SIM.  In this mode expert_cache_lookup and
 * expert_cache_prefetch return MOE_ERR_INVALID_ARG (their _device forms take
 * their place), expert_cache_release does nothing, and expert_cache_stats /
 * expert_cache_trace synchronise the device. */

/* Device lookup (MOE_CACHE_DEVICE only): enqueues on `stream` the lookup of the
 * experts ids_dev[0..n) (device int32, e.g. as written by moe_route_topk) of
 * `layer`, tagged `step`, and the fills of its misses; kernels that run later on
 * `stream` see the updated slot table.  slots_out_dev (device int32 [n], or
 * NULL) receives the slot of each id after the lookup.  Ids outside [0, E) raise MOE_ERR_RANGE
 * and a step with more distinct experts than slots MOE_ERR_BUDGET in the device
 * flags (moe_sync_check); such a lookup changes nothing in the cache and writes
 * -1 to every slots_out_dev entry.  Lookups must be
 * ordered: issue them on one stream. */
MOE_API int expert_cache_lookup_device(moe_cache *c, int step, int layer, const int32_t *ids_dev, int n,
                                       int32_t *slots_out_dev, void *stream);

/* Device prefetch (MOE_CACHE_DEVICE only): the speculative insert of
 * expert_cache_prefetch with device ids (int32 [n], e.g. a routing result or
 * a fixed list): non-resident ids are placed like misses, counted as
 * prefetches and logged with MOE_EVENT_PREFETCH; resident ids are left
 * untouched.  The decisions are enqueued on `stream`; the fills run on the
 * cache's copy stream after everything queued on `stream` before this call,
 * so work queued next on `stream` overlaps them, and the next device lookup
 * or prefetch waits for them.  A victim may be any slot outside this call's
 * set: work queued on `stream` after this call must not read slots returned
 * by an earlier lookup, unless LRU cannot evict them (no lookup in between
 * and capacity >= that lookup's distinct experts + this call's: the earlier
 * set's stamps are newer than every victim's).  Errors as for
 * expert_cache_lookup_device (range and budget errors in the device flags,
 * changing nothing). */
MOE_API int expert_cache_prefetch_device(moe_cache *c, int step, int layer, const int32_t *ids_dev, int n,
                                         void *stream);

/* Wait for the cache's copies and free everything it owns. */
MOE_API int expert_cache_destroy(moe_cache *c);

/* Demand lookup of the experts one step needs at `layer` (host call).
 *   ids_host  host int32 [n]; the step's set is the ascending unique ids
 *   slots_out host int32 [n] or NULL: slot of each ids_host[i]
 *   hit_out   host uint8 [n] or NULL: 1 if ids_host[i] was resident
 * Each id in ascending order takes one recency stamp: a resident id is a hit;
 * a missing one takes the lowest free slot, else evicts the least recently
 * used slot whose expert is not in this step's set.  Fills are queued on the
 * cache's copy stream, each after the last recorded reader of its victim
 * slot; the changed slot-table entries are written on `compute_stream`, which
 * is then made to wait for the fills.  MOE_ERR_BUDGET (no state change) if
 * the set is larger than the capacity; MOE_ERR_RANGE for ids outside [0, E). */
MOE_API int expert_cache_lookup(moe_cache *c, int step, int layer, const int32_t *ids_host, int n,
                        int32_t *slots_out, uint8_t *hit_out, void *compute_stream);

/* Speculative insert: non-resident ids are placed like misses (counted as
 * prefetches, logged with MOE_EVENT_PREFETCH) and their fills queued; resident
 * ids are left untouched (no recency refresh).  Does not wait on anything;
 * the next lookup on a compute stream orders the fills before its use.
 * Errors as for expert_cache_lookup. */
MOE_API int expert_cache_prefetch(moe_cache *c, int step, int layer, const int32_t *ids_host, int n);

/* Record, on `compute_stream`, the point after which the slots returned by
 * the last lookup are no longer read (call after enqueueing the FFN).  A
 * lookup that finds unreleased slots releases them on the stream of the
 * previous lookup first. */
MOE_API int expert_cache_release(moe_cache *c, void *compute_stream);

/* Device slot table int32 [L x E] (-1 = absent; a host array under
 * HOST_SIM) and the slot pool base.  Owned by the cache. */
MOE_API int expert_cache_slot_table(moe_cache *c, const int32_t **dev_slot_of, const void **pool);

MOE_API int expert_cache_stats(moe_cache *c, moe_cache_stats *out);

/* Copy events [first, first + cap) of the decision log into buf; *n_out =
 * number copied. */
MOE_API int expert_cache_trace(moe_cache *c, size_t first, moe_cache_event *buf, size_t cap,
                       size_t *n_out);

/* ======================================================================= */
/* Decode stack driver: for each layer, pre-norm + route -> (lookup) -> FFN */
/* with fused residual x += MoE(rmsnorm(x)); attention is the identity       */
/* ======================================================================= */

/* ======================================================================= */
/* Host tier: expert FFN on host cores, from the host store (the paper's    */
/* run recipe computes the experts it keeps in host memory on the CPU,      */
/* sec. 6, Fig. 3)                                                          */
/* ======================================================================= */

typedef struct moe_host_tier moe_host_tier;

/* A pool of `threads` host threads (the calling thread is one of them; 0 = every core the process may run
 * on).  Idle threads spin briefly, then sleep. */
MOE_API int moe_host_tier_create(int threads, moe_host_tier **out);
MOE_API int moe_host_tier_destroy(moe_host_tier *t);

/* y_out[h] = sum_j weights[j] * (W_d^j silu(W_g^j x) * (W_u^j x))[h], j = 0..n-1 in that order, for one
 * token, on the pool's threads (synchronous; host memory only; fp32 accumulation):
 *   x        host fp32 [H]
 *   blobs    host array [n] of host expert blobs (layout above), e.g. in the pinned host store
 *   weights  host fp32 [n]
 *   y_out    host fp32 [H], overwritten
 * The gate/up rows are split over the threads, then (after all have finished) the output rows; each output
 * row is summed by one thread in rank order, so the result does not depend on the thread count.
 * w_dtype MOE_F32, MOE_BF16 or MOE_INT4G128; H, I multiples of 128; 0 <= n <= MOE_MAX_TOPK
 * (MOE_ERR_INVALID_ARG otherwise; n = 0 writes zeros). */
MOE_API int moe_host_expert_ffn(moe_host_tier *t, const float *x, int H, int I, int w_dtype, int n,
                                const void *const *blobs, const float *weights, float *y_out);

typedef struct moe_stack moe_stack;

/* A decoder self-attention block before each MoE block (moe_attention_decode),
 * in place of the identity. */
typedef struct {
    int n_heads, n_kv, head_dim, max_pos;
    float theta;                    /* rotary base */
    int start_pos;                  /* position of the first decode step (caches hold 0..start_pos-1) */
    const void *const *w_qkv;       /* host array [L] of device bf16 [(n_heads + 2 n_kv) head_dim x H] */
    const void *const *w_o;         /* host array [L] of device bf16 [H x n_heads head_dim] */
    void *const *k_cache;           /* host array [L] of device key caches, layout of moe_attention_decode */
    void *const *v_cache;           /* host array [L] of device value caches */
} moe_attention_desc;

typedef struct {
    int n_layers, H, I, E, k;
    int w_dtype;                    /* expert storage type */
    int router_dtype;               /* MOE_F32 or MOE_BF16 */
    const void *const *router_w;    /* host array [L] of device [E x H] router weights */
    const void *const *shared_w;    /* host array [L] of device shared-expert blobs, or NULL */
    moe_cache *cache;               /* residency of the routed experts */
    int max_tokens;                 /* largest T passed to moe_stack_decode_step (<= 16) */
    int max_prefill_tokens;         /* largest T passed to moe_stack_prefill (0: no prefill) */
    int prefetch;                   /* one-token decode under a budget: after each layer, prefetch up to this
                                       many experts of the next layer -- its most often demanded ones that
                                       are not resident (ties: lower id); 0 = off */
    int recall;                     /* one-token decode under a budget: reverse rotation (sec. 4, Fig. 2: a
                                       recurring context returns the slot group to a prior set).  The stack
                                       keeps up to this many snapshots of past tokens -- the token's layer-0
                                       expert set as its context signature (the routing result of the
                                       hidden state, Fig. 1) and its expert set at every layer.  When a
                                       token's layer-0 set shares >= recall_overlap experts with a snapshot
                                       (the most shared; ties: the most recent), the stack prefetches that
                                       snapshot's layer l+1 set after each layer l's release.  At the end of
                                       a token its snapshot replaces one with the same signature, else the
                                       oldest.  0 = off; at most 4096 */
    int recall_overlap;             /* 1..k shared layer-0 experts a recall needs (0 means k) */
    const moe_attention_desc *attention; /* NULL: attention is the identity.  Otherwise each layer is
                                       x <- x + Attn(rmsnorm(x)) then the MoE block; one-token steps only,
                                       the position advancing by one per step from start_pos; copied at
                                       creation (the arrays, not the device buffers they point to) */
    int host_threads;               /* a cache with a host tier (moe_cache_desc.host_layers / host_quota): the
                                       stack's moe_host_tier threads (0 = every core).  Each one-token step
                                       then publishes its ids, weights and normalised input to host memory,
                                       the host looks up, the GPU runs the fills and the GPU-resident experts
                                       while the host tier computes the host-served ones from the store, and a
                                       small kernel adds their sum to x.  One-token decode only (max_tokens 1,
                                       no prefill, no attention block) */
} moe_stack_desc;

MOE_API int moe_stack_create(const moe_stack_desc *desc, moe_stack **out);
MOE_API int moe_stack_destroy(moe_stack *s);

/* One decode step over every layer, in place on x (device fp32 [T x H]):
 * x <- x + MoE_l(rmsnorm(x)) for l = 0..L-1 (unit-gain RMS norm, eps 1e-6).  logit_bias is device fp32 [L x T x E]
 * added to each layer's router logits, or NULL.  Unless the cache was created
 * with PRELOAD or DEVICE, each layer copies its ids to the host (one
 * synchronisation per layer), runs the lookup, then enqueues the FFN and
 * releases the slots.  With a DEVICE cache nothing waits for the host: each
 * layer enqueues its routing, the fused top-k + lookup and the FFN; for one
 * token the FFN's gate/up launch also streams the layer's missing experts from
 * the host store into their slots (the resident experts' gate/up runs
 * meanwhile), for more tokens a fill launch precedes the FFN.
 * ids_out (device int32 [L x T x k]), weights_out (device fp32 [L x T x k]) and
 * logits_out (device fp32 [L x T x E]: each layer's router logits, bias
 * included, as the top-k saw them) receive each layer's routing when non-NULL. */
MOE_API int moe_stack_decode_step(moe_stack *s, int step, float *x, int T, const float *logit_bias,
                          int32_t *ids_out, float *weights_out, float *logits_out, void *stream);

/* moe_stack_decode_step for one token (T = 1), as a replayed HIP graph.  With a
 * MOE_CACHE_DEVICE cache nothing in a step waits for the host, so the first call
 * captures the step's launches (every layer's routing, fused top-k + lookup,
 * and expert FFN with its fills) and later calls replay them after setting the step tag
 * on the device; a call with other x / logit_bias / ids_out / weights_out /
 * logits_out pointers captures again (keep the buffers fixed and refill them).  Results
 * and residency decisions are those of moe_stack_decode_step.  Without a device
 * cache it is moe_stack_decode_step. */
MOE_API int moe_stack_decode_graph(moe_stack *s, int step, float *x, const float *logit_bias, int32_t *ids_out,
                                   float *weights_out, float *logits_out, void *stream);

/* Prompt evaluation (prefill; its rate is reported beside decode in the table
 * of sec. 8.1) over every layer, in place on x (device fp32 [T x H]):
 * x <- x + MoE_l(rmsnorm(x)) for l = 0..L-1, with each layer's routing on the
 * matrix cores when the router is bf16 and T >= 16, and its expert FFN by
 * moe_prefill_grouped (bf16 activations on the matrix cores; w_dtype MOE_BF16 or
 * MOE_INT4G128).  Under a budget each layer copies its T*k ids to the host and
 * runs one lookup for the chunk's distinct experts, which must fit in the cache
 * (MOE_ERR_BUDGET otherwise).  1 <= T <= max_prefill_tokens; ids_out / weights_out /
 * logits_out as for moe_stack_decode_step; `step` is the residency step of the chunk. */
MOE_API int moe_stack_prefill(moe_stack *s, int step, float *x, int T, int32_t *ids_out, float *weights_out,
                              float *logits_out, void *stream);

/* Mean device time (ms) of one launch of kernel `which` (0 = router logits and
 * top-k, 1 = expert gate/up + SwiGLU, 2 = expert down + combine, 3 = the whole
 * expert FFN as the decode step issues it, both launches; 4 = the attention
 * block, its five launches, at the last step's position -- this rewrites the
 * caches' entries of that position).  Each
 * layer's launch of the last decode step is re-issued with the same
 * arguments, in step order, captured into one HIP graph on a private stream
 * (ordered after `stream`); the graph is replayed n times between two HIP
 * events (multi-token steps under a budget replay only the last layer, whose
 * slots are still current).  A graph of fewer than 32 launches repeats the
 * sequence until it holds at least 32 (R repeats); in a stack without a budget
 * (every expert resident) repeat r of an expert launch (which 1-3) reads
 * experts (e + r) mod E in place of the step's experts e, so that the repeats
 * stream many experts instead of re-reading a few from the last-level cache;
 * which + 8 (9, 10, 11) keeps the step's own experts in every repeat.
 * Outputs go to scratch buffers: the residual stream and the residency state
 * are untouched.  Synchronous. */
MOE_API int moe_stack_kernel_time(moe_stack *s, int which, int n, void *stream, double *mean_ms);

/* Offline residency bound (host call; no device work).  For a demand trace in
 * which step i needs the distinct keys keys[offsets[i] .. offsets[i+1])
 * resident together (key = layer * E + expert, < n_keys; offsets[0] = 0), the
 * fewest fills any replacement policy with `capacity` slots needs, compulsory
 * fills included: Belady's farthest-next-use rule at step granularity.  It
 * bounds from below what the LRU residency (sec. 4's conventional policy) or
 * any other policy can do on the same trace.  MOE_ERR_BUDGET if a step has more
 * than `capacity` keys; MOE_ERR_RANGE for a key outside [0, n_keys);
 * MOE_ERR_INVALID_ARG for bad offsets or a key repeated within a step. */
MOE_API int moe_opt_fills(const int32_t *keys, const int32_t *offsets, int n_steps, int n_keys, int capacity,
                          uint64_t *fills_out);

/* Measurement aid, not part of the method: streams `bytes` of device memory
 * once, with the 16-byte nontemporal loads the expert kernels use for weight
 * rows (each wave issues four 1 KiB pieces before consuming any), so that a
 * caller timing it gets the HBM read rate those kernels can reach.  buf: device
 * memory, 16-byte aligned, bytes a multiple of 16 (< 2^31 * 16 KiB); sink:
 * device float [1], written only in the unlikely case that the data xor to a
 * fixed pattern.  Enqueued on `stream`. */
MOE_API int moe_hbm_read_probe(const void *buf, size_t bytes, float *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_BUDGET_H */
