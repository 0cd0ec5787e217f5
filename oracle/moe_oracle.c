/*
 * moe_oracle.c -- CPU oracle for one Mixture-of-Experts decode step under an
 * expert-memory budget.  TEST INFRASTRUCTURE ONLY: the tests, the smoke check
 * and the benchmark's CPU-baseline leg load it; the product path never does.
 * It shares no code, header or table with the HIP library.
 *
 * What it computes, and the passage each part follows:
 *   - routing (paper sec. 3: an MoE routes each token through a subset of its
 *     experts; Fig. 1: the routing result carries the hidden state h and the
 *     routing vector r): logits z = W_r h, the k largest logits ranked by
 *     (z descending, expert id ascending), weights = softmax over those k.
 *   - expert FFN: the SwiGLU feed-forward block (Shazeer 2020), as used by the
 *     Qwen3-class MoE of the paper's Table 2: silu(W_g x) * (W_u x), then W_d.
 *   - combine: y = sum over the k selected experts, in rank order, of weight
 *     times expert output, plus the shared expert with weight 1.
 *   - stacking: each MoE block reads the RMS-normalised residual stream
 *     (unit gain) and adds its output back: x <- x + MoE(rmsnorm(x)).
 *   - residency (paper sec. 4 and Fig. 1: a host tier holds every sub-module,
 *     the accelerator holds slots, a lookup table maps sub-module id to slot,
 *     selective load brings sub-modules in and evict makes room; sec. 4 names
 *     least-recently-used eviction as the conventional policy; sec. 5:
 *     memory-constrained execution): an LRU slot table of fixed capacity,
 *     and the rotary slot group of sec. 4 and Fig. 2 (the slots form a ring
 *     that is rotated forward, cyclic replacement instead of recency order;
 *     how the rotation is steered is not disclosed, so the steering here is
 *     our reading: a per-slot charge raised by hits, spent by the passing
 *     hand).
 *   - offline bound on residency: the fewest fills any replacement policy
 *     could need for a demand trace (Belady's farthest-next-use rule at step
 *     granularity), the yardstick against which LRU's fills are reported.
 *
 * Readings where the paper is silent (all of it; it withholds its method):
 *   no router bias or noise; softmax over the selected k only (equal to a full
 *   softmax renormalised over the k); ties broken by lower expert id, -0 equal
 *   to +0; non-finite logits are an error; a step's lookups take its ascending
 *   unique expert ids, one recency stamp each; a miss takes the lowest free
 *   slot, else evicts the least recently used slot whose expert is not needed
 *   by the same step; int4 weights are scale * q with q a two's-complement
 *   nibble (low nibble = even element) and one bf16 scale per 128 elements.
 *
 * Arithmetic is fp64 throughout (weights are exact in fp64); each dot product
 * is summed in index order, so the result does not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_F32 0
#define OR_BF16 1
#define OR_INT4G128 2

#define OR_OK 0
#define OR_ERR_ARG (-1)
#define OR_ERR_RANGE (-2)
#define OR_ERR_NONFINITE (-3)
#define OR_ERR_BUDGET (-4)

/* ------------------------------------------------------------ weights --- */

static double bf16_value(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* A row-major [rows x cols] weight matrix in one of the storage types. */
typedef struct {
    int dtype, rows, cols;
    const uint8_t *data;   /* f32 / bf16 elements, or packed nibbles */
    const uint8_t *scales; /* int4 only: bf16 [rows x cols/128] */
} matrix;

static double weight_at(const matrix *m, int r, int c)
{
    size_t idx = (size_t)r * m->cols + c;
    if (m->dtype == OR_F32) {
        float f;
        memcpy(&f, m->data + 4 * idx, 4);
        return f;
    }
    if (m->dtype == OR_BF16) {
        uint16_t b;
        memcpy(&b, m->data + 2 * idx, 2);
        return bf16_value(b);
    }
    /* int4, group 128: two elements per byte, low nibble first */
    uint8_t byte = m->data[idx / 2];
    int nib = (c % 2 == 0) ? (byte & 0xF) : (byte >> 4);
    int q = nib >= 8 ? nib - 16 : nib;
    uint16_t sb;
    memcpy(&sb, m->scales + 2 * ((size_t)r * (m->cols / 128) + c / 128), 2);
    return bf16_value(sb) * q;
}

/* Expert blob = [W_gu (2I x H, row 2i = gate i, row 2i+1 = up i) ; W_d (H x I)];
 * int4 matrices carry their scales right after their packed nibbles. */
static void expert_matrices(const uint8_t *blob, int dtype, int H, int I, matrix *gu, matrix *d)
{
    gu->dtype = d->dtype = dtype;
    gu->rows = 2 * I; gu->cols = H;
    d->rows = H; d->cols = I;
    if (dtype == OR_INT4G128) {
        size_t gu_q = (size_t)2 * I * H / 2, gu_s = (size_t)2 * I * (H / 128) * 2;
        size_t d_q = (size_t)H * I / 2;
        gu->data = blob;
        gu->scales = blob + gu_q;
        d->data = blob + gu_q + gu_s;
        d->scales = d->data + d_q;
    } else {
        size_t es = dtype == OR_F32 ? 4 : 2;
        gu->data = blob;
        gu->scales = NULL;
        d->data = blob + (size_t)2 * I * H * es;
        d->scales = NULL;
    }
}

/* One dequantised weight of an expert blob: matrix 0 = W_gu, 1 = W_d. */
double oracle_expert_weight(const void *blob, int dtype, int H, int I, int which, int r, int c)
{
    matrix gu, d;
    expert_matrices((const uint8_t *)blob, dtype, H, I, &gu, &d);
    return weight_at(which == 0 ? &gu : &d, r, c);
}

size_t oracle_expert_bytes(int H, int I, int dtype)
{
    if (dtype == OR_INT4G128)
        return (size_t)3 * H * I / 2 + (size_t)3 * H * I / 128 * 2;
    return (size_t)3 * H * I * (dtype == OR_F32 ? 4 : 2);
}

/* ---------------------------------------------------------- pre-norm --- */

/* h[t,:] = x[t,:] / sqrt(mean_i x[t,i]^2 + eps): the RMS normalisation a
 * pre-norm decoder (such as the Qwen3-class model of the paper's Table 2)
 * applies to the input of each MoE block, with unit gain. */
int oracle_rmsnorm(const float *x, int T, int H, double eps, double *h)
{
    if (T < 0 || H <= 0)
        return OR_ERR_ARG;
    for (int t = 0; t < T; t++) {
        double ss = 0.0;
        for (int i = 0; i < H; i++)
            ss += (double)x[(size_t)t * H + i] * (double)x[(size_t)t * H + i];
        double inv = 1.0 / sqrt(ss / H + eps);
        for (int i = 0; i < H; i++)
            h[(size_t)t * H + i] = (double)x[(size_t)t * H + i] * inv;
    }
    return OR_OK;
}

/* ------------------------------------------------------------ routing --- */

/* z[t*E + e] = sum_i W_r[e, i] x[t, i]   (router weights f32 or bf16). */
int oracle_router_logits(const float *x, const void *w_router, int w_dtype, int T, int H, int E,
                         double *z)
{
    if (T < 0 || H <= 0 || E <= 0 || (w_dtype != OR_F32 && w_dtype != OR_BF16))
        return OR_ERR_ARG;
    matrix W = {w_dtype, E, H, (const uint8_t *)w_router, NULL};
    for (int t = 0; t < T; t++)
        for (int e = 0; e < E; e++) {
            double acc = 0.0;
            for (int i = 0; i < H; i++)
                acc += weight_at(&W, e, i) * (double)x[(size_t)t * H + i];
            z[(size_t)t * E + e] = acc;
        }
    return OR_OK;
}

/* Top-k of each token's fp32 logits, ranked by (z desc, id asc), and the
 * softmax over the selected k.  k rounds of "best not yet taken". */
int oracle_topk_softmax(const float *z, int T, int E, int k, int32_t *ids, double *w)
{
    if (T < 0 || E <= 0 || k <= 0 || k > E)
        return OR_ERR_ARG;
    int status = OR_OK;
    char *taken = malloc((size_t)E);
    for (int t = 0; t < T; t++) {
        const float *zt = z + (size_t)t * E;
        int finite = 1;
        for (int e = 0; e < E; e++)
            if (!isfinite(zt[e]))
                finite = 0;
        if (!finite) {
            for (int j = 0; j < k; j++) {
                ids[(size_t)t * k + j] = -1;
                w[(size_t)t * k + j] = 0.0;
            }
            status = OR_ERR_NONFINITE;
            continue;
        }
        memset(taken, 0, (size_t)E);
        for (int j = 0; j < k; j++) {
            int best = -1;
            for (int e = 0; e < E; e++) {
                if (taken[e])
                    continue;
                /* strictly greater wins; equal values keep the lower id */
                if (best < 0 || zt[e] > zt[best])
                    best = e;
            }
            taken[best] = 1;
            ids[(size_t)t * k + j] = best;
        }
        double zmax = zt[ids[(size_t)t * k]];
        double sum = 0.0;
        for (int j = 0; j < k; j++) {
            double s = exp((double)zt[ids[(size_t)t * k + j]] - zmax);
            w[(size_t)t * k + j] = s;
            sum += s;
        }
        for (int j = 0; j < k; j++)
            w[(size_t)t * k + j] /= sum;
    }
    free(taken);
    return status;
}

/* ---------------------------------------------------------- expert FFN --- */

/* y[h] = sum_i W_d[h, i] * a[i],  a[i] = silu(W_g[i,:] x) * (W_u[i,:] x). */
int oracle_expert_forward(const float *x, int H, int I, const void *blob, int dtype, double *y)
{
    if (H <= 0 || I <= 0 || H % 128 || I % 128)
        return OR_ERR_ARG;
    matrix gu, d;
    expert_matrices((const uint8_t *)blob, dtype, H, I, &gu, &d);
    double *a = malloc(sizeof(double) * (size_t)I);
#pragma omp parallel for schedule(static)
    for (int i = 0; i < I; i++) {
        double g = 0.0, u = 0.0;
        for (int c = 0; c < H; c++) {
            g += weight_at(&gu, 2 * i, c) * (double)x[c];
            u += weight_at(&gu, 2 * i + 1, c) * (double)x[c];
        }
        a[i] = g / (1.0 + exp(-g)) * u;
    }
#pragma omp parallel for schedule(static)
    for (int h = 0; h < H; h++) {
        double acc = 0.0;
        for (int i = 0; i < I; i++)
            acc += weight_at(&d, h, i) * a[i];
        y[h] = acc;
    }
    free(a);
    return OR_OK;
}

/* y[t,:] = sum_j w[t,j] * expert_{ids[t,j]}(x[t,:])  (rank order)  + shared(x[t,:]).
 * Routed experts of the layer sit at experts_base + e * expert_stride. */
int oracle_moe_ffn(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                   const double *w, const void *experts_base, size_t expert_stride, int dtype,
                   const void *shared_blob, double *y)
{
    if (T < 0 || k <= 0 || E <= 0)
        return OR_ERR_ARG;
    for (size_t p = 0; p < (size_t)T * k; p++)
        if (ids[p] < 0 || ids[p] >= E)
            return OR_ERR_RANGE;
    double *ye = malloc(sizeof(double) * (size_t)H);
    int st = OR_OK;
    for (int t = 0; t < T && st == OR_OK; t++) {
        double *yt = y + (size_t)t * H;
        for (int h = 0; h < H; h++)
            yt[h] = 0.0;
        for (int j = 0; j < k && st == OR_OK; j++) {
            const uint8_t *blob = (const uint8_t *)experts_base + (size_t)ids[(size_t)t * k + j] * expert_stride;
            st = oracle_expert_forward(x + (size_t)t * H, H, I, blob, dtype, ye);
            for (int h = 0; h < H; h++)
                yt[h] += w[(size_t)t * k + j] * ye[h];
        }
        if (shared_blob && st == OR_OK) {
            st = oracle_expert_forward(x + (size_t)t * H, H, I, shared_blob, dtype, ye);
            for (int h = 0; h < H; h++)
                yt[h] += ye[h];
        }
    }
    free(ye);
    return st;
}

/* ------------------------------------------------------ LRU residency --- */

/* One residency decision.  kind: 0 hit, 1 miss, 2 prefetch insert.
 * victim_key = layer * E + expert of the evicted entry, or -1. */
typedef struct {
    int32_t t, layer, expert, kind, slot, victim_key;
} oracle_event;

#define OR_POLICY_LRU 0
#define OR_POLICY_ROTARY 1

typedef struct {
    int C, L, E;
    int policy;           /* OR_POLICY_LRU or OR_POLICY_ROTARY */
    int charge_max;       /* rotary: the most charge a slot can hold */
    int32_t *key_of_slot; /* layer * E + expert, or -1 for a free slot */
    uint64_t *stamp;      /* LRU: recency stamp of each slot */
    int *charge;          /* rotary: charge of each slot */
    int hand;             /* rotary: the ring position the next rotation starts from */
    uint64_t ctr;
    oracle_event *ev;
    size_t n_ev, cap_ev;
    uint64_t hits, misses, prefetches, evictions;
} oracle_lru;

static oracle_lru *residency_new(int capacity, int L, int E, int preload, int policy, int charge_max)
{
    if (capacity < 1 || L < 1 || E < 1 || (preload && capacity < L * E) || charge_max < 0)
        return NULL;
    oracle_lru *c = calloc(1, sizeof *c);
    c->C = capacity;
    c->L = L;
    c->E = E;
    c->policy = policy;
    c->charge_max = charge_max;
    c->charge = calloc((size_t)capacity, sizeof(int));
    c->key_of_slot = malloc(sizeof(int32_t) * (size_t)capacity);
    c->stamp = calloc((size_t)capacity, sizeof(uint64_t));
    for (int s = 0; s < capacity; s++)
        c->key_of_slot[s] = -1;
    if (preload)
        for (int key = 0; key < L * E; key++) {
            c->key_of_slot[key] = key;
            c->stamp[key] = ++c->ctr;
        }
    return c;
}

oracle_lru *oracle_lru_new(int capacity, int L, int E, int preload)
{
    return residency_new(capacity, L, E, preload, OR_POLICY_LRU, 0);
}

/* Rotary slot group (sec. 4, Figs. 1-2): the C slots form a ring with a hand.
 * Our steering of the rotation: a demand hit raises its slot's charge by one
 * (at most charge_max); a new entry starts uncharged.  A miss with no free slot
 * rotates the hand forward one slot at a time: a slot whose expert the current
 * step needs is passed over unchanged, a charged slot gives up one charge and
 * is passed over, and the first uncharged slot is the victim; the new entry
 * takes it and the hand moves on past it.  With charge_max = 0 this is cyclic
 * (first-in first-out) replacement. */
oracle_lru *oracle_rotary_new(int capacity, int L, int E, int charge_max, int preload)
{
    return residency_new(capacity, L, E, preload, OR_POLICY_ROTARY, charge_max);
}

void oracle_lru_free(oracle_lru *c)
{
    if (!c)
        return;
    free(c->key_of_slot);
    free(c->stamp);
    free(c->charge);
    free(c->ev);
    free(c);
}

static int slot_holding(const oracle_lru *c, int32_t key)
{
    for (int s = 0; s < c->C; s++)
        if (c->key_of_slot[s] == key)
            return s;
    return -1;
}

static void log_event(oracle_lru *c, int t, int layer, int e, int kind, int slot, int victim)
{
    if (c->n_ev == c->cap_ev) {
        c->cap_ev = c->cap_ev ? 2 * c->cap_ev : 1024;
        c->ev = realloc(c->ev, sizeof(oracle_event) * c->cap_ev);
    }
    oracle_event v = {t, layer, e, kind, slot, victim};
    c->ev[c->n_ev++] = v;
}

/* Ascending unique copy of ids; returns the count. */
static int ascending_unique(const int32_t *ids, int n, int32_t *out)
{
    int m = 0;
    for (int i = 0; i < n; i++) {
        int seen = 0;
        for (int j = 0; j < m; j++)
            if (out[j] == ids[i])
                seen = 1;
        if (!seen)
            out[m++] = ids[i];
    }
    for (int i = 1; i < m; i++) /* insertion sort */
        for (int j = i; j > 0 && out[j - 1] > out[j]; j--) {
            int32_t tmp = out[j];
            out[j] = out[j - 1];
            out[j - 1] = tmp;
        }
    return m;
}

static int in_step(const oracle_lru *c, int layer, const int32_t *R, int m, int32_t key)
{
    for (int j = 0; j < m; j++)
        if (key == layer * c->E + R[j])
            return 1;
    return 0;
}

/* Where a non-resident key goes: the lowest free slot; else, LRU: the slot with
 * the smallest stamp whose key is not in R (the step's set stays resident);
 * rotary: the slot at which the forward rotation stops (see oracle_rotary_new).
 * Some slot outside R exists whenever R holds a key that is not resident. */
static int place(oracle_lru *c, int layer, const int32_t *R, int m, int32_t *victim)
{
    for (int s = 0; s < c->C; s++)
        if (c->key_of_slot[s] < 0) {
            *victim = -1;
            return s;
        }
    if (c->policy == OR_POLICY_ROTARY) {
        for (;;) {
            int s = c->hand;
            c->hand = (c->hand + 1) % c->C;
            if (in_step(c, layer, R, m, c->key_of_slot[s]))
                continue;
            if (c->charge[s] > 0) {
                c->charge[s]--;
                continue;
            }
            *victim = c->key_of_slot[s];
            return s;
        }
    }
    int best = -1;
    for (int s = 0; s < c->C; s++) {
        if (in_step(c, layer, R, m, c->key_of_slot[s]))
            continue;
        if (best < 0 || c->stamp[s] < c->stamp[best])
            best = s;
    }
    *victim = c->key_of_slot[best];
    return best;
}

/* Demand lookup (prefetch = 0) or speculative insert (prefetch = 1) of the
 * experts `ids[0..n)` of one layer, tagged with step t. */
int oracle_lru_lookup(oracle_lru *c, int t, int layer, const int32_t *ids, int n, int prefetch)
{
    if (!c || layer < 0 || layer >= c->L || n < 0)
        return OR_ERR_ARG;
    for (int i = 0; i < n; i++)
        if (ids[i] < 0 || ids[i] >= c->E)
            return OR_ERR_RANGE;
    int32_t *R = malloc(sizeof(int32_t) * (size_t)(n ? n : 1));
    int m = ascending_unique(ids, n, R);
    if (m > c->C) {
        free(R);
        return OR_ERR_BUDGET;
    }
    for (int j = 0; j < m; j++) {
        int32_t key = layer * c->E + R[j];
        int s = slot_holding(c, key);
        if (s >= 0) {
            if (prefetch)
                continue; /* resident: a prefetch leaves it untouched */
            c->stamp[s] = ++c->ctr;
            if (c->charge[s] < c->charge_max)
                c->charge[s]++;
            c->hits++;
            log_event(c, t, layer, R[j], 0, s, -1);
            continue;
        }
        int32_t victim;
        s = place(c, layer, R, m, &victim);
        if (victim >= 0)
            c->evictions++;
        c->key_of_slot[s] = key;
        c->stamp[s] = ++c->ctr;
        c->charge[s] = 0;
        if (prefetch)
            c->prefetches++;
        else
            c->misses++;
        log_event(c, t, layer, R[j], prefetch ? 2 : 1, s, victim);
    }
    free(R);
    return OR_OK;
}

size_t oracle_lru_n_events(const oracle_lru *c) { return c->n_ev; }

/* Copies events [first, first + n) into out; returns how many were copied. */
size_t oracle_lru_events(const oracle_lru *c, size_t first, oracle_event *out, size_t n)
{
    if (first >= c->n_ev)
        return 0;
    if (n > c->n_ev - first)
        n = c->n_ev - first;
    memcpy(out, c->ev + first, n * sizeof(oracle_event));
    return n;
}

void oracle_lru_stats(const oracle_lru *c, uint64_t out[4])
{
    out[0] = c->hits;
    out[1] = c->misses;
    out[2] = c->prefetches;
    out[3] = c->evictions;
}

/* Slot of (layer, expert), or -1 when it is not resident. */
int oracle_lru_slot_of(const oracle_lru *c, int layer, int expert)
{
    return slot_holding(c, layer * c->E + expert);
}

int oracle_lru_occupancy(const oracle_lru *c)
{
    int n = 0;
    for (int s = 0; s < c->C; s++)
        n += c->key_of_slot[s] >= 0;
    return n;
}

/* ------------------------------------------------------------------------
 * Offline bound: the fewest fills any replacement policy needs for a demand
 * trace (Belady's farthest-next-use rule, applied at step granularity).
 *
 * Step i needs the distinct keys keys[offsets[i] .. offsets[i+1]) resident
 * together.  A missing key is filled; when all C slots are taken, the victim
 * is the resident key outside step i whose next step of use is the farthest
 * (a key never used again counts as infinitely far; ties: the smaller key).
 * Returns the number of fills (compulsory ones included), or -1 if a step
 * needs more than C keys or an argument is invalid.
 */
long long oracle_opt_misses(const int32_t *keys, const int32_t *offsets, int n_steps, int n_keys, int C)
{
    if (n_steps < 0 || n_keys < 1 || C < 1 || (n_steps > 0 && (!keys || !offsets)))
        return -1;
    const int32_t never = INT32_MAX;
    size_t n = n_steps > 0 ? (size_t)offsets[n_steps] : 0;
    int32_t *nxt = malloc((n + 1) * sizeof *nxt);      /* next step of use of each occurrence's key */
    int32_t *last = malloc((size_t)n_keys * sizeof *last);
    int32_t *res_key = malloc((size_t)C * sizeof *res_key);
    int32_t *res_next = malloc((size_t)C * sizeof *res_next);
    int32_t *where = malloc((size_t)n_keys * sizeof *where);   /* index in res_*, or -1 */
    uint8_t *in_step = calloc((size_t)n_keys, 1);
    long long misses = -1;
    if (!nxt || !last || !res_key || !res_next || !where || !in_step)
        goto out;
    for (int k = 0; k < n_keys; k++) {
        last[k] = never;
        where[k] = -1;
    }
    for (int i = n_steps - 1; i >= 0; i--) {
        for (int32_t p = offsets[i]; p < offsets[i + 1]; p++) {
            if (keys[p] < 0 || keys[p] >= n_keys)
                goto out;
            nxt[p] = last[keys[p]];
        }
        for (int32_t p = offsets[i]; p < offsets[i + 1]; p++)
            last[keys[p]] = i;
    }
    int nres = 0;
    long long fills = 0;
    for (int i = 0; i < n_steps; i++) {
        if (offsets[i + 1] - offsets[i] > C)
            goto out;
        for (int32_t p = offsets[i]; p < offsets[i + 1]; p++)
            in_step[keys[p]] = 1;
        for (int32_t p = offsets[i]; p < offsets[i + 1]; p++) {
            const int32_t k = keys[p];
            if (where[k] >= 0) {
                res_next[where[k]] = nxt[p];
                continue;
            }
            fills++;
            if (nres == C) {
                int v = -1;
                for (int r = 0; r < nres; r++) {
                    if (in_step[res_key[r]])
                        continue;
                    if (v < 0 || res_next[r] > res_next[v] ||
                        (res_next[r] == res_next[v] && res_key[r] < res_key[v]))
                        v = r;
                }
                if (v < 0)
                    goto out;
                where[res_key[v]] = -1;
                nres--;
                res_key[v] = res_key[nres];
                res_next[v] = res_next[nres];
                if (v < nres)
                    where[res_key[v]] = v;
            }
            res_key[nres] = k;
            res_next[nres] = nxt[p];
            where[k] = nres++;
        }
        for (int32_t p = offsets[i]; p < offsets[i + 1]; p++)
            in_step[keys[p]] = 0;
    }
    misses = fills;
out:
    free(nxt);
    free(last);
    free(res_key);
    free(res_next);
    free(where);
    free(in_step);
    return misses;
}
