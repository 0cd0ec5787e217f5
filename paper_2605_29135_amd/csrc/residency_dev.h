// residency_dev.h -- the device lookup of the slot table as a block-wide device
// function (NT threads, kDevPT slots staged per thread), shared by the lookup
// kernel and by the fused one-token top-k + lookup kernel.  See
// residency_dev.hip for what it decides.
#pragma once
#include "device_common.h"
#include "internal.h"

namespace moe {
namespace devres {

constexpr int kWaveDev = 64;
constexpr int kDevPT = 4;        // slots each thread stages
constexpr int kFastVictims = 8;  // LRU: up to this many victims per step are picked by wave minima, more by a sort
// Threads of the lookup block for a capacity: 256 up to 1024 slots, else 1024.
constexpr int dev_threads(int C) { return C <= kDevPT * 256 ? 256 : 1024; }
static_assert(kDevPT * 1024 == kDevMaxSlots, "the largest lookup block stages every slot");

// The lookup's global reads that do not depend on the step's ids, held in registers: each thread's share of
// the slot keys and their stamps or charges, one entry of the layer's row of the slot table, one counter and
// the step number.  Issued first, so that a caller can overlap them with forming the ids.
struct DevStaged {
    int32_t row;
    int step_v;
    unsigned long long sc0;
    int32_t kv[kDevPT];
    uint64_t sv[kDevPT];
};

template <bool ROTARY, int NT>
__device__ __forceinline__ void dev_stage_issue(const DevResidency &r, const DevLookup &p, DevStaged &st) {
    const int tid = threadIdx.x;
    // clamped indices, no branches: every read is in flight at once
    st.row = r.slot_of_key[p.layer * p.E + min(tid, p.E - 1)];
    st.step_v = p.step_dev ? p.step_dev[0] : p.step;
    st.sc0 = r.scal[min(tid, kDevScalars - 1)];
#pragma unroll
    for (int u = 0; u < kDevPT; ++u) {
        const int sc = min(tid + u * NT, p.C - 1);
        st.kv[u] = r.key_of_slot[sc];
        if constexpr (ROTARY) st.sv[u] = r.charge[sc];
        else st.sv[u] = r.stamp[sc];
    }
}

// ---- fill clock (DevResidency::clk) ----
__device__ __forceinline__ unsigned long long clk_now() { return (unsigned long long)wall_clock64(); }

__device__ __forceinline__ int clk_lane() { return int(blockIdx.x + blockIdx.y) & (kClkLanes - 1); }

// A block that filled from t0 to t1 (called by every thread; lane 0 of wave 0 records).
__device__ __forceinline__ void clk_record_fill(unsigned long long *clk, unsigned long long t0, unsigned long long t1) {
    if (threadIdx.x == 0) {
        atomicMin(clk + kClkFillStart + clk_lane(), t0);
        atomicMax(clk + kClkFillEnd + clk_lane(), t1);
    }
}

// A block of a filling launch that computed and ended at t1.
__device__ __forceinline__ void clk_record_compute(unsigned long long *clk, unsigned long long t1) {
    if (threadIdx.x == 0) atomicMax(clk + kClkComputeEnd + clk_lane(), t1);
}

// Folds the last filling launch's record into the totals and clears it (one thread; the launch has ended,
// being earlier on the stream).
__device__ __forceinline__ void clk_fold(unsigned long long *clk) {
    unsigned long long fs = ~0ull, fe = 0, ce = 0;
#pragma unroll
    for (int i = 0; i < kClkLanes; ++i) {
        fs = min(fs, clk[kClkFillStart + i]);
        fe = max(fe, clk[kClkFillEnd + i]);
        ce = max(ce, clk[kClkComputeEnd + i]);
    }
    if (fe == 0 && ce == 0) return;  // nothing recorded since the last fold
    if (fe > 0 && fe > fs) {
        const unsigned long long from = fs > ce ? fs : ce;
        if (fe > from) clk[kClkStall] += fe - from;
        clk[kClkFill] += fe - fs;
        clk[kClkFolds] += 1;
    }
#pragma unroll
    for (int i = 0; i < kClkLanes; ++i) {
        clk[kClkFillStart + i] = ~0ull;
        clk[kClkFillEnd + i] = 0;
        clk[kClkComputeEnd + i] = 0;
    }
}

// One int per wave in cnt[]: the block total, and the sum over the waves ahead of `wave`.
template <int NW>
__device__ __forceinline__ int wave_prefix(const int *cnt, int wave, int &total) {
    int pre = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        pre += w < wave ? cnt[w] : 0;
        tot += cnt[w];
    }
    total = tot;
    return pre;
}

// The lookup's LDS: the staged slot state and the step's working sets.
template <bool ROTARY, int NT>
struct DevLds {
    static constexpr int NS = kDevPT * NT;  // slots staged (a power of two)
    static constexpr int NW = NT / kWaveDev;
    int32_t key_of[NS];
    uint64_t stamp[ROTARY ? 1 : NS];  // LRU: recency stamps; also the sort buffer of the victims
    uint16_t charge[ROTARY ? NS : 1];
    uint32_t present[MOE_MAX_EXPERTS / 32];
    int32_t R[MOE_MAX_EXPERTS];
    int32_t slot_of_e[MOE_MAX_EXPERTS];  // slot of each expert of the step, by expert id
    int32_t pre[MOE_MAX_EXPERTS];        // slot of each expert of the layer before the step
    unsigned long long scal_sh[kDevScalars];
    int step_sh;
    int bad_sh;
    int wcnt[NW];
    unsigned long long vic_w[ROTARY ? 1 : NW][kFastVictims];
    int vic[ROTARY ? 1 : MOE_MAX_EXPERTS];
};

// The staged registers into LDS (no ids needed: a caller may do this while the ids are formed).  A block
// barrier must follow before dev_lookup_body.
template <bool ROTARY, int NT>
__device__ __forceinline__ void dev_stage_lds(DevLds<ROTARY, NT> &L, const DevLookup &p, const DevStaged &st) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int u = 0; u < kDevPT; ++u) {
        if (u * NT >= p.C) break;  // uniform
        const int s = tid + u * NT;
        if (s < p.C) {
            L.key_of[s] = st.kv[u];
            if constexpr (ROTARY) L.charge[s] = uint16_t(st.sv[u]);
            else L.stamp[s] = st.sv[u];
        }
    }
    if (tid < p.E) L.pre[tid] = st.row;
    if (tid < kDevScalars) L.scal_sh[tid] = st.sc0;
    if (tid < MOE_MAX_EXPERTS / 32) L.present[tid] = 0u;
    if (tid == 0) {
        L.bad_sh = 0;
        L.step_sh = st.step_v;
    }
}

// FORMED: the caller has already set the step's presence bits and its ascending experts R (with bad_sh set
// for an id out of range), before the barrier that precedes this call.
template <bool ROTARY, int NT, bool FORMED = false>
__device__ __forceinline__ void dev_lookup_body(DevLds<ROTARY, NT> &L, const DevResidency &r, const DevLookup &p,
                                                const int32_t *ids, int n, int32_t *__restrict__ slots_out,
                                                int *err) {
    constexpr int NS = DevLds<ROTARY, NT>::NS;
    constexpr int NW = DevLds<ROTARY, NT>::NW;
    int32_t *key_of = L.key_of;
    uint64_t *stamp = L.stamp;
    uint16_t *charge = L.charge;
    uint32_t *present = L.present;
    int32_t *R = L.R, *slot_of_e = L.slot_of_e, *pre = L.pre;
    unsigned long long *scal_sh = L.scal_sh;
    int &step_sh = L.step_sh, &bad_sh = L.bad_sh;
    int *wcnt = L.wcnt;
    auto &vic_w = L.vic_w;
    int *vic = L.vic;
    const int tid = threadIdx.x, lane = tid & (kWaveDev - 1), wave = tid / kWaveDev;
    const int C = p.C, E = p.E, layer = p.layer;
    if constexpr (!FORMED) {
        for (int i = tid; i < n; i += NT) {
            const int e = ids[i];
            if (e < 0 || e >= E) atomicOr(&bad_sh, 1);
            else atomicOr(&present[e >> 5], 1u << (e & 31));
        }
        __syncthreads();
    }
    // the step's unique experts: every thread counts them; thread w writes word w's experts at its offset
    const int nw = (E + 31) / 32;
    int m = 0;
    for (int w = 0; w < nw; ++w) m += __popc(present[w]);
    if (bad_sh || m > C) {  // uniform
        if (tid == 0) {
            atomicOr(err, bad_sh ? kErrRange : kErrBudget);  // no state change, as the host lookup
            r.n_fill[0] = 0;                                  // nothing for the fill kernel to do
        }
        if (slots_out)  // no rank placed: later kernels that read the slots by rank skip them all
            for (int i = tid; i < n; i += NT) slots_out[i] = -1;
        return;
    }
    if constexpr (!FORMED) {
        if (tid < nw) {
            int off = 0;
            for (int w = 0; w < tid; ++w) off += __popc(present[w]);
            for (uint32_t b = present[tid]; b; b &= b - 1u) R[off++] = tid * 32 + __builtin_ctz(b);
        }
        __syncthreads();
    }
    auto pinned = [&](int k2) {  // is slot key k2 an expert of this step?
        const int e2 = k2 - layer * E;
        return e2 >= 0 && e2 < E && ((present[e2 >> 5] >> (e2 & 31)) & 1u);
    };
    int n_fill = 0;
    unsigned long long ctr = scal_sh[kScalCtr], hand = scal_sh[kScalHand], next_free = scal_sh[kScalNextFree],
                       hits = scal_sh[kScalHits], misses = scal_sh[kScalMisses],
                       evictions = scal_sh[kScalEvictions], n_ev = scal_sh[kScalEvents],
                       prefetches = scal_sh[kScalPrefetches];
    // a prefetch inserts the step's non-resident experts (events PREFETCH) and leaves resident ones untouched
    const bool pf = p.prefetch != 0;
    if constexpr (!ROTARY) {
        // LRU in closed form.  Every expert of the step takes the next stamp in ascending-id order, and no slot
        // outside the step changes while the step is decided (hits and new entries are the step's own slots,
        // which are never victims).  So expert j takes stamp ctr + 1 + j and event n_ev + j; a resident one
        // keeps its slot; the q-th miss takes free slot next_free + q while free slots last, and after that the
        // least recently used slots outside the step in ascending stamp order.  Thread j decides expert j
        // (m <= MOE_MAX_EXPERTS <= NT).  A prefetch takes stamps and events for its misses only, in order.
        const bool act = tid < m;
        const int e = act ? R[tid] : 0;
        const int spre = act ? pre[e] : 0;
        const bool miss = act && spre < 0;
        const unsigned long long bal = __ballot(miss);
        if (lane == 0) wcnt[wave] = __popcll(bal);
        __syncthreads();
        int nm;
        const int q = wave_prefix<NW>(wcnt, wave, nm) + __popcll(bal & __lanemask_lt());  // misses ahead of j
        const long long nf0 = (long long)next_free, nfree = (long long)C - nf0;
        const int n_need = nm > nfree ? int(nm - nfree) : 0;  // uniform
        if (n_need > 0) {
            // candidates: occupied slots (0 .. next_free - 1; the free ones above are filled first) outside the
            // step, keyed (stamp << 12) | slot
            if (n_need <= kFastVictims) {
                // each wave takes its share's n_need smallest keys (per-thread sorted lists, one wave minimum
                // per pick); lane 0 merges the NW lists
                unsigned long long cand[kDevPT];
#pragma unroll
                for (int u = 0; u < kDevPT; ++u) {
                    const long long s = tid + u * NT;
                    cand[u] = ~0ull;
                    if (s < nf0 && !pinned(key_of[s])) cand[u] = (stamp[s] << 12) | (unsigned long long)s;
                }
#pragma unroll
                for (int a = 1; a < kDevPT; ++a)  // insertion sort, unrolled
#pragma unroll
                    for (int b = a; b > 0; --b) {
                        const unsigned long long x = cand[b - 1], y = cand[b];
                        cand[b - 1] = x < y ? x : y;
                        cand[b] = x < y ? y : x;
                    }
                for (int k2 = 0; k2 < n_need; ++k2) {
                    const unsigned long long best = dev::wave_reduce_u64<false>(cand[0]);
                    if (lane == 0) vic_w[wave][k2] = best;
                    if (cand[0] == best) {  // unique keys: only the owner matches
#pragma unroll
                        for (int u = 0; u + 1 < kDevPT; ++u) cand[u] = cand[u + 1];
                        cand[kDevPT - 1] = ~0ull;
                    }
                }
                __syncthreads();
                if (wave == 0) {  // the n_need smallest of the waves' NW * n_need picks, by wave minima
                    unsigned long long c0 = ~0ull, c1 = ~0ull;
                    if (lane < NW * n_need) c0 = vic_w[lane / n_need][lane % n_need];
                    if (lane + kWaveDev < NW * n_need) c1 = vic_w[(lane + kWaveDev) / n_need][(lane + kWaveDev) % n_need];
                    for (int k2 = 0; k2 < n_need; ++k2) {
                        const unsigned long long best = dev::wave_reduce_u64<false>(c0 < c1 ? c0 : c1);
                        if (lane == 0) vic[k2] = int(best & 4095ull);
                        if (c0 == best) c0 = ~0ull;  // unique keys: one lane owns it
                        if (c1 == best) c1 = ~0ull;
                    }
                }
            } else {
                // many victims (prefill steps): a bitonic sort of every staged slot's key in the stamp array,
                // non-candidates flagged by the top bit so that they rank after every candidate; then the
                // stamps are put back from the sorted keys
                constexpr unsigned long long kNotCand = 1ull << 63;
                unsigned long long kk[kDevPT];
#pragma unroll
                for (int u = 0; u < kDevPT; ++u) {
                    const int s = tid + u * NT;
                    kk[u] = ~0ull;
                    if (s < C)
                        kk[u] = ((s < nf0 && !pinned(key_of[s])) ? 0ull : kNotCand) | (stamp[s] << 12) |
                                (unsigned long long)s;
                }
                __syncthreads();  // every stamp read before the keys overwrite them
#pragma unroll
                for (int u = 0; u < kDevPT; ++u) stamp[tid + u * NT] = kk[u];
                __syncthreads();
                for (int kb = 2; kb <= NS; kb <<= 1)
                    for (int jb = kb >> 1; jb > 0; jb >>= 1) {
                        for (int i = tid; i < NS; i += NT) {
                            const int l = i ^ jb;
                            if (l > i) {
                                const unsigned long long a = stamp[i], b = stamp[l];
                                if ((a > b) == ((i & kb) == 0)) {
                                    stamp[i] = b;
                                    stamp[l] = a;
                                }
                            }
                        }
                        __syncthreads();
                    }
                for (int k2 = tid; k2 < n_need; k2 += NT) vic[k2] = int(stamp[k2] & 4095ull);
#pragma unroll
                for (int u = 0; u < kDevPT; ++u) kk[u] = stamp[tid + u * NT];
                __syncthreads();  // every sorted key read before the stamps are put back
#pragma unroll
                for (int u = 0; u < kDevPT; ++u)
                    if (kk[u] != ~0ull) stamp[int(kk[u] & 4095ull)] = (kk[u] & ~kNotCand) >> 12;
            }
            __syncthreads();
        }
        if (act) {
            int s = spre, victim = -1;
            if (miss) {
                s = q < nfree ? int(nf0) + q : vic[q - int(nfree)];
                victim = key_of[s];
                const int key = layer * E + e;
                if (victim >= 0) r.slot_of_key[victim] = -1;
                key_of[s] = key;
                r.slot_of_key[key] = s;
                r.fill_src[q] = (long long)layer * p.layer_stride + (long long)e * p.expert_stride;
                r.fill_slot[q] = s;
            }
            slot_of_e[e] = s;
            if (miss || !pf) {
                const unsigned long long rank = (unsigned long long)(pf ? q : tid);
                stamp[s] = ctr + 1 + rank;
                r.stamp[s] = ctr + 1 + rank;  // the only slots the step changes
                if (miss) r.key_of_slot[s] = layer * E + e;
                const unsigned long long ev = n_ev + rank;
                const int kind = miss ? (pf ? MOE_EVENT_PREFETCH : MOE_EVENT_MISS) : MOE_EVENT_HIT;
                if (ev < (unsigned long long)r.cap_events) r.events[ev] = moe_cache_event{step_sh, layer, e, kind, s, victim};
            }
        }
        const int n_dec = pf ? nm : m;  // decisions logged
        ctr += (unsigned long long)n_dec;
        n_ev += (unsigned long long)n_dec;
        next_free += (unsigned long long)(nm < nfree ? nm : nfree);
        if (pf) {
            prefetches += (unsigned long long)nm;
        } else {
            hits += (unsigned long long)(m - nm);
            misses += (unsigned long long)nm;
        }
        evictions += (unsigned long long)n_need;  // free slots held no expert
        n_fill = nm;
    } else {
        // Rotary: lane 0 walks the step's experts in order.  A hit adds a charge; a miss takes the lowest free
        // slot, else the slot where the hand stops: it turns forward past the step's own slots, taking one
        // charge from each charged slot, to the first uncharged one.  Some slot holds an expert outside the step
        // and each full turn takes a charge from every such slot, so the hand stops within charge_max + 1 turns.
        if (tid == 0) {
            for (int j = 0; j < m; ++j) {
                const int e = R[j];
                int s = pre[e], victim = -1;
                const bool miss = s < 0;
                if (!miss) {
                    slot_of_e[e] = s;
                    if (pf) continue;
                    if (charge[s] < p.charge_max) ++charge[s];
                    ++hits;
                } else {
                    if (next_free < (unsigned long long)C) {
                        s = int(next_free++);
                    } else {
                        for (;;) {
                            s = int(hand);
                            hand = hand + 1 == (unsigned long long)C ? 0 : hand + 1;
                            if (pinned(key_of[s])) continue;
                            if (charge[s] > 0) {
                                --charge[s];
                                continue;
                            }
                            break;
                        }
                    }
                    const int key = layer * E + e;
                    victim = key_of[s];
                    if (victim >= 0) {
                        r.slot_of_key[victim] = -1;
                        ++evictions;
                    }
                    key_of[s] = key;
                    r.slot_of_key[key] = s;
                    charge[s] = 0;
                    if (pf) ++prefetches;
                    else ++misses;
                    r.fill_src[n_fill] = (long long)layer * p.layer_stride + (long long)e * p.expert_stride;
                    r.fill_slot[n_fill] = s;
                    ++n_fill;
                }
                slot_of_e[e] = s;
                const int kind = miss ? (pf ? MOE_EVENT_PREFETCH : MOE_EVENT_MISS) : MOE_EVENT_HIT;
                if (n_ev < (unsigned long long)r.cap_events)
                    r.events[n_ev] = moe_cache_event{step_sh, layer, e, kind, s, victim};
                ++n_ev;
            }
        }
    }
    if (tid == 0) {
        r.scal[kScalCtr] = ctr;
        r.scal[kScalHand] = hand;
        r.scal[kScalNextFree] = next_free;
        r.scal[kScalHits] = hits;
        r.scal[kScalMisses] = misses;
        r.scal[kScalEvictions] = evictions;
        r.scal[kScalEvents] = n_ev;
        r.scal[kScalPrefetches] = prefetches;
        r.n_fill[0] = n_fill;
    }
    __syncthreads();
    if (slots_out)
        for (int i = tid; i < n; i += NT) slots_out[i] = slot_of_e[ids[i]];
    if constexpr (ROTARY)  // the hand's turn changes charges along its path
        for (int s = tid; s < C; s += NT) {
            r.key_of_slot[s] = key_of[s];
            r.charge[s] = charge[s];
        }
}

}  // namespace devres
}  // namespace moe
