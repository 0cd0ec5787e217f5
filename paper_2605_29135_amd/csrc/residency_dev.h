// residency_dev.h -- the device lookup of the slot table as a block-wide device
// function (kDevThreads threads), shared by the lookup kernel and by the fused
// one-token top-k + lookup kernel.  See residency_dev.hip for what it decides.
#pragma once
#include "device_common.h"
#include "internal.h"

namespace moe {
namespace devres {

constexpr int kDevThreads = 256;
constexpr int kDevPerThread = kDevMaxSlots / kDevThreads;  // slots each thread stages, at most
// PT = slots each thread stages (ceil(C / kDevThreads) <= PT): 4 up to 1024 slots, else kDevPerThread.
constexpr int dev_pt(int C) { return C <= 4 * kDevThreads ? 4 : kDevPerThread; }
constexpr int kWaveDev = 64;
constexpr int kFastVictims = 8;  // LRU: up to this many victims per step are chosen in one pass

// The lookup's global reads that do not depend on the step's ids, held in registers: each thread's share of
// the slot keys and their stamps or charges, one entry of the layer's row of the slot table, one counter and
// the step number.  Issued first, so that a caller can overlap them with forming the ids.
template <int PT>
struct DevStaged {
    int32_t row;
    int step_v;
    unsigned long long sc0;
    int32_t kv[PT];
    uint64_t sv[PT];
};

template <bool ROTARY, int PT>
__device__ __forceinline__ void dev_stage_issue(const DevResidency &r, const DevLookup &p, DevStaged<PT> &st) {
    const int tid = threadIdx.x;
    // clamped indices, no branches: every read is in flight at once
    st.row = r.slot_of_key[p.layer * p.E + min(tid, p.E - 1)];
    st.step_v = p.step_dev ? p.step_dev[0] : p.step;
    st.sc0 = r.scal[min(tid, kDevScalars - 1)];
#pragma unroll
    for (int u = 0; u < PT; ++u) {
        const int sc = min(tid + u * kDevThreads, p.C - 1);
        st.kv[u] = r.key_of_slot[sc];
        if constexpr (ROTARY) st.sv[u] = r.charge[sc];
        else st.sv[u] = r.stamp[sc];
    }
}

template <bool ROTARY, int PT>
__device__ __forceinline__ void dev_lookup_body(const DevResidency &r, const DevLookup &p, const DevStaged<PT> &st,
                                                const int32_t *ids, int n, int32_t *__restrict__ slots_out,
                                                int *err) {
    __shared__ int32_t key_of[PT * kDevThreads];
    __shared__ uint64_t stamp[ROTARY ? 1 : PT * kDevThreads];
    __shared__ uint16_t charge[ROTARY ? PT * kDevThreads : 1];
    __shared__ uint32_t present[MOE_MAX_EXPERTS / 32];
    __shared__ int32_t R[MOE_MAX_EXPERTS];
    __shared__ int32_t slot_of_e[MOE_MAX_EXPERTS];  // slot of each expert of the step, by expert id
    __shared__ int32_t pre[MOE_MAX_EXPERTS];        // slot of each expert of the layer before the step
    __shared__ unsigned long long scal_sh[kDevScalars];
    __shared__ int step_sh;
    __shared__ int bad_sh, need_sh;
    __shared__ unsigned long long red_v[kDevThreads / kWaveDev];
    __shared__ int red_s[kDevThreads / kWaveDev];
    __shared__ unsigned long long vic_w[ROTARY ? 1 : kDevThreads / kWaveDev][kFastVictims];
    __shared__ int vic[kFastVictims];
    __shared__ int n_need_sh;
    const int tid = threadIdx.x;
    const int C = p.C, E = p.E, layer = p.layer;
    {
        const int32_t id0 = ids[min(tid, max(n - 1, 0))];
#pragma unroll
        for (int u = 0; u < PT; ++u) {
            if (u * kDevThreads >= C) break;  // uniform
            const int s = tid + u * kDevThreads;
            if (s < C) {
                key_of[s] = st.kv[u];
                if constexpr (ROTARY) charge[s] = uint16_t(st.sv[u]);
                else stamp[s] = st.sv[u];
            }
        }
        if (tid < E) pre[tid] = st.row;
        if (tid < kDevScalars) scal_sh[tid] = st.sc0;
        if (tid < MOE_MAX_EXPERTS / 32) present[tid] = 0u;
        if (tid == 0) {
            bad_sh = 0;
            step_sh = st.step_v;
        }
        __syncthreads();
        for (int i = tid; i < n; i += kDevThreads) {
            const int e = i == tid ? id0 : ids[i];  // steps of more than one block of ids read the rest here
            if (e < 0 || e >= E) atomicOr(&bad_sh, 1);
            else atomicOr(&present[e >> 5], 1u << (e & 31));
        }
    }
    __syncthreads();
    // the step's unique experts: every thread counts them; thread w writes word w's experts at its offset
    const int nw = (E + 31) / 32;
    int m = 0;
    for (int w = 0; w < nw; ++w) m += __popc(present[w]);
    if (bad_sh || m > C) {  // uniform
        if (tid == 0) {
            atomicOr(err, bad_sh ? kErrRange : kErrBudget);  // no state change, as the host lookup
            r.n_fill[0] = 0;                                  // nothing for the fill kernel to do
        }
        return;
    }
    if (tid < nw) {
        int off = 0;
        for (int w = 0; w < tid; ++w) off += __popc(present[w]);
        for (uint32_t b = present[tid]; b; b &= b - 1u) R[off++] = tid * 32 + __builtin_ctz(b);
    }
    __syncthreads();
    auto pinned = [&](int k2) {  // is slot key k2 an expert of this step?
        const int e2 = k2 - layer * E;
        return e2 >= 0 && e2 < E && ((present[e2 >> 5] >> (e2 & 31)) & 1u);
    };
    // lane 0 of the block keeps the counters in registers
    unsigned long long ctr = 0, hand = 0, next_free = 0, hits = 0, misses = 0, evictions = 0, n_ev = 0;
    int n_fill = 0;
    if (tid == 0) {
        ctr = scal_sh[kScalCtr];
        hand = scal_sh[kScalHand];
        next_free = scal_sh[kScalNextFree];
        hits = scal_sh[kScalHits];
        misses = scal_sh[kScalMisses];
        evictions = scal_sh[kScalEvictions];
        n_ev = scal_sh[kScalEvents];
    }
    auto log = [&](int e, int kind, int s, int victim) {
        if (n_ev < (unsigned long long)r.cap_events) r.events[n_ev] = moe_cache_event{step_sh, layer, e, kind, s, victim};
        ++n_ev;
    };
    auto place = [&](int e, int s) {  // lane 0: the new entry (layer, e) takes slot s
        const int key = layer * E + e;
        const int victim = key_of[s];
        if (victim >= 0) {
            r.slot_of_key[victim] = -1;
            ++evictions;
        }
        key_of[s] = key;
        r.slot_of_key[key] = s;
        if constexpr (ROTARY) charge[s] = 0;
        else stamp[s] = ++ctr;
        ++misses;
        log(e, MOE_EVENT_MISS, s, victim);
        slot_of_e[e] = s;
        r.fill_src[n_fill] = (long long)layer * p.layer_stride + (long long)e * p.expert_stride;
        r.fill_slot[n_fill] = s;
        ++n_fill;
    };
    // LRU in one pass.  Every expert of the step takes the next stamp in walk order, and every slot outside
    // the step keeps its stamp while the step is walked (hits and new entries are the step's own slots,
    // which are never victims).  So the q-th miss of the walk takes free slot next_free + q while free slots
    // last, and after that the least recently used slots outside the step in ascending stamp order: when
    // the step has at most 64 experts and at most kFastVictims such victims, the victims are picked first
    // (each wave takes its share's smallest (stamp, slot) keys by repeated wave minima, lane 0 merges the
    // four lists) and wave 0 then places every expert at once, lane j the j-th.  Otherwise lane 0 walks.
    bool walked = false;  // uniform
    if constexpr (!ROTARY) {
        const int lane = tid & (kWaveDev - 1), wave = tid / kWaveDev;
        const unsigned long long nf0 = scal_sh[kScalNextFree];
        const long long nfree = (long long)C - (long long)nf0;
        if (m <= kWaveDev) {
            if (wave == 0) {
                const int nm = __popcll(__ballot(lane < m && pre[R[lane]] < 0));
                if (lane == 0) n_need_sh = nm > nfree ? int(nm - nfree) : 0;
            }
            __syncthreads();
            const int n_need = n_need_sh;
            if (n_need <= kFastVictims) {
                if (n_need > 0) {
                    // candidates: occupied slots (0 .. next_free - 1) outside the step, keyed (stamp << 12) |
                    // slot; each thread's sorted ascending, so that its head is its least recent
                    unsigned long long cand[PT];
#pragma unroll
                    for (int u = 0; u < PT; ++u) {
                        const long long s = tid + u * kDevThreads;
                        cand[u] = ~0ull;
                        if (s < (long long)nf0 && !pinned(key_of[s]))
                            cand[u] = (stamp[s] << 12) | (unsigned long long)s;
                    }
#pragma unroll
                    for (int a = 1; a < PT; ++a)  // insertion sort, unrolled
#pragma unroll
                        for (int b = a; b > 0; --b) {
                            const unsigned long long x = cand[b - 1], y = cand[b];
                            cand[b - 1] = x < y ? x : y;
                            cand[b] = x < y ? y : x;
                        }
                    for (int q = 0; q < n_need; ++q) {
                        const unsigned long long best = dev::wave_reduce_u64<false>(cand[0]);
                        if (lane == 0) vic_w[wave][q] = best;
                        if (cand[0] == best) {  // unique keys: only the owner matches
#pragma unroll
                            for (int u = 0; u + 1 < PT; ++u) cand[u] = cand[u + 1];
                            cand[PT - 1] = ~0ull;
                        }
                    }
                    __syncthreads();
                    if (tid == 0) {
                        int pos[kDevThreads / kWaveDev] = {};
                        for (int q = 0; q < n_need; ++q) {
                            int bw = 0;
                            unsigned long long bv = ~0ull;
                            for (int w = 0; w < kDevThreads / kWaveDev; ++w)
                                if (pos[w] < n_need && vic_w[w][pos[w]] < bv) {
                                    bv = vic_w[w][pos[w]];
                                    bw = w;
                                }
                            vic[q] = int(bv & 4095ull);
                            ++pos[bw];
                        }
                    }
                }
                if (wave == 0) {
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");  // lane 0's victims to its wave
                    __builtin_amdgcn_wave_barrier();
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
                    const bool act = lane < m;
                    const int e = act ? R[lane] : 0;
                    const int spre = act ? pre[e] : 0;
                    const bool miss = act && spre < 0;
                    const unsigned long long mmask = __ballot(miss);
                    const int q = __popcll(mmask & __lanemask_lt());  // misses ahead of this one
                    const int nm = __popcll(mmask);
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
                    if (act) {
                        stamp[s] = scal_sh[kScalCtr] + 1 + (unsigned long long)lane;
                        slot_of_e[e] = s;
                        const unsigned long long ev = scal_sh[kScalEvents] + (unsigned long long)lane;
                        if (ev < (unsigned long long)r.cap_events)
                            r.events[ev] = moe_cache_event{step_sh, layer, e, miss ? MOE_EVENT_MISS : MOE_EVENT_HIT,
                                                           s, victim};
                    }
                    const int n_evict = __popcll(__ballot(miss && victim >= 0));
                    if (lane == 0) {
                        ctr += (unsigned long long)m;
                        next_free += (unsigned long long)(nm < nfree ? nm : nfree);
                        hits += (unsigned long long)(m - nm);
                        misses += (unsigned long long)nm;
                        evictions += (unsigned long long)n_evict;
                        n_ev += (unsigned long long)m;
                        n_fill = nm;
                    }
                }
                walked = true;
            }
        }
    }
    // Otherwise lane 0 of the block walks the step's experts in order, with no block barrier, until an LRU
    // miss finds no free slot; then the whole block looks for the least recently used slot outside the step,
    // lane 0 places the expert there, and the walk goes on.  A resident expert of the step keeps its slot for
    // the whole step (victims are never the step's own), so the row read at the start stays valid.
    int j = 0;  // lane 0's position in R
    while (!walked) {
        if (tid == 0) {
            need_sh = 0;
            for (; j < m; ++j) {
                const int e = R[j];
                const int s = pre[e];
                if (s >= 0) {
                    if constexpr (ROTARY) {
                        if (charge[s] < p.charge_max) ++charge[s];
                    } else {
                        stamp[s] = ++ctr;
                    }
                    ++hits;
                    slot_of_e[e] = s;
                    log(e, MOE_EVENT_HIT, s, -1);
                } else if (next_free < (unsigned long long)C) {
                    place(e, int(next_free++));
                } else if constexpr (ROTARY) {
                    // some slot holds an expert outside the step, and each full turn takes a charge from
                    // every such slot, so the hand stops within charge_max + 1 turns
                    int s2;
                    for (;;) {
                        s2 = int(hand);
                        hand = hand + 1 == (unsigned long long)C ? 0 : hand + 1;
                        if (pinned(key_of[s2])) continue;
                        if (charge[s2] > 0) {
                            --charge[s2];
                            continue;
                        }
                        break;
                    }
                    place(e, s2);
                } else {
                    need_sh = 1;  // R[j] waits for the block-wide search
                    break;
                }
            }
        }
        __syncthreads();
        if (!need_sh) break;  // every thread read the same value after the barrier
        if constexpr (!ROTARY) {
            // least recently used slot outside the step (stamps are unique)
            unsigned long long best = ~0ull;
            int bs = -1;
            for (int s = tid; s < C; s += kDevThreads)
                if (!pinned(key_of[s]) && stamp[s] < best) {
                    best = stamp[s];
                    bs = s;
                }
#pragma unroll
            for (int off = kWaveDev / 2; off > 0; off >>= 1) {
                const unsigned long long ob = __shfl_xor(best, off);
                const int os = __shfl_xor(bs, off);
                if (ob < best) {
                    best = ob;
                    bs = os;
                }
            }
            if ((tid & (kWaveDev - 1)) == 0) {
                red_v[tid / kWaveDev] = best;
                red_s[tid / kWaveDev] = bs;
            }
            __syncthreads();
            if (tid == 0) {
                for (int w = 1; w < kDevThreads / kWaveDev; ++w)
                    if (red_v[w] < best) {
                        best = red_v[w];
                        bs = red_s[w];
                    }
                place(R[j], bs);
                ++j;
            }
            // the search read need_sh and the state before lane 0 changes them in the next round
            __syncthreads();
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
        r.n_fill[0] = n_fill;
    }
    __syncthreads();
    if (slots_out)
        for (int i = tid; i < n; i += kDevThreads) slots_out[i] = slot_of_e[ids[i]];
    for (int s = tid; s < C; s += kDevThreads) {
        r.key_of_slot[s] = key_of[s];
        if constexpr (ROTARY) r.charge[s] = charge[s];
        else r.stamp[s] = stamp[s];
    }
}

}  // namespace devres
}  // namespace moe
