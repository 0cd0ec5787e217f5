// analysis.cpp -- offline residency bound: the fewest fills any replacement
// policy needs for a demand trace in which each step's experts must be
// resident together (Belady's farthest-next-use rule at step granularity:
// a miss with every slot taken evicts the resident key outside the current
// step whose next step of use is the farthest).  It is the yardstick for the
// LRU residency of the paper's sec. 4 comparison.
#include <stdint.h>

#include <set>
#include <utility>
#include <vector>

#include "internal.h"

extern "C" {

int moe_opt_fills(const int32_t *keys, const int32_t *offsets, int n_steps, int n_keys, int capacity,
                  uint64_t *fills_out) {
    if (!fills_out || n_steps < 0 || n_keys < 1 || capacity < 1 || (n_steps > 0 && (!keys || !offsets)))
        return moe::fail(MOE_ERR_INVALID_ARG, "opt bound: bad argument");
    if (n_steps > 0 && offsets[0] != 0) return moe::fail(MOE_ERR_INVALID_ARG, "opt bound: offsets[0] must be 0");
    for (int i = 0; i < n_steps; ++i)
        if (offsets[i + 1] < offsets[i]) return moe::fail(MOE_ERR_INVALID_ARG, "opt bound: offsets must not decrease");
    const size_t n = n_steps > 0 ? size_t(offsets[n_steps]) : 0;
    for (size_t p = 0; p < n; ++p)
        if (keys[p] < 0 || keys[p] >= n_keys)
            return moe::fail(MOE_ERR_RANGE, "opt bound: key %d outside [0, %d)", keys[p], n_keys);
    const int32_t never = INT32_MAX;
    // next step in which each occurrence's key is needed again
    std::vector<int32_t> nxt(n), last(size_t(n_keys), never);
    std::vector<int32_t> mark(size_t(n_keys), -1);
    for (int i = n_steps - 1; i >= 0; --i) {
        for (int32_t p = offsets[i]; p < offsets[i + 1]; ++p) {
            if (mark[keys[p]] == i) return moe::fail(MOE_ERR_INVALID_ARG, "opt bound: key repeated within a step");
            mark[keys[p]] = i;
            nxt[p] = last[keys[p]];
        }
        for (int32_t p = offsets[i]; p < offsets[i + 1]; ++p) last[keys[p]] = i;
    }
    // evictable resident keys, the farthest next use first (ties: smaller key)
    auto cmp = [](const std::pair<int32_t, int32_t> &a, const std::pair<int32_t, int32_t> &b) {
        return a.first != b.first ? a.first > b.first : a.second < b.second;
    };
    std::set<std::pair<int32_t, int32_t>, decltype(cmp)> evictable(cmp);
    std::vector<int32_t> next_of(size_t(n_keys), -1);
    std::vector<char> resident(size_t(n_keys), 0);
    int nres = 0;
    uint64_t fills = 0;
    for (int i = 0; i < n_steps; ++i) {
        if (offsets[i + 1] - offsets[i] > capacity)
            return moe::fail(MOE_ERR_BUDGET, "opt bound: step %d needs %d keys, capacity %d", i,
                             offsets[i + 1] - offsets[i], capacity);
        for (int32_t p = offsets[i]; p < offsets[i + 1]; ++p)  // the step's own keys stay resident
            if (resident[keys[p]]) evictable.erase({next_of[keys[p]], keys[p]});
        for (int32_t p = offsets[i]; p < offsets[i + 1]; ++p) {
            const int32_t k = keys[p];
            if (!resident[k]) {
                ++fills;
                if (nres == capacity) {
                    const auto v = *evictable.begin();  // non-empty: the step has at most `capacity` keys
                    evictable.erase(evictable.begin());
                    resident[v.second] = 0;
                    --nres;
                }
                resident[k] = 1;
                ++nres;
            }
            next_of[k] = nxt[p];
        }
        for (int32_t p = offsets[i]; p < offsets[i + 1]; ++p) evictable.insert({next_of[keys[p]], keys[p]});
    }
    *fills_out = fills;
    moe::clear_error();
    return MOE_OK;
}

}  // extern "C"
