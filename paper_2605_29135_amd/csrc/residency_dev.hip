// residency_dev.hip -- the slot table's replacement decisions made on the device.
//
// The residency of sec. 4 and Fig. 1 (host tier, slot group, lookup table from
// sub-module id to slot, selective load, evict) with every decision taken by a
// kernel, so that a decode step enqueues route -> lookup -> fills -> expert FFN
// for every layer without waiting for the host.  One lookup kernel per step
// (one block): it stages the slot keys and their stamps (LRU) or charges
// (rotary) in LDS, forms the step's ascending unique experts from a presence
// bitmap, and takes the same decisions, in the same order, as the host runtime:
// a hit refreshes its slot; a miss takes the lowest free slot, else the least
// recently used slot whose expert the step does not need (LRU: every expert of
// the step decided at once by its own thread, the victims picked first) or the
// slot where the forward rotation stops (rotary: one lane turns the hand over the
// LDS copy).  Each decision is logged, the slot table is updated in place, and
// the misses form a fill list that the fill kernel then streams from pinned host
// memory.
#include "residency_dev.h"

namespace moe {
namespace {

using namespace devres;
// Loads each fill thread keeps in flight.  With 32 blocks per expert that is 256 KiB of PCIe reads in flight
// per fill: a sweep of blocks x loads (256 KiB to 2 MiB per fill) over the decode stack measured the
// smallest in flight fastest (2 MiB: 75 tokens/s, 1 MiB: 77.8, 256 KiB: 80.0).
constexpr int kFillUnrollDev = 2;
constexpr int kFillThreads = 256;
constexpr int kFillsInFlight = 4;  // fills streamed at once

template <bool ROTARY, int NT>
__global__ __launch_bounds__(NT) void dev_lookup_kernel(DevResidency r, DevLookup p, const int32_t *__restrict__ ids,
                                                        int n, int32_t *__restrict__ slots_out, int *err) {
    __shared__ DevLds<ROTARY, NT> L;
    DevStaged st;
    dev_stage_issue<ROTARY, NT>(r, p, st);
    if (threadIdx.x == NT - 1 && r.clk) clk_fold(r.clk);
    dev_stage_lds<ROTARY, NT>(L, p, st);
    __syncthreads();
    dev_lookup_body<ROTARY, NT>(L, r, p, ids, n, slots_out, err);
}

// Block (x, y) streams its share of fills y, y + gridDim.y, ...; blocks past the lookup's fill count exit.
// The grid covers a few fills at a time: a prefetch of a whole layer (hundreds of fills) then keeps the
// same bytes in flight as a decode step's fills and leaves most compute units to the kernels it overlaps.
// With clk (demand fills) each block that streamed something records its span in the fill clock.
__global__ __launch_bounds__(kFillThreads) void dev_fill_kernel(const long long *__restrict__ src_off,
                                                               const int32_t *__restrict__ slot,
                                                               const int32_t *__restrict__ n_fill,
                                                               const uint8_t *__restrict__ host_dev,
                                                               uint8_t *__restrict__ pool, long long bytes,
                                                               unsigned long long *clk) {
    const int nf = n_fill[0];
    const unsigned long long t0 = clk && int(blockIdx.y) < nf ? clk_now() : 0ull;
    const size_t n16 = size_t(bytes) / 16;
    const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const size_t beg = size_t(blockIdx.x) * per;
    const size_t end = beg + per < n16 ? beg + per : n16;
    for (int f = blockIdx.y; f < nf; f += gridDim.y) {
        const uint4 *src = reinterpret_cast<const uint4 *>(host_dev + src_off[f]);
        uint4 *dst = reinterpret_cast<uint4 *>(pool + size_t(slot[f]) * size_t(bytes));
        for (size_t i = beg + threadIdx.x; i < end; i += size_t(kFillThreads) * kFillUnrollDev) {
            uint4 v[kFillUnrollDev];
#pragma unroll
            for (int u = 0; u < kFillUnrollDev; ++u) {
                const size_t j = i + size_t(u) * kFillThreads;
                v[u] = j < end ? src[j] : make_uint4(0u, 0u, 0u, 0u);
            }
#pragma unroll
            for (int u = 0; u < kFillUnrollDev; ++u) {
                const size_t j = i + size_t(u) * kFillThreads;
                if (j < end) dst[j] = v[u];
            }
        }
    }
    if (t0) clk_record_fill(clk, t0, clk_now());
}

__global__ void set_int_kernel(int *p, int v) { *p = v; }

}  // namespace

hipError_t launch_set_int(int *p, int v, hipStream_t s) {
    set_int_kernel<<<1, 1, 0, s>>>(p, v);
    return hipGetLastError();
}

hipError_t launch_dev_lookup(const DevResidency &r, const DevLookup &p, const int32_t *ids, int n, int32_t *slots_out,
                             int *err, hipStream_t s) {
    if (p.C < 1 || p.C > kDevMaxSlots || p.E < 1 || p.E > MOE_MAX_EXPERTS || p.layer < 0 || p.layer >= p.L || n < 0)
        return hipErrorInvalidValue;
    const bool small = dev_threads(p.C) == 256;
    if (p.rotary && small) dev_lookup_kernel<true, 256><<<1, 256, 0, s>>>(r, p, ids, n, slots_out, err);
    else if (p.rotary) dev_lookup_kernel<true, 1024><<<1, 1024, 0, s>>>(r, p, ids, n, slots_out, err);
    else if (small) dev_lookup_kernel<false, 256><<<1, 256, 0, s>>>(r, p, ids, n, slots_out, err);
    else dev_lookup_kernel<false, 1024><<<1, 1024, 0, s>>>(r, p, ids, n, slots_out, err);
    return hipGetLastError();
}

hipError_t launch_dev_fill(const DevResidency &r, const uint8_t *host_dev, uint8_t *pool, long long expert_bytes,
                           int max_fills, hipStream_t s, bool demand) {
    if (max_fills < 1) return hipSuccess;
    if (expert_bytes <= 0 || expert_bytes % 16) return hipErrorInvalidValue;
    long long bpf = expert_bytes / (64 << 10);  // 32 blocks for a 9 MiB blob
    bpf = bpf < 4 ? 4 : (bpf > 32 ? 32 : bpf);
    const int ny = max_fills < kFillsInFlight ? max_fills : kFillsInFlight;
    dev_fill_kernel<<<dim3(unsigned(bpf), unsigned(ny)), kFillThreads, 0, s>>>(r.fill_src, r.fill_slot,
                                                                                     r.n_fill, host_dev, pool,
                                                                                     expert_bytes,
                                                                                     demand ? r.clk : nullptr);
    return hipGetLastError();
}

}  // namespace moe
