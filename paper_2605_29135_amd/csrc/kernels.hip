// kernels.hip -- gfx950 kernels of the MoE decode step.
//
// Every kernel streams weight rows with 16-byte loads per lane, so one wave
// instruction moves 1 KiB of a row; dot products reduce across the 64-wide
// wave with cross-lane shuffles.  fp32 accumulation throughout; bf16 and int4
// weights widen to fp32 exactly in registers.
#include <limits.h>
#include <math.h>

#include "internal.h"
#include "device_common.h"
#include "residency_dev.h"
#include "../../include/moe_budget.h"

namespace moe {
namespace {

using namespace dev;


constexpr int kDownRows = 2; // output rows per wave in the down projection (fallback kernel)
// Output rows per wave of down_combine_lds_kernel: one (two, sharing the LDS reads of the activations,
// measured slower on config 4: 6.62 against 6.39 us).
constexpr int kDownWaveRows = 1;
#ifndef MOE_DOWN_BLOCK
#define MOE_DOWN_BLOCK 512
#endif
// Threads per block of down_combine_lds_kernel: each block stages the token's activations once for its
// kDownBlock / 64 output rows (512: 6.66 -> 6.33 us for config 4's bf16 down, 4.36 -> 4.10 us for config 5's
// int4 against 256; 1024 would leave half the compute units without a block at H = 2048).
constexpr int kDownBlock = MOE_DOWN_BLOCK;
constexpr int kDownSlots = 4; // 16-byte chunks per lane per pass of the down projection
constexpr float kRmsEps = 1e-6f;
constexpr int kRouterMfmaMinTokens = 16;  // from this many tokens on, bf16 routers run on the matrix cores

// ---------------------------------------------------------------- top-k ---
// Order-preserving 32-bit key of a finite float (-0 ranks with +0).
__device__ __forceinline__ uint32_t order_key(float z) {
    uint32_t u = __float_as_uint(z);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float order_key_value(uint32_t key) {  // inverse of order_key (-0 comes back +0)
    return __uint_as_float((key & 0x80000000u) ? (key ^ 0x80000000u) : ~key);
}

struct TopkScratch {  // per wave, in LDS: the selected ids and logits in rank order
    int32_t rid[MOE_MAX_TOPK];
    float rz[MOE_MAX_TOPK];
};

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Top-k of one token's E (<= 256) logits by one wave: ids ranked by (z desc, id
// asc) and the softmax over the k selected.  Each entry is a 64-bit rank key
// (order key of z, then the complement of its id, so that a larger key is
// ahead); every lane sorts its (up to 4) keys in registers, then k rounds each
// take the wave maximum of the lanes' heads -- the next entry in rank order --
// and the owning lane advances its list.
// The wave's loads of the logits: lane l takes entries l, l + 64, l + 128, l + 192, every load unconditional
// (clamped index) so that the four are in flight together; entries past E are masked by topk_wave_ranked.
__device__ __forceinline__ void topk_wave_load(const float *z, int E, float *zv) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int m = 0; m < 4; ++m) zv[m] = z[min(lane + kWave * m, E - 1)];
}

__device__ void topk_wave_ranked(const float *zv, int E, int k, int32_t *ids, float *wout, int *err,
                                 TopkScratch *sc) {
    const int lane = threadIdx.x & (kWave - 1);
    uint64_t c[4];
    bool bad = false;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const int e = lane + kWave * m;
        const bool live = e < E;
        const float v = live ? zv[m] : 0.f;
        if (live && !isfinite(v)) bad = true;
        // a live key is at least order_key(-FLT_MAX) << 32 > 0, so 0 never outranks a live entry
        c[m] = live ? (uint64_t(order_key(v)) << 32) | uint64_t(~uint32_t(e)) : 0ull;
    }
    if (__any(bad)) {
        if (lane < k) {
            ids[lane] = -1;
            wout[lane] = 0.f;
            sc->rid[lane] = -1;
        }
        if (lane == 0) atomicOr(err, kErrNonfinite);
        __builtin_amdgcn_wave_barrier();
        return;
    }
    auto cswap = [&](int a, int b) {  // descending
        const uint64_t x = c[a], y = c[b];
        c[a] = x > y ? x : y;
        c[b] = x > y ? y : x;
    };
    cswap(0, 1);
    cswap(2, 3);
    cswap(0, 2);
    cswap(1, 3);
    cswap(1, 2);
    for (int r = 0; r < k; ++r) {
        // the top key among the lanes' heads; the lowest id among heads sharing it (rare) by a second reduce
        const uint32_t hk = uint32_t(c[0] >> 32);
        const uint32_t top = wave_reduce_u32<true>(hk);
        const uint64_t tied = __ballot(hk == top);
        int wl = int(__builtin_ctzll(tied));
        if (__popcll(tied) > 1) {
            const uint32_t lo = hk == top ? uint32_t(c[0]) : 0u;  // complement of the id: larger is lower
            const uint32_t lo_top = wave_reduce_u32<true>(lo);    // every lane takes part (not under the &&)
            wl = int(__builtin_ctzll(__ballot(hk == top && lo == lo_top)));
        }
        const uint64_t best = (uint64_t(top) << 32) | uint64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(c[0])), wl)));
        const int id = int(~uint32_t(best));
        if (lane == wl) {
            c[0] = c[1];
            c[1] = c[2];
            c[2] = c[3];
            c[3] = 0ull;
        }
        if (lane == 0) {
            sc->rid[r] = id;
            sc->rz[r] = order_key_value(uint32_t(best >> 32));
        }
    }
    wave_lds_sync();
    // softmax against the top logit, the denominator summed in rank order
    const float z0 = sc->rz[0];
    const float ez = lane < k ? expf(sc->rz[lane] - z0) : 0.f;
    float sum = 0.f;
    for (int j = 0; j < k; ++j) sum += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ez), j));
    if (lane < k) {
        ids[lane] = sc->rid[lane];
        wout[lane] = ez / sum;
    }
}

__device__ void topk_wave(const float *z, int E, int k, int32_t *ids, float *wout, int *err, TopkScratch *sc) {
    float zv[4];
    topk_wave_load(z, E, zv);
    topk_wave_ranked(zv, E, k, ids, wout, err, sc);
}

// One wave per token.
// With `pub` (one token), the wave also publishes its ids to host memory: the
// ids, then a system-scope fence, then the sequence number `seq` in pub->seq,
// so a host that sees the new sequence number reads complete ids.
__global__ __launch_bounds__(kBlock) void topk_softmax_kernel(const float *__restrict__ logits, int T,
                                                              int E, int k, int32_t *__restrict__ ids,
                                                              float *__restrict__ wout, int *err,
                                                              IdsMailbox *pub, uint32_t seq,
                                                              const float *__restrict__ h_src, float *h_pub,
                                                              int H) {
    __shared__ TopkScratch sc[kBlock / kWave];
    const int wave = threadIdx.x / kWave;
    const int t = blockIdx.x * (kBlock / kWave) + wave;
    if (t >= T) return;
    topk_wave(logits + size_t(t) * E, E, k, ids + size_t(t) * k, wout + size_t(t) * k, err, &sc[wave]);
    if (pub && t == 0) {
        const int lane = threadIdx.x & (kWave - 1);
        if (lane < k) {  // this lane wrote ids[lane] and wout[lane] itself
            pub->ids[lane] = ids[lane];
            pub->w[lane] = wout[lane];
        }
        if (h_pub)
            for (int i = 4 * lane; i < H; i += 4 * kWave)
                *reinterpret_cast<float4 *>(h_pub + i) = *reinterpret_cast<const float4 *>(h_src + i);
        __threadfence_system();
        if (lane == 0) __hip_atomic_store(&pub->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

// One token's top-k fused with the device lookup of its experts (MOE_CACHE_DEVICE
// decode): every thread first issues its reads of the slot state, then wave 0
// ranks the experts and writes ids and weights while the other waves stage the
// slot state in LDS, then the whole block takes the slot table's decisions for
// them -- one launch and one global round trip before the decisions.
template <bool ROTARY, int NT>
__global__ __launch_bounds__(NT) void topk_lookup_kernel(const float *__restrict__ logits, int E, int k,
                                                             int32_t *__restrict__ ids, float *__restrict__ wout,
                                                             int *err, DevResidency r, DevLookup p,
                                                             int32_t *__restrict__ slots_out) {
    __shared__ TopkScratch sc;
    __shared__ int32_t ids_l[MOE_MAX_TOPK];
    __shared__ devres::DevLds<ROTARY, NT> L;
    float zv[4];  // wave 0: the logits, loaded before the slot state so that ranking waits for them alone
    if (threadIdx.x < kWave) topk_wave_load(logits, E, zv);
    devres::DevStaged st;
    devres::dev_stage_issue<ROTARY, NT>(r, p, st);
    if (threadIdx.x == NT - 1 && r.clk) devres::clk_fold(r.clk);  // the previous filling launch's record
    const int lane = threadIdx.x & (kWave - 1);
    if (threadIdx.x < kWave) {
        topk_wave_ranked(zv, E, k, ids, wout, err, &sc);
        // (keeps the staging below -- it waits for the slot-state loads -- after the ranking, which needs only
        // the logits: the compiler may otherwise hoist the staging that both branches share above it)
        asm volatile("" ::: "memory");
        const int id = lane < k ? sc.rid[lane] : 0;  // the ranked ids (-1 if non-finite)
        if (lane < k) ids_l[lane] = id;
        devres::dev_stage_lds<ROTARY, NT>(L, p, st);  // wave 0's share (it clears the presence bits)
        // the step's ascending experts and presence bits from the k distinct ids
        int rank = 0;
        for (int j = 0; j < k; ++j) rank += __builtin_amdgcn_readlane(id, j) < id;
        const bool bad = lane < k && (id < 0 || id >= E);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");  // the cleared bits before the new ones
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        if (lane < k && !bad) {
            L.R[rank] = id;
            atomicOr(&L.present[id >> 5], 1u << (id & 31));
        }
        if (__any(bad) && lane == 0) L.bad_sh = 1;
    } else {
        devres::dev_stage_lds<ROTARY, NT>(L, p, st);  // the other waves stage while wave 0 ranks
    }
    __syncthreads();
    devres::dev_lookup_body<ROTARY, NT, true>(L, r, p, ids_l, k, slots_out, err);
}

// --------------------------------------------------------------- router ---
// z[t, e] = W_r[e, :] . h_t (+ bias[t, e]) with h_t = x_t, or with NORM
// h_t = x_t / sqrt(mean(x_t^2) + eps); one wave per (token, expert row).  Each
// wave holds the whole token row (one 16-byte column chunk per lane and
// pass), so it forms the norm itself; wave 0 of the token's first block
// stores h_t for the expert FFN.  The same GEMV serves the attention block's
// projections; `bias` may be `logits` itself (an in-place residual add: each
// element is read and then written by the same lane).
template <int DT, int NCH, bool NORM, bool FULL>
__global__ __launch_bounds__(kBlock) void router_logits_kernel(const float *__restrict__ x,
                                                               const uint8_t *__restrict__ w, int H,
                                                               int E, const float *bias, float *logits,
                                                               float *__restrict__ h_out) {
    constexpr int EPC = Fmt<DT>::EPC;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int e = blockIdx.x * (kBlock / kWave) + wave;
    const int t = blockIdx.y;
    const float *xt = x + size_t(t) * H;
    const uint8_t *row = w + size_t(e < E ? e : 0) * row_bytes_of(DT, H);
    uint4 wv[NCH];
    float xv[NCH][EPC];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {  // x first: waiting for it never waits for the weight loads
        const int col0 = (c * kWave + lane) * EPC;
        if ((FULL || col0 < H)) {
            load_x<DT>(xt, col0, xv[c]);
        } else {
#pragma unroll
            for (int q = 0; q < EPC; ++q) xv[c][q] = 0.f;
        }
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int col0 = (c * kWave + lane) * EPC;
        // (a wave past E reads row 0 and stores nothing: no branch, so the loads are in flight together)
        wv[c] = (FULL || col0 < H) ? load16(row + row_bytes_of(DT, col0)) : make_uint4(0, 0, 0, 0);
    }
    if constexpr (NORM) {
        float ss = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
            for (int q = 0; q < EPC; ++q) ss = fmaf(xv[c][q], xv[c][q], ss);
        const float inv = rsqrtf(wave_sum(ss) / float(H) + kRmsEps);
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
            for (int q = 0; q < EPC; ++q) xv[c][q] *= inv;
        if (h_out && blockIdx.x == 0 && wave == 0) {
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                const int col0 = (c * kWave + lane) * EPC;
                if ((FULL || col0 < H)) {
                    float4 *o = reinterpret_cast<float4 *>(h_out + size_t(t) * H + col0);
#pragma unroll
                    for (int q = 0; q < EPC / 4; ++q)
                        o[q] = make_float4(xv[c][4 * q], xv[c][4 * q + 1], xv[c][4 * q + 2], xv[c][4 * q + 3]);
                }
            }
        }
    }
    if (e < E) {
        float acc = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; ++c) acc += chunk_dot<DT>(wv[c], xv[c]);
        acc = wave_sum(acc);
        if (lane == 0) logits[size_t(t) * E + e] = acc + (bias ? bias[size_t(t) * E + e] : 0.f);
    }
}

// ------------------------------------------------- router on the matrix cores ---
// For many tokens (a prefill chunk) the router is a [T x H] x [H x E] product.
// Each x value is split exactly into three bf16 terms x = x1 + x2 + x3
// (x1 = bf16(x), x2 = bf16(x - x1), x3 = bf16(x - x1 - x2): 24 mantissa bits in
// all), so with bf16 router weights every MFMA product is exact and the fp32
// result differs from a sequential fp32 dot product only in summation order.
typedef __bf16 rbf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 rbf16x2 __attribute__((ext_vector_type(2)));
typedef float rfloatx2 __attribute__((ext_vector_type(2)));
typedef float rfloatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t rpack2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(rfloatx2{lo, hi}, rbf16x2));
}

// Eight fp32 values -> three bf16x8 terms whose sum is exact.
__device__ __forceinline__ void split3(const float *v, rbf16x8 &t1, rbf16x8 &t2, rbf16x8 &t3) {
    uint32_t a[4], b[4], c[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float x0 = v[2 * e], x1 = v[2 * e + 1];
        a[e] = rpack2(x0, x1);
        const float r0 = x0 - __uint_as_float(a[e] << 16), r1 = x1 - __uint_as_float(a[e] & 0xffff0000u);
        b[e] = rpack2(r0, r1);
        const float q0 = r0 - __uint_as_float(b[e] << 16), q1 = r1 - __uint_as_float(b[e] & 0xffff0000u);
        c[e] = rpack2(q0, q1);
    }
    t1 = __builtin_bit_cast(rbf16x8, make_uint4(a[0], a[1], a[2], a[3]));
    t2 = __builtin_bit_cast(rbf16x8, make_uint4(b[0], b[1], b[2], b[3]));
    t3 = __builtin_bit_cast(rbf16x8, make_uint4(c[0], c[1], c[2], c[3]));
}

constexpr int kRouterTileT = 16;   // tokens per block (one MFMA row block)
constexpr int kRouterTileE = 32;   // experts per block (two 16-column MFMA blocks)
constexpr int kRouterKWaves = 8;   // waves per block, each over its own slice of the H range
constexpr int kRouterRound = 8;    // 32-wide k steps whose loads a wave issues together

// h = x / sqrt(mean(x^2) + eps), one wave per token.
__global__ __launch_bounds__(kBlock) void rmsnorm_rows_kernel(const float *__restrict__ x, int T, int H,
                                                              float *__restrict__ h) {
    const int lane = threadIdx.x & (kWave - 1);
    const int t = blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
    if (t >= T) return;
    const float4 *xr = reinterpret_cast<const float4 *>(x + size_t(t) * H);
    float ss = 0.f;
    for (int c = lane; c < H / 4; c += kWave) {
        const float4 v = xr[c];
        ss = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, ss))));
    }
    const float inv = rsqrtf(wave_sum(ss) / float(H) + kRmsEps);
    float4 *hr = reinterpret_cast<float4 *>(h + size_t(t) * H);
    for (int c = lane; c < H / 4; c += kWave) {
        const float4 v = xr[c];
        hr[c] = make_float4(v.x * inv, v.y * inv, v.z * inv, v.w * inv);
    }
}

// logits[t, e] = sum_i W[e, i] x[t, i] (+ bias[t, e]); W bf16 [E x H], H % 32 == 0.
// A block takes 16 tokens x 32 experts; its 8 waves split the H range into
// contiguous slices of 32-wide k steps, each wave issuing the loads of up to 8
// steps before its first product (lane (lr = l % 16, lg = l / 16) supplies
// x[t0 + lr][k + 8lg .. +7] and W[e0 + 16j + lr][k + 8lg .. +7]), and the
// waves' partial tiles are summed through LDS in wave order.
__global__ __launch_bounds__(kRouterKWaves * kWave) void router_mfma_kernel(const float *__restrict__ x,
                                                                           const uint16_t *__restrict__ w, int T,
                                                                           int H, int E,
                                                                           const float *__restrict__ bias,
                                                                           float *__restrict__ logits) {
    __shared__ float red[kRouterKWaves][2 * 4 * kWave];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int lr = lane % 16, lg = lane / 16;
    const int t0 = blockIdx.y * kRouterTileT, e0 = blockIdx.x * kRouterTileE;
    const float *xr = x + size_t(min(t0 + lr, T - 1)) * H + 8 * lg;
    const uint16_t *wr0 = w + size_t(min(e0 + lr, E - 1)) * H + 8 * lg;
    const uint16_t *wr1 = w + size_t(min(e0 + 16 + lr, E - 1)) * H + 8 * lg;
    const int nk = H / 32;                                     // k steps in all
    const int ns = (nk + kRouterKWaves - 1) / kRouterKWaves;   // steps per wave
    const int s_lo = wave * ns, s_hi = min(nk, s_lo + ns);     // this wave's steps (wave-uniform)
    rfloatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    static_assert(kRouterRound == 8, "the load fence below names eight steps");
    for (int r0 = s_lo; r0 < s_hi; r0 += kRouterRound) {
        u32x4 xa[kRouterRound], xb[kRouterRound], wa[kRouterRound], wb[kRouterRound];
#pragma unroll
        for (int r = 0; r < kRouterRound; ++r) {  // every load issued (step clamped), products only for live steps
            const int k = 32 * min(r0 + r, nk - 1);
            xa[r] = *reinterpret_cast<const u32x4 *>(xr + k);
            xb[r] = *reinterpret_cast<const u32x4 *>(xr + k + 4);
            wa[r] = *reinterpret_cast<const u32x4 *>(wr0 + k);
            wb[r] = *reinterpret_cast<const u32x4 *>(wr1 + k);
        }
        // One fence over every loaded register: the compiler cannot move a load past it, so the round's loads
        // are in flight together and the wave waits once (left to itself it interleaves each step's loads with
        // the previous step's products, one load latency per step).
#define RFENCE(r) "+v"(xa[r]), "+v"(xb[r]), "+v"(wa[r]), "+v"(wb[r])
        asm volatile("" : RFENCE(0), RFENCE(1), RFENCE(2), RFENCE(3), RFENCE(4), RFENCE(5), RFENCE(6), RFENCE(7));
#undef RFENCE
#pragma unroll
        for (int r = 0; r < kRouterRound; ++r) {
            // a step past the wave's slice multiplies zero weights (no branch around the products)
            const bool live = r0 + r < s_hi;
            const float v[8] = {__uint_as_float(xa[r].x), __uint_as_float(xa[r].y), __uint_as_float(xa[r].z),
                                __uint_as_float(xa[r].w), __uint_as_float(xb[r].x), __uint_as_float(xb[r].y),
                                __uint_as_float(xb[r].z), __uint_as_float(xb[r].w)};
            const u32x4 z4 = {0u, 0u, 0u, 0u};
            const rbf16x8 b0 = __builtin_bit_cast(rbf16x8, live ? wa[r] : z4);
            const rbf16x8 b1 = __builtin_bit_cast(rbf16x8, live ? wb[r] : z4);
            rbf16x8 a1, a2, a3;
            split3(v, a1, a2, a3);
            // smallest terms first
            acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a3, b0, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a3, b1, acc1, 0, 0, 0);
            acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, b0, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, b1, acc1, 0, 0, 0);
            acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b0, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b1, acc1, 0, 0, 0);
        }
    }
    // lane holds C[t = t0 + 4lg + q][e = e0 + 16j + lr] in acc_j[q]; entry (j, q, lane) of the tile is
    // red[.][(j * 4 + q) * 64 + lane]
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        red[wave][q * kWave + lane] = acc0[q];
        red[wave][(4 + q) * kWave + lane] = acc1[q];
    }
    __syncthreads();
    const int i = threadIdx.x;  // one tile entry per thread: 8 x 64 entries, 512 threads
    float v = 0.f;
#pragma unroll
    for (int wv = 0; wv < kRouterKWaves; ++wv) v += red[wv][i];
    const int j = i / (4 * kWave), q = (i / kWave) % 4, l = i % kWave;
    const int t = t0 + 4 * (l / 16) + q, e = e0 + 16 * j + l % 16;
    if (t < T && e < E) logits[size_t(t) * E + e] = v + (bias ? bias[size_t(t) * E + e] : 0.f);
}

// ------------------------------------------------------------- grouping ---
// Group table in the workspace (int32):
//   [0] groups (routed + shared)  [1] routed groups  [2] valid routed pairs  [3] unused
//   slot[G] start[G] count[G] pairs[P + T]     with G = T*k + 1, P = T*k
// Pair p = t*k + j is (token t, rank j); the shared expert's pairs are P + t.
// Groups list the distinct valid experts in ascending id; a group's pairs
// are ascending.  slot -2 marks the shared expert's group.
__device__ __forceinline__ int *group_slot(int *g, int T, int k) { return g + 4; }
__device__ __forceinline__ int *group_start(int *g, int T, int k) { return g + 4 + (T * k + 1); }
__device__ __forceinline__ int *group_count(int *g, int T, int k) { return g + 4 + 2 * (T * k + 1); }
__device__ __forceinline__ int *group_pairs(int *g, int T, int k) { return g + 4 + 3 * (T * k + 1); }

__global__ __launch_bounds__(kBlock) void group_pairs_kernel(const int32_t *__restrict__ ids, int T,
                                                             int k, int E,
                                                             const int32_t *__restrict__ slot_of,
                                                             int has_shared, int *groups, int *err) {
    __shared__ int e_eff[kBlock], s_eff[kBlock], first[kBlock];
    const int P = T * k;  // <= 256
    const int tid = threadIdx.x;
    int e = -1, s = -1;
    if (tid < P) {
        e = ids[tid];
        if (e < 0 || e >= E) {
            atomicOr(err, kErrRange);
            e = -1;
        } else {
            s = slot_of ? slot_of[e] : e;
            if (s < 0) {
                atomicOr(err, kErrNotResident);
                e = -1;
            }
        }
    }
    e_eff[tid] = e;
    s_eff[tid] = s;
    __syncthreads();
    int is_first = 0, rank = 0;
    if (e >= 0) {
        is_first = 1;
        for (int q = 0; q < P; ++q) {
            const int eq = e_eff[q];
            if (eq < 0) continue;
            if (eq == e && q < tid) is_first = 0;
            if (eq < e || (eq == e && q < tid)) ++rank;
        }
    }
    first[tid] = is_first;
    __syncthreads();
    int *gs = group_slot(groups, T, k), *gst = group_start(groups, T, k), *gc = group_count(groups, T, k);
    int *gp = group_pairs(groups, T, k);
    if (e >= 0) {
        gp[rank] = tid;
        if (is_first) {
            int gidx = 0, cnt = 0;
            for (int q = 0; q < P; ++q) {
                if (first[q] && e_eff[q] < e) ++gidx;
                if (e_eff[q] == e) ++cnt;
            }
            gs[gidx] = s;
            gst[gidx] = rank;
            gc[gidx] = cnt;
        }
    }
    if (tid == 0) {
        int ng = 0, nv = 0;
        for (int q = 0; q < P; ++q) {
            ng += first[q];
            nv += e_eff[q] >= 0;
        }
        int total = ng;
        if (has_shared) {
            gs[ng] = -2;
            gst[ng] = nv;
            gc[ng] = T;
            for (int t = 0; t < T; ++t) gp[nv + t] = P + t;
            total = ng + 1;
        }
        groups[0] = total;
        groups[1] = ng;
        groups[2] = nv;
    }
}

// A missing expert streamed by a gate/up launch: kFillGuBlocks blocks stream its rows (128 waves, each
// with a row pair in flight per pass: 1 MiB for bf16 rows of 2048, 256 KiB for int4) and kFillSlices
// blocks copy its down part.  Swept on both benchmark shapes (8-48 blocks, 16-64 pieces): 32 and 32 were
// the fastest or within noise of it on each.
constexpr int kFillGuBlocks = 32;
constexpr int kFillSlices = 32;

// 16-byte store with the nontemporal hint (a filled slot is not read again by this launch).
__device__ __forceinline__ void store16_stream(uint8_t *p, uint4 v) {
    const u32x4 t = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(t, reinterpret_cast<u32x4 *>(p));
}

// Copies the down part of every blob in the fill list from the host store to its slot: fl.slices pieces
// per blob, one block each, two 16-byte loads per thread in flight.
__device__ __forceinline__ void copy_down_parts(const FfnFill &fl, size_t expert_bytes) {
    const int nf = min(fl.n[0], MOE_MAX_TOPK);  // a one-token step fills at most k <= MOE_MAX_TOPK blobs
    const size_t n16 = (expert_bytes - size_t(fl.doff)) / 16;
    const size_t per = (n16 + size_t(fl.slices) - 1) / size_t(fl.slices);
    for (int it = blockIdx.x; it < nf * fl.slices; it += gridDim.x) {
        const int f = it / fl.slices, piece = it - f * fl.slices;
        const size_t beg = size_t(piece) * per;
        const size_t end = beg + per < n16 ? beg + per : n16;
        const uint4 *src = reinterpret_cast<const uint4 *>(fl.host + fl.src[f] + fl.doff);
        uint4 *dst = reinterpret_cast<uint4 *>(fl.pool + size_t(fl.slot[f]) * expert_bytes + size_t(fl.doff));
        for (size_t i = beg + threadIdx.x; i < end; i += size_t(2 * kBlock)) {
            const size_t j = i + kBlock;
            const uint4 a = src[i];
            const uint4 b = j < end ? src[j] : make_uint4(0u, 0u, 0u, 0u);
            dst[i] = a;
            if (j < end) dst[j] = b;
        }
    }
}

// -------------------------------------------------------------- gate/up ---
// act[p, i] = w_p * silu(W_g[i] . x_t) * (W_u[i] . x_t) for every pair p of one
// expert group.  One wave per row pair (gate row 2i, up row 2i+1): the pair's
// weights are loaded once into registers and applied to each token of the
// group.  ONE_TOKEN: T == 1, groups are the k ranks (+ shared), no table;
// with plan.fill it also performs the step's fills (FfnFill): a missing
// expert's rows come from the host store, plan.fill.blocks blocks stream them
// (each wave a row pair per pass) and store them into the slot, and one more
// row of blocks copies the blobs' down parts.
template <int DT, int NCH, bool ONE_TOKEN, bool FULL>
__global__ __launch_bounds__(kBlock) void gateup_kernel(
    const float *__restrict__ x, int T, int H, int I, int E, int k, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ slot_of, const uint8_t *__restrict__ pool, size_t expert_bytes,
    const uint8_t *__restrict__ shared_w, const float *__restrict__ weights, int *groups,
    float *__restrict__ act, int *err, FfnPlan plan) {
    constexpr int EPC = Fmt<DT>::EPC;
    // One token: the block stages x in LDS once instead of every wave reading it.  int4 (a wave streams
    // 2 KiB of weights but would read 8 KiB of x): as fp16 pairs with per-chunk scales (STAGE_X).  bf16:
    // as fp32, read chunk by chunk just before its products, which frees the registers that held the
    // wave's x (STAGE_XF; config 4's gate/up 10.5 -> 9.95 us).  f32 weights keep per-wave x.
    constexpr bool STAGE_X = ONE_TOKEN && DT == INT4;
    constexpr bool STAGE_XF = ONE_TOKEN && DT == BF16;
    constexpr int NXF = (NCH * kWave * EPC / 4 + kBlock - 1) / kBlock;  // float4 of x per thread (STAGE_XF)
    const int lane = threadIdx.x & (kWave - 1);
    const int g = blockIdx.y;
    const uint8_t *blob;
    uint8_t *dst = nullptr;  // a missing expert streamed in by this launch: its rows are stored here too
    int istride = 0;         // then the wave's row pairs lie this far apart (0: one row pair per wave)
    int pstart = 0, pcount = 1, single = 0;
    const int *pairs = nullptr;
    unsigned long long *clk = nullptr;  // a filling launch: its blocks stamp the fill clock
    unsigned long long t_fill = 0;      // when this block began filling
    int i = blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave);
    const int P = T * k;
    // One token whose slots the device lookup wrote: every load that the blob's address depends on (the
    // rank's slot, the fill count, the fill list across the wave's lanes) is issued at once, and the token's
    // x after them, so that one wait covers the chain and x stays in flight into the weight stream.
    int s_ld = 0, nf_ld = 0, fslot = -1;
    long long fsrc = 0;
    bool dev_slot = false;
    if constexpr (ONE_TOKEN) {
        clk = plan.fill.n ? plan.fill.clk : nullptr;
        if (plan.fill.n && g == int(gridDim.y) - 1) {
            const bool busy = int(blockIdx.x) < min(plan.fill.n[0], MOE_MAX_TOPK) * plan.fill.slices;
            const unsigned long long t0 = clk && busy ? devres::clk_now() : 0ull;
            copy_down_parts(plan.fill, expert_bytes);
            if (t0) devres::clk_record_fill(clk, t0, devres::clk_now());
            return;
        }
        single = g;  // pair index: rank g, or T*k + 0 = k for the shared expert
        dev_slot = g < k && !plan.n;
        if (dev_slot) {
            // (the block-uniform words go through vector loads: earlier kernels on the stream wrote them)
            if (plan.fill.n) {
                nf_ld = load_stream_word(plan.fill.n);
                if (lane < min(E, MOE_MAX_TOPK)) {  // (the fill list holds E entries)
                    fslot = plan.fill.slot[lane];
                    fsrc = plan.fill.src[lane];
                }
            }
            s_ld = load_stream_word((plan.rank_slot ? plan.rank_slot : ids) + g);
        }
    } else {
        if (g >= groups[0]) return;
    }
    if (!STAGE_X && !STAGE_XF && i >= I) return;  // when x is staged, every wave joins the block's staging below
    float xv[STAGE_X || STAGE_XF ? 1 : NCH][EPC];
    float4 xf[STAGE_XF ? NXF : 1];  // STAGE_XF: this thread's share of x, loaded before the weight stream
    uint4 xq[STAGE_X ? NCH : 1][4];       // staged int4 path: the chunk's activations as fp16 pairs
    float xbias[NCH];                     // ... the chunk's bias term
    int xsh_[NCH];                        // ... and its exponent shift
    float wp0 = 1.f;  // combine weight of the first pair (1 for the shared expert)
    if constexpr (!ONE_TOKEN) {
        pstart = group_start(groups, T, k)[g];
        pairs = group_pairs(groups, T, k);
    }
    if constexpr (STAGE_XF) {
        const float4 *xt4 = reinterpret_cast<const float4 *>(x);  // (one token)
        wp0 = single < P ? weights[single] : 1.f;
#pragma unroll
        for (int r = 0; r < NXF; ++r) xf[r] = load_f4(xt4 + min(r * kBlock + int(threadIdx.x), H / 4 - 1));
    }
    if constexpr (!STAGE_X && !STAGE_XF) {
        // The first pair's activations are loaded before the weight stream: loads
        // retire in issue order, so waiting for x never waits for the weights.
        const int p0 = ONE_TOKEN ? single : pairs[pstart];
        wp0 = p0 < P ? weights[p0] : 1.f;
        const float *xt = x + size_t(p0 < P ? p0 / k : p0 - P) * H;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int col0 = (c * kWave + lane) * EPC;
            if ((FULL || col0 < H)) {
                load_x<DT>(xt, col0, xv[c]);
            } else {
#pragma unroll
                for (int q = 0; q < EPC; ++q) xv[c][q] = 0.f;
            }
        }
    }
    // Staged int4 token: this thread's share of x (eight elements per round) is loaded before the weight
    // stream, so that packing it waits only for these loads.
    float4 xa[STAGE_X ? NCH : 1][2];
    if constexpr (STAGE_X) {
        const float4 *xt4 = reinterpret_cast<const float4 *>(x + size_t(single < P ? single / k : single - P) * H);
#pragma unroll
        for (int r = 0; r < NCH; ++r) {
            const int f = r * kBlock + threadIdx.x;
            const bool in = FULL || (f >> 2) * EPC < H;  // (H is a multiple of 128: a chunk is in or out whole)
            xa[r][0] = in ? xt4[2 * f] : make_float4(0.f, 0.f, 0.f, 0.f);
            xa[r][1] = in ? xt4[2 * f + 1] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
    if constexpr (ONE_TOKEN) {
        // (the loaded values pass through an empty asm after the x loads, so that no use of them -- and no
        // wait for them -- is scheduled before x is in flight)
        if (dev_slot) asm volatile("" : "+v"(s_ld), "+v"(nf_ld), "+v"(fslot), "+v"(fsrc)::"memory");
        if (g < k && plan.n) {
            // slots known on the host: no device lookups.  Selected with the block-uniform rank so that
            // the offsets stay argument (scalar) loads rather than one indexed load before the weights.
            long long off = plan.off[0];
#pragma unroll
            for (int j = 1; j < MOE_MAX_TOPK; ++j)
                if (g == j) off = plan.off[j];
            if (off < 0) return;  // a rank the host tier computes
            blob = pool + off;
        } else if (dev_slot) {
            int s;
            if (plan.rank_slot) {  // the device lookup's slot for this rank (it flagged bad ids itself)
                s = s_ld;
            } else {
                const int e = s_ld;
                if (e < 0 || e >= E) {
                    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(err, kErrRange);
                    return;
                }
                s = slot_of ? slot_of[e] : e;
                asm volatile("" : "+v"(s));  // (the wait for this dependent load stays on this path)
            }
            if (s < 0) {
                if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(err, kErrNotResident);
                return;
            }
            blob = pool + size_t(s) * expert_bytes;
            if (plan.fill.n) {
                // the lanes holding a fill of this slot (at most one: a step fills a slot once)
                const unsigned long long m = __ballot(lane < min(nf_ld, MOE_MAX_TOPK) && fslot == s);
                if (m) {
                    const int f = __ffsll((long long)m) - 1;
                    const unsigned lo = __builtin_amdgcn_readlane(unsigned(fsrc), f);
                    const unsigned hi = __builtin_amdgcn_readlane(unsigned((unsigned long long)fsrc >> 32), f);
                    dst = plan.fill.pool + size_t(s) * expert_bytes;
                    blob = plan.fill.host + (long long)(((unsigned long long)hi << 32) | lo);
                    if (int(blockIdx.x) >= plan.fill.blocks) return;
                    istride = plan.fill.blocks * (kBlock / kWave);
                    if (clk) t_fill = devres::clk_now();
                }
            }
        } else {
            blob = shared_w;
        }
    } else {
        const int s = group_slot(groups, T, k)[g];
        pcount = group_count(groups, T, k)[g];
        blob = s == -2 ? shared_w : pool + size_t(s) * expert_bytes;
    }
    const size_t rb = row_bytes_of(DT, H);
    for (bool first = true;; first = false) {
    const int iw = i < I ? i : I - 1;  // staging x: a wave past I loads a valid row and stores nothing
    const uint8_t *gate = blob + size_t(2 * iw) * rb + row_bytes_of(DT, lane * EPC);  // this lane's first chunk
    const uint8_t *up = gate + rb;
    uint4 wg[NCH], wu[NCH];
    float sg[NCH], su[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int col0 = (c * kWave + lane) * EPC;
        const bool in = (FULL || col0 < H);
        wg[c] = in ? load16_stream(gate + size_t(c) * 16 * kWave) : make_uint4(0, 0, 0, 0);
        wu[c] = in ? load16_stream(up + size_t(c) * 16 * kWave) : make_uint4(0, 0, 0, 0);
        if constexpr (DT == INT4) {
            const uint16_t *sc = reinterpret_cast<const uint16_t *>(blob + size_t(I) * H);
            const int groups_per_row = H / 128;
            sg[c] = in ? bf16_bits_to_float(sc[size_t(2 * iw) * groups_per_row + col0 / 128]) : 0.f;
            su[c] = in ? bf16_bits_to_float(sc[size_t(2 * iw + 1) * groups_per_row + col0 / 128]) : 0.f;
        }
    }
    if constexpr (STAGE_XF) {
      if (first) {  // x into LDS while the weight loads are in flight
        extern __shared__ float4 xsf[];
#pragma unroll
        for (int r = 0; r < NXF; ++r)
            if (r * kBlock + int(threadIdx.x) < H / 4) xsf[r * kBlock + threadIdx.x] = xf[r];
        __syncthreads();
        if (i >= I) return;
      }
    }
    if constexpr (STAGE_X) {
      if (first) {
        // The token row is the same for every wave of the block: it is staged in LDS once, while the
        // weight loads are in flight, as fp16 pairs (stage8_i4h: thread f packs the eight elements of
        // dword f % 4 of chunk slot f / 4), transposed to [chunk][dword][lane] so that each read of a
        // dword's word is 64 consecutive 16-byte words; each chunk slot's exponent shift and bias term
        // follow.
        extern __shared__ uint4 xsh[];
        int2 *xaux = reinterpret_cast<int2 *>(xsh + NCH * 4 * kWave);
        wp0 = single < P ? weights[single] : 1.f;
        // x passes through an empty asm after the weight loads: otherwise the compiler hoists the staging's
        // first steps above the loop, and their wait for x holds the weight loads back
#pragma unroll
        for (int r = 0; r < NCH; ++r)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                float &a = xa[r][h].x, &b = xa[r][h].y, &c = xa[r][h].z, &d = xa[r][h].w;
                asm volatile("" : "+v"(a), "+v"(b), "+v"(c), "+v"(d)::"memory");
            }
#pragma unroll
        for (int r = 0; r < NCH; ++r) {  // NCH * 64 chunk slots x 4 dwords = NCH rounds of the block
            const int f = r * kBlock + threadIdx.x, gs = f >> 2, q = f & 3;
            float v[8];
            const float4 a = xa[r][0], b = xa[r][1];
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
            int sh;
            float bias;
            const uint4 w = stage8_i4h(v, sh, bias);
            xsh[((gs / kWave) * 4 + q) * kWave + (gs % kWave)] = w;
            if (q == 0) xaux[gs] = make_int2(__float_as_int(bias), sh);
        }
        __syncthreads();
        if (i >= I) return;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
#pragma unroll
            for (int q = 0; q < 4; ++q) xq[c][q] = xsh[(c * 4 + q) * kWave + lane];
            const int2 au = xaux[c * kWave + lane];
            xbias[c] = __int_as_float(au.x);
            xsh_[c] = -au.y;
        }
      }
    }
    if (dst && i < I) {  // the missing expert's row pair (and int4 scales) into its slot
        uint8_t *dg = dst + (gate - blob);  // the same place in the slot
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int col0 = (c * kWave + lane) * EPC;
            if ((FULL || col0 < H)) {
                store16_stream(dg + size_t(c) * 16 * kWave, wg[c]);
                store16_stream(dg + rb + size_t(c) * 16 * kWave, wu[c]);
                if constexpr (DT == INT4) {
                    if (col0 % 128 == 0) {  // one lane per quantisation group; bf16 -> float -> bf16 is exact
                        uint16_t *sc = reinterpret_cast<uint16_t *>(dst + size_t(I) * H);
                        const int groups_per_row = H / 128;
                        sc[size_t(2 * iw) * groups_per_row + col0 / 128] = uint16_t(__float_as_uint(sg[c]) >> 16);
                        sc[size_t(2 * iw + 1) * groups_per_row + col0 / 128] = uint16_t(__float_as_uint(su[c]) >> 16);
                    }
                }
            }
        }
    }
    for (int q = 0; q < pcount; ++q) {
        const int p = ONE_TOKEN ? single : pairs[pstart + q];
        if (!STAGE_X && !STAGE_XF && q > 0) {  // (a staged token is one pair)
            const float *xt = x + size_t(p < P ? p / k : p - P) * H;
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                const int col0 = (c * kWave + lane) * EPC;
                if ((FULL || col0 < H)) load_x<DT>(xt, col0, xv[STAGE_X || STAGE_XF ? 0 : c]);
            }
        }
        float ga = 0.f, ua = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            if constexpr (STAGE_X) {
                ga += ldexpf((chunk_dot_i4h(wg[c], xq[c]) - xbias[c]) * sg[c], xsh_[c]);
                ua += ldexpf((chunk_dot_i4h(wu[c], xq[c]) - xbias[c]) * su[c], xsh_[c]);
            } else {
                float xl[EPC];  // this chunk's x: from LDS (STAGE_XF) or the wave's registers
                if constexpr (STAGE_XF) {
                    extern __shared__ float4 xsf[];
                    const int col0 = (c * kWave + lane) * EPC;
#pragma unroll
                    for (int h = 0; h < EPC / 4; ++h) {
                        const float4 v = (FULL || col0 < H) ? xsf[col0 / 4 + h] : make_float4(0.f, 0.f, 0.f, 0.f);
                        xl[4 * h] = v.x;
                        xl[4 * h + 1] = v.y;
                        xl[4 * h + 2] = v.z;
                        xl[4 * h + 3] = v.w;
                    }
                } else {
#pragma unroll
                    for (int h = 0; h < EPC; ++h) xl[h] = xv[STAGE_XF ? 0 : c][h];
                }
                float dg = chunk_dot<DT>(wg[c], xl), du = chunk_dot<DT>(wu[c], xl);
                if constexpr (DT == INT4) {
                    dg *= sg[c];
                    du *= su[c];
                }
                ga += dg;
                ua += du;
            }
        }
        ga = wave_sum(ga);
        ua = wave_sum(ua);
        // the pair's combine weight is folded in here
        const float wp = q == 0 ? wp0 : (p < P ? weights[p] : 1.f);
        if (lane == 0) act[size_t(p) * I + i] = wp * (ga * __builtin_amdgcn_rcpf(1.f + __expf(-ga)) * ua);
    }
    if (!istride) break;  // block-uniform; no barrier follows the first pass
    i += istride;
    if (i >= I) break;
    }
    if (clk) {  // (wave 0 of the block records: waves past I returned early only when not staging x)
        if (t_fill) devres::clk_record_fill(clk, t_fill, devres::clk_now());
        else devres::clk_record_compute(clk, devres::clk_now());
    }
}

// ------------------------------------------------------ down + combine ---
// y[t, h] (+)= sum_j W_d^{e_tj}[h, :] . act[t*k + j] + W_d^shared[h, :] . act[T*k + t], where the
// gate/up kernel has already scaled act[t*k + j] by the combine weight w[t, j].
// One block per (row tile, token); the token's k (+1) down rows for output h
// form one virtual row of (k+1) * I elements that the wave streams in 16-byte
// chunks; the combine weight is folded into the activations held in registers,
// which every output row of the wave reuses.
template <int DT>
__global__ __launch_bounds__(kBlock) void down_combine_kernel(
    int T, int H, int I, int E, int k, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ slot_of, const uint8_t *__restrict__ pool, size_t expert_bytes,
    const uint8_t *__restrict__ shared_w, size_t d_off, const float *__restrict__ act,
    float *__restrict__ y, int accumulate) {
    constexpr int EPC = Fmt<DT>::EPC;
    // entry j: slot (-2 shared expert, -1 skipped) and activation row
    __shared__ int ent_slot[MOE_MAX_TOPK + 1];
    __shared__ int ent_p[MOE_MAX_TOPK + 1];
    const int t = blockIdx.y;
    const int NE = k + (shared_w != nullptr);
    if (threadIdx.x < NE) {
        const int j = threadIdx.x;
        int sl = -1, p;
        if (j < k) {
            p = t * k + j;
            const int e = ids[p];
            if (e >= 0 && e < E) {
                sl = slot_of ? slot_of[e] : e;
                if (sl < 0) sl = -1;
            }
        } else {
            p = T * k + t;
            sl = -2;
        }
        ent_slot[j] = sl;
        ent_p[j] = p;
    }
    __syncthreads();
    const int lane = threadIdx.x & (kWave - 1);
    const int h0 = (blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave)) * kDownRows;
    if (h0 >= H) return;
    const size_t rb = row_bytes_of(DT, I);
    const int cpr = int(rb / 16);  // chunks per expert row
    const int total = NE * cpr;
    const size_t d_sc = d_off + size_t(H) * I / 2;  // int4 scales of W_d
    const int groups_per_row = I / 128;
    float acc[kDownRows];
#pragma unroll
    for (int r = 0; r < kDownRows; ++r) acc[r] = 0.f;
    for (int base = 0; base < total; base += kWave * kDownSlots) {
        float av[kDownSlots][EPC];
        const uint8_t *rp[kDownSlots];
        const uint16_t *sp[kDownSlots];
        bool ok[kDownSlots];
#pragma unroll
        for (int s = 0; s < kDownSlots; ++s) {
            const int gch = base + s * kWave + lane;
            ok[s] = false;
            rp[s] = pool;  // (a global pointer, so the loads below stay global loads)
            sp[s] = reinterpret_cast<const uint16_t *>(pool);
            if (gch < total) {
                const int j = gch / cpr, c = gch - j * cpr;
                const int sl = ent_slot[j];
                if (sl != -1) {
                    const uint8_t *blob = sl == -2 ? shared_w : pool + size_t(sl) * expert_bytes;
                    ok[s] = true;
                    rp[s] = blob + d_off + size_t(c) * 16;
                    if constexpr (DT == INT4)
                        sp[s] = reinterpret_cast<const uint16_t *>(blob + d_sc) + (c * EPC) / 128;
                    load_x<DT>(act + size_t(ent_p[j]) * I, c * EPC, av[s]);
                }
            }
        }
        uint4 wv[kDownRows][kDownSlots];
#pragma unroll
        for (int r = 0; r < kDownRows; ++r)
#pragma unroll
            for (int s = 0; s < kDownSlots; ++s)
                wv[r][s] = (ok[s] && h0 + r < H) ? load16_stream(rp[s] + size_t(h0 + r) * rb) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int r = 0; r < kDownRows; ++r)
#pragma unroll
            for (int s = 0; s < kDownSlots; ++s)
                if (ok[s] && h0 + r < H) {
                    float d = chunk_dot<DT>(wv[r][s], av[s]);
                    if constexpr (DT == INT4) d *= bf16_bits_to_float(sp[s][size_t(h0 + r) * groups_per_row]);
                    acc[r] += d;
                }
    }
#pragma unroll
    for (int r = 0; r < kDownRows; ++r) {
        const float v = wave_sum(acc[r]);
        const int h = h0 + r;
        if (lane == 0 && h < H) {
            float *o = y + size_t(t) * H + h;
            *o = accumulate ? *o + v : v;
        }
    }
}

// The same down + combine with every chunk of a wave's output row issued at
// once (NS 16-byte chunks per lane, NS * 64 >= (k+1) * I / elements-per-chunk).
// The token's activations (combine weights already folded in by the gate/up
// kernel) are contiguous rows t*k .. t*k+k-1 plus the shared row T*k + t: each
// thread issues its staging loads first, then the weight loads go out back to
// back without branches (an invalid chunk loads from the pool base and is
// masked), and only then are the staged values written to LDS.
// R output rows per wave, BT / 64 waves per block, one block per (row tile, token).
template <int DT, int NS, int R, int BT>
__global__ __launch_bounds__(BT) void down_combine_lds_kernel(
    int T, int H, int I, int E, int k, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ slot_of, const uint8_t *__restrict__ pool, size_t expert_bytes,
    const uint8_t *__restrict__ shared_w, size_t d_off, const float *__restrict__ act,
    float *__restrict__ y, int accumulate, FfnPlan plan) {
    constexpr int EPC = Fmt<DT>::EPC;
    // int4 weights: the activations are staged as fp16 pairs (stage8_i4h), [4][chunks] words then an
    // (exponent shift, bias term) pair per chunk; thread f of staging round m = f / BT packs dword f % 4
    // of chunk f / 4, RH rounds covering the NS * 64 chunk slots.  Otherwise as fp32, [(k+1) x I / 4]
    // float4, SM float4 per thread: (k+1) I <= NS * 64 * EPC <= SM * 4 * BT.
    constexpr bool HALF = DT == INT4;
    constexpr int RH = (NS * 256 + BT - 1) / BT;
    constexpr int SM = HALF ? 2 * RH : (NS * EPC * kWave + 4 * BT - 1) / (4 * BT);
    extern __shared__ float4 aw4[];
    const int t = blockIdx.y;
    const int NE = k + (shared_w != nullptr);
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    // 1. where the entries live, resolved by every wave for itself (lane j < NE: entry j) into its own LDS
    // table, so that no block barrier stands before the weight loads.  Entry j: byte offset of its blob from
    // `pool` (the shared expert's too, so that every address derives from a kernel argument and stays a global
    // load), or kAbsent when it contributes nothing.  Its loads go out before the staging loads, whose wait they
    // then skip.  (Vector loads: the ids and the slot table are written by earlier kernels on the stream.)
    __shared__ long long ent_tab[BT / kWave][MOE_MAX_TOPK + 1];
    // Each lane loads the entry of rank min(lane, k - 1) before anything else: with host-known slots its byte
    // offset among the kernel arguments, otherwise its slot (device lookup) or expert id from one uniformly
    // chosen array.
    const int jl = min(lane, k - 1);
    long long o_ld = -1;  // with host-known slots: the rank's byte offset (-1: a rank the host tier computes)
    int v_ld = -1;        // otherwise: the rank's slot or expert id
    if (plan.n)
        o_ld = plan.off[jl];
    else
        v_ld = (plan.rank_slot ? plan.rank_slot : ids + size_t(t) * k)[jl];
    // 2. staging loads, unconditional (an index past the activations reads the token's first ones, which are
    // never written to LDS: the chunks there lie past `total`), so that the wait for the entries below can
    // count them as still in flight.  (No select on the loaded value: it would turn each load into a branch.)
    const int n4 = NE * I / 4, routed4 = k * I / 4;
    const float4 *src_routed = reinterpret_cast<const float4 *>(act) + size_t(t) * routed4;
    const float4 *src_shared = reinterpret_cast<const float4 *>(act) + (size_t(T) * k + t) * (I / 4) - routed4;
    float4 stage[SM];
    if constexpr (HALF) {
#pragma unroll
        for (int m = 0; m < RH; ++m) {
            const int i = 2 * (threadIdx.x + m * BT);  // (routed4 is even: a pair lies on one side)
            const float4 *sp = i < n4 ? (i < routed4 ? src_routed : src_shared) + i : src_routed;
            stage[2 * m] = load_f4(sp);
            stage[2 * m + 1] = load_f4(sp + 1);
        }
    } else {
#pragma unroll
        for (int m = 0; m < SM; ++m) {
            const int i = threadIdx.x + m * BT;
            stage[m] = load_f4(i < n4 ? (i < routed4 ? src_routed : src_shared) + i : src_routed);
        }
    }
    // (the entries' values pass through an empty asm after the staging loads: no use of them, and no wait
    // for them, is scheduled before those are in flight)
    asm volatile("" : "+v"(o_ld), "+v"(v_ld)::"memory");
    constexpr long long kAbsent = -0x7fffffffffffffffLL - 1;  // (the shared expert's offset may be negative)
    if (lane < NE) {
        long long off = kAbsent;
        if (lane < k) {
            if (plan.n) {
                if (o_ld >= 0) off = o_ld;
            } else {
                int sl = v_ld;
                if (!plan.rank_slot) {  // an expert id: checked, then its slot (a dependent load, on this path only,
                    // waited for inside it so that the common path below does not wait for the staging loads)
                    sl = (sl >= 0 && sl < E) ? (slot_of ? slot_of[sl] : sl) : -1;
                    asm volatile("" : "+v"(sl));
                }
                if (sl >= 0) off = (long long)sl * (long long)expert_bytes;
            }
        } else {
            off = (long long)(shared_w - pool);
        }
        ent_tab[wid][lane] = off;
    }
    wave_lds_sync();
    // 3. weight loads of this wave's R output rows.  Workgroup b runs on XCD b mod 8: consecutive row tiles
    // go to the same XCD, so the blocks that share a cache line of int4 row scales share one L2.
    const int nb = gridDim.x;
    const int tile = (nb & 7) ? int(blockIdx.x) : int(blockIdx.x & 7) * (nb >> 3) + int(blockIdx.x >> 3);
    const int h0 = (tile * (BT / kWave) + (threadIdx.x / kWave)) * R;  // the wave's first row
    const size_t rb = row_bytes_of(DT, I);
    const unsigned cpr = unsigned(rb / 16);  // chunks per expert row
    const unsigned total = unsigned(NE) * cpr;
    uint4 wv[R][NS];
    float sv[R][NS];
    bool ok[NS];
    unsigned j = unsigned(lane) / cpr, c = unsigned(lane) - j * cpr;  // chunk lane + 64 s = entry j, column chunk c
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const bool in = unsigned(s * kWave + lane) < total;
        const long long o = ent_tab[wid][in ? j : 0u];
        ok[s] = in && o != kAbsent;
        const uint8_t *blob = pool + (ok[s] ? o : 0);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int h = min(h0 + r, H - 1);
            const size_t row_off = d_off + size_t(h) * rb;
            wv[r][s] = load16_stream(ok[s] ? blob + row_off + size_t(c) * 16 : pool);
            if constexpr (DT == INT4) {
                const size_t sc_off = d_off + size_t(H) * rb + size_t(h) * (I / 128) * 2;  // this row's scales
                sv[r][s] = bf16_bits_to_float(*reinterpret_cast<const uint16_t *>(
                    ok[s] ? blob + sc_off + size_t(c * EPC / 128) * 2 : pool));
            }
        }
        c += kWave;
        while (c >= cpr) {
            c -= cpr;
            ++j;
        }
    }
    // 4. staged activations to LDS; chunk g of the virtual row covers elements [g * EPC, +EPC)
    uint4 *xs = reinterpret_cast<uint4 *>(aw4);
    int2 *xaux = reinterpret_cast<int2 *>(xs + 4 * total);
    if constexpr (HALF) {
#pragma unroll
        for (int m = 0; m < RH; ++m) {
            const unsigned f = threadIdx.x + m * BT, g = f >> 2, q = f & 3u;
            const float v[8] = {stage[2 * m].x, stage[2 * m].y, stage[2 * m].z, stage[2 * m].w,
                                stage[2 * m + 1].x, stage[2 * m + 1].y, stage[2 * m + 1].z, stage[2 * m + 1].w};
            int sh;
            float bias;
            const uint4 w = stage8_i4h(v, sh, bias);  // (every lane: quad exchanges)
            if (g < total) {
                xs[q * total + g] = w;
                if (q == 0) xaux[g] = make_int2(__float_as_int(bias), sh);
            }
        }
    } else {
#pragma unroll
        for (int m = 0; m < SM; ++m) {
            const int i = threadIdx.x + m * BT;
            if (i < n4) aw4[i] = stage[m];
        }
    }
    __syncthreads();
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (HALF && ok[s]) {
            const unsigned g = s * kWave + lane;
            uint4 xq[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) xq[q] = xs[q * total + g];
            const int2 au = xaux[g];
#pragma unroll
            for (int r = 0; r < R; ++r)
                acc[r] += ldexpf((chunk_dot_i4h(wv[r][s], xq) - __int_as_float(au.x)) * sv[r][s], -au.y);
        } else if (!HALF && ok[s]) {
            const int g = s * kWave + lane;
            float av[EPC];
#pragma unroll
            for (int q = 0; q < EPC / 4; ++q) {
                const float4 a4 = aw4[g * (EPC / 4) + q];
                av[4 * q] = a4.x;
                av[4 * q + 1] = a4.y;
                av[4 * q + 2] = a4.z;
                av[4 * q + 3] = a4.w;
            }
#pragma unroll
            for (int r = 0; r < R; ++r) {
                float d = chunk_dot<DT>(wv[r][s], av);
                if constexpr (DT == INT4) d *= sv[r][s];
                acc[r] += d;
            }
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float v = wave_sum(acc[r]);
        const int hrow = h0 + r;
        if (lane == 0 && hrow < H) {
            float *o = y + size_t(t) * H + hrow;
            *o = accumulate ? *o + v : v;
        }
    }
}

// -------------------------------------------------------------- combine ---
__global__ __launch_bounds__(kBlock) void combine_kernel(const float *__restrict__ yp,
                                                         const float *__restrict__ w,
                                                         const float *__restrict__ ys, int T, int k,
                                                         int H, float *__restrict__ y, int accumulate) {
    const size_t idx = size_t(blockIdx.x) * kBlock + threadIdx.x;
    if (idx >= size_t(T) * H) return;
    const int t = int(idx / H), h = int(idx - size_t(t) * H);
    float acc = 0.f;
    for (int j = 0; j < k; ++j) acc += w[size_t(t) * k + j] * yp[(size_t(t) * k + j) * H + h];
    if (ys) acc += ys[idx];
    y[idx] = accumulate ? y[idx] + acc : acc;
}

// ------------------------------------------------------------ slot table ---
// Expert fills as one kernel: each block streams a share of one expert blob
// from pinned host memory (read over PCIe) into its HBM slot; block (0, 0) also
// writes the slot-table changes of the batch.  Later kernels on the stream see
// both.  Each thread keeps kFillUnroll 16-byte loads of host memory
// outstanding; with 32 blocks per 9 MiB blob that is 256 KiB in flight per
// fill, which measured faster than 1 or 2 MiB (the device-decision fill kernel
// has the same shape).
constexpr int kFillUnroll = 2;
constexpr int kHostFillsInFlight = 4;  // fills streamed at once
__global__ __launch_bounds__(kBlock) void fill_slots_kernel(FillBatch b) {
    if (blockIdx.y == 0 && blockIdx.x == 0)
        for (int i = threadIdx.x; i < b.n_tab; i += kBlock) b.table[b.tab_idx[i]] = b.tab_val[i];
    const size_t n16 = size_t(b.bytes) / 16;
    const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const size_t beg = size_t(blockIdx.x) * per;
    const size_t end = beg + per < n16 ? beg + per : n16;
    // A bounded grid walks the batch: a few fills saturate the link, and the rest of the chip stays free
    // for the compute a prefetch overlaps.
    for (int f = blockIdx.y; f < b.n; f += gridDim.y) {
        const uint4 *src = reinterpret_cast<const uint4 *>(b.src[f]);
        uint4 *dst = reinterpret_cast<uint4 *>(b.dst[f]);
        for (size_t i = beg + threadIdx.x; i < end; i += size_t(kBlock) * kFillUnroll) {
            uint4 v[kFillUnroll];
#pragma unroll
            for (int u = 0; u < kFillUnroll; ++u) {
                const size_t j = i + size_t(u) * kBlock;
                v[u] = j < end ? src[j] : make_uint4(0u, 0u, 0u, 0u);
            }
#pragma unroll
            for (int u = 0; u < kFillUnroll; ++u) {
                const size_t j = i + size_t(u) * kBlock;
                if (j < end) dst[j] = v[u];
            }
        }
    }
}

constexpr int kSlotBatch = 32;
struct SlotUpdates {
    int n;
    int32_t index[kSlotBatch];
    int32_t value[kSlotBatch];
};

__global__ void slot_update_kernel(int32_t *table, SlotUpdates u) {
    const int i = threadIdx.x;
    if (i < u.n) table[u.index[i]] = u.value[i];
}

// ------------------------------------------------------- kernel tables ---
template <int NCH>
constexpr int nch_index() { return NCH == 1 ? 0 : NCH == 2 ? 1 : NCH == 4 ? 2 : 3; }

int elems_per_chunk(int dtype) { return dtype == F32 ? 4 : dtype == BF16 ? 8 : 32; }

int chunks_per_row(int H, int dtype) {
    const int epc = elems_per_chunk(dtype);
    const int need = (H + kWave * epc - 1) / (kWave * epc);
    for (int n : {1, 2, 4, 8})
        if (need <= n) return n;
    return -1;
}

// Launch with each argument converted to the kernel's parameter type.
template <typename... Params, typename... Args>
hipError_t launch(void (*kernel)(Params...), dim3 grid, dim3 block, size_t shmem, hipStream_t s, Args... args) {
    kernel<<<grid, block, shmem, s>>>(static_cast<Params>(args)...);
    return hipGetLastError();
}

}  // namespace

// ---------------------------------------------- allocation-free workspace ---
// The expert FFN's workspace for callers that cannot allocate (moe_expert_ffn_grouped_noalloc): one fixed
// array per device, held until the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory: its device address is looked up once per device (noalloc_scratch_setup) and only that
// address is ever handed to kernels.
__device__ __align__(256) unsigned char scratch[MOE_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kScratchDevices = 64;
void *g_scratch[kScratchDevices] = {};
}  // namespace

// ===================================================================== host

int noalloc_scratch_setup() {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail_hip(e, "scratch: hipGetDevice");
    if (dev < 0 || dev >= kScratchDevices) return fail(MOE_ERR_INVALID_ARG, "scratch: device %d out of range", dev);
    if (g_scratch[dev]) return MOE_OK;
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) return fail_hip(e, "scratch: hipGetSymbolAddress");
    g_scratch[dev] = ptr;
    return MOE_OK;
}

void *noalloc_scratch() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return nullptr;
    return g_scratch[dev];
}

size_t expert_blob_bytes(int H, int I, int dtype) {
    if (dtype == INT4) return size_t(3) * H * I / 2 + size_t(3) * H * I / 128 * 2;
    return size_t(3) * H * I * (dtype == F32 ? 4 : 2);
}

size_t down_offset(int H, int I, int dtype) {
    if (dtype == INT4) return size_t(I) * H + size_t(2) * I * (H / 128) * 2;
    return size_t(2) * I * H * (dtype == F32 ? 4 : 2);
}

static size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

size_t ffn_workspace_bytes(int T, int k, int I) {
    const size_t act = align256(sizeof(float) * size_t(T * k + T) * I);
    const size_t grp = align256(sizeof(int) * size_t(4 + 3 * (T * k + 1) + T * k + T));
    return act + grp;
}

FfnWorkspace ffn_workspace(void *base, int T, int k, int I) {
    FfnWorkspace w;
    w.act = static_cast<float *>(base);
    w.groups = reinterpret_cast<int *>(static_cast<char *>(base) +
                                       align256(sizeof(float) * size_t(T * k + T) * I));
    return w;
}

bool ffn_shape_supported(int H, int I, int dtype) {
    if (H <= 0 || I <= 0 || H % 128 || I % 128) return false;
    if (dtype != F32 && dtype != BF16 && dtype != INT4) return false;
    return chunks_per_row(H, dtype) > 0;
}

bool router_shape_supported(int H, int dtype) {
    if (H <= 0 || H % 128) return false;
    if (dtype != F32 && dtype != BF16) return false;
    return chunks_per_row(H, dtype) > 0;
}

hipError_t launch_router_logits(const float *x, const void *w, int w_dtype, int T, int H, int E,
                                const float *bias, float *logits, bool norm, float *h_out, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (!x) {
        if (bias == logits) return hipSuccess;
        return hipMemcpyAsync(logits, bias, sizeof(float) * size_t(T) * E, hipMemcpyDeviceToDevice, s);
    }
    if (w_dtype == BF16 && T >= kRouterMfmaMinTokens && (!norm || h_out)) {
        // many tokens: (pre-norm, then) the router product on the matrix cores
        const float *src = x;
        if (norm) {
            rmsnorm_rows_kernel<<<(T + 3) / 4, kBlock, 0, s>>>(x, T, H, h_out);
            const hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            src = h_out;
        }
        const dim3 g((E + kRouterTileE - 1) / kRouterTileE, (T + kRouterTileT - 1) / kRouterTileT);
        router_mfma_kernel<<<g, kRouterKWaves * kWave, 0, s>>>(src, static_cast<const uint16_t *>(w), T, H, E, bias,
                                                               logits);
        return hipGetLastError();
    }
    const dim3 grid((E + 3) / 4, T);
    const auto *wp = static_cast<const uint8_t *>(w);
    const int nch = chunks_per_row(H, w_dtype);
    float *hp = norm ? h_out : nullptr;
    // FULL: every lane's chunk slots lie inside the row (H = nch * 64 * elements per chunk), no bound checks
    const bool full = H == nch * kWave * elems_per_chunk(w_dtype);
#define ROUTER_LAUNCH(DT, N, F)                                                                     \
    (norm ? launch(router_logits_kernel<DT, N, true, F>, grid, kBlock, 0, s, x, wp, H, E, bias, logits, hp) \
          : launch(router_logits_kernel<DT, N, false, F>, grid, kBlock, 0, s, x, wp, H, E, bias, logits, hp))
#define ROUTER_CASE(DT, N)                                                                          \
    if (w_dtype == DT && nch == N) return full ? ROUTER_LAUNCH(DT, N, true) : ROUTER_LAUNCH(DT, N, false);
    ROUTER_CASE(F32, 1) ROUTER_CASE(F32, 2) ROUTER_CASE(F32, 4) ROUTER_CASE(F32, 8)
    ROUTER_CASE(BF16, 1) ROUTER_CASE(BF16, 2) ROUTER_CASE(BF16, 4) ROUTER_CASE(BF16, 8)
#undef ROUTER_CASE
#undef ROUTER_LAUNCH
    return hipErrorInvalidValue;
}

hipError_t launch_topk_lookup(const float *logits, int E, int k, int32_t *ids, float *weights, int *err_flags,
                              const DevResidency &r, const DevLookup &p, int32_t *slots_out, hipStream_t s) {
    if (p.C < 1 || p.C > kDevMaxSlots || p.E != E || E > MOE_MAX_EXPERTS || k < 1 || k > MOE_MAX_TOPK ||
        p.layer < 0 || p.layer >= p.L)
        return hipErrorInvalidValue;
    const bool small = devres::dev_threads(p.C) == 256;
#define TL_LAUNCH(RT, NTV) \
    topk_lookup_kernel<RT, NTV><<<1, NTV, 0, s>>>(logits, E, k, ids, weights, err_flags, r, p, slots_out)
    if (p.rotary && small) TL_LAUNCH(true, 256);
    else if (p.rotary) TL_LAUNCH(true, 1024);
    else if (small) TL_LAUNCH(false, 256);
    else TL_LAUNCH(false, 1024);
#undef TL_LAUNCH
    return hipGetLastError();
}

hipError_t launch_topk_softmax(const float *logits, int T, int E, int k, int32_t *ids, float *weights,
                               int *err_flags, hipStream_t s, IdsMailbox *pub, uint32_t seq, const float *h_src,
                               float *h_pub, int H) {
    if (T == 0) return hipSuccess;
    if (pub && T != 1) return hipErrorInvalidValue;
    if (h_pub && (!pub || !h_src || H % 4)) return hipErrorInvalidValue;
    topk_softmax_kernel<<<(T + 3) / 4, kBlock, 0, s>>>(logits, T, E, k, ids, weights, err_flags, pub, seq, h_src,
                                                       h_pub, H);
    return hipGetLastError();
}

namespace {
__global__ __launch_bounds__(kBlock) void add_kernel(float *__restrict__ x, const float *__restrict__ y, int n) {
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i < n) x[i] += y[i];
}
}  // namespace

hipError_t launch_add(float *x, const float *y, int n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    add_kernel<<<(n + kBlock - 1) / kBlock, kBlock, 0, s>>>(x, y, n);
    return hipGetLastError();
}

hipError_t launch_expert_ffn(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                             const float *weights, const int32_t *slot_of, const void *pool,
                             size_t expert_bytes, int dtype, const void *shared_w, float *y,
                             bool accumulate, const FfnWorkspace &ws, int *err_flags, hipStream_t s,
                             const FfnPlan *plan, int parts) {
    FfnPlan pl1;
    if (plan && T == 1) {
        if (plan->n == k) {
            pl1 = *plan;
            pl1.fill = FfnFill{};  // slots known on the host: nothing left to fill
        } else {
            pl1.fill = plan->fill;
            pl1.rank_slot = plan->rank_slot;
        }
    }
    if (pl1.fill.n) {  // fills performed by the gate/up launch
        const size_t doff = size_t(pl1.fill.doff);
        if (!slot_of || !(parts & kFfnGateUp) || doff != down_offset(H, I, dtype) || doff % 16 ||
            (expert_bytes - doff) % 16 || !pl1.fill.host || !pl1.fill.pool)
            return hipErrorInvalidValue;
        const int nbx = (I + 3) / 4;
        pl1.fill.blocks = kFillGuBlocks < nbx ? kFillGuBlocks : nbx;
        pl1.fill.slices = kFillSlices;
    }
    if (T == 0) return hipSuccess;
    const bool one = T == 1;
    const int has_shared = shared_w != nullptr;
    const auto *pl = static_cast<const uint8_t *>(pool);
    const auto *sw = static_cast<const uint8_t *>(shared_w);
    if (!one && (parts & kFfnGateUp)) {
        group_pairs_kernel<<<1, kBlock, 0, s>>>(ids, T, k, E, slot_of, has_shared, ws.groups, err_flags);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int groups = one ? k + has_shared : (T * k < E ? T * k : E) + has_shared;
    const dim3 ggrid((I + 3) / 4, groups + (pl1.fill.n ? 1 : 0));  // + the blocks copying down parts
    const int nch = chunks_per_row(H, dtype);
    // One-token int4 x staging covers every lane's chunk slot: [nch][4][64] words of fp16 pairs, then an
    // (exponent shift, bias term) pair per slot.
    // (bf16: the token's x as fp32)
    const size_t x_lds = dtype == INT4 ? size_t(nch) * kWave * (4 * 16 + 8) : dtype == BF16 ? size_t(H) * 4 : 0;
    // The down kernel: the LDS form when a token's k (+1) activation rows fit in LDS and NS chunks per lane
    // cover them, else the plain one.
    const size_t doff = down_offset(H, I, dtype);
    const int acc = accumulate ? 1 : 0;
    const int NE = k + has_shared;
    const int epc = elems_per_chunk(dtype);
    const int need = (NE * (I / epc) + kWave - 1) / kWave;
    // (int4: per chunk of 32 activations, four 16-byte words of fp16 pairs and an 8-byte shift and bias)
    const size_t lds = dtype == INT4 ? size_t(NE) * (I / 32) * 72 : sizeof(float) * size_t(NE) * I;
    int ns = 0;
    for (int n : {1, 2, 3, 4, 6, 8, 9, 12, 16})
        if (!ns && need <= n) ns = n;
    const bool lds_down = ns && lds <= 64 * 1024;
    bool launched = !(parts & kFfnGateUp);
    // FULL: every lane's chunk slots lie inside the row (H = nch * 64 * elements per chunk), no bound checks
    const bool full = H == nch * kWave * elems_per_chunk(dtype);
#define GU_LAUNCH(DT, N, F)                                                                         \
    (one ? launch(gateup_kernel<DT, N, true, F>, ggrid, kBlock, x_lds, s, x, T, H, I, E, k, ids,    \
                  slot_of, pl, expert_bytes, sw, weights, ws.groups, ws.act, err_flags, pl1)        \
         : launch(gateup_kernel<DT, N, false, F>, ggrid, kBlock, 0, s, x, T, H, I, E, k, ids,       \
                  slot_of, pl, expert_bytes, sw, weights, ws.groups, ws.act, err_flags, FfnPlan{}))
#define GU_CASE(DT, N)                                                                              \
    if (!launched && dtype == DT && nch == N) {                                                     \
        e = full ? GU_LAUNCH(DT, N, true) : GU_LAUNCH(DT, N, false);                                \
        launched = true;                                                                            \
    }
    hipError_t e = hipSuccess;
    GU_CASE(F32, 1) GU_CASE(F32, 2) GU_CASE(F32, 4) GU_CASE(F32, 8)
    GU_CASE(BF16, 1) GU_CASE(BF16, 2) GU_CASE(BF16, 4) GU_CASE(BF16, 8)
    GU_CASE(INT4, 1) GU_CASE(INT4, 2) GU_CASE(INT4, 4) GU_CASE(INT4, 8)
#undef GU_CASE
#undef GU_LAUNCH
    if (!launched) return hipErrorInvalidValue;
    if (e != hipSuccess) return e;
    if (!(parts & kFfnDown)) return hipSuccess;
    if (lds_down) {
        constexpr int rows = kDownBlock / kWave * kDownWaveRows;  // output rows per block
        const dim3 grid((H + rows - 1) / rows, T);
#define DN_CASE(DT, N)                                                                               \
        if (dtype == DT && ns == N)                                                                  \
            return launch(down_combine_lds_kernel<DT, N, kDownWaveRows, kDownBlock>, grid, kDownBlock, lds, s, T, H, \
                          I, E, k, ids, slot_of, pl, expert_bytes, sw, doff, ws.act, y, acc, pl1);
#define DN_ALL(N) DN_CASE(F32, N) DN_CASE(BF16, N) DN_CASE(INT4, N)
        DN_ALL(1) DN_ALL(2) DN_ALL(3) DN_ALL(4) DN_ALL(6) DN_ALL(8) DN_ALL(9) DN_ALL(12) DN_ALL(16)
#undef DN_ALL
#undef DN_CASE
        return hipErrorInvalidValue;
    }
    const dim3 dgrid((H + 4 * kDownRows - 1) / (4 * kDownRows), T);
    if (dtype == F32)
        return launch(down_combine_kernel<F32>, dgrid, kBlock, 0, s, T, H, I, E, k, ids, slot_of, pl,
                      expert_bytes, sw, doff, ws.act, y, acc);
    if (dtype == BF16)
        return launch(down_combine_kernel<BF16>, dgrid, kBlock, 0, s, T, H, I, E, k, ids, slot_of, pl,
                      expert_bytes, sw, doff, ws.act, y, acc);
    return launch(down_combine_kernel<INT4>, dgrid, kBlock, 0, s, T, H, I, E, k, ids, slot_of, pl,
                  expert_bytes, sw, doff, ws.act, y, acc);
}

hipError_t launch_combine(const float *y_partial, const float *weights, const float *y_shared, int T,
                          int k, int H, float *y, bool accumulate, hipStream_t s) {
    const size_t n = size_t(T) * H;
    if (n == 0) return hipSuccess;
    combine_kernel<<<unsigned((n + kBlock - 1) / kBlock), kBlock, 0, s>>>(y_partial, weights, y_shared, T,
                                                                          k, H, y, accumulate ? 1 : 0);
    return hipGetLastError();
}

namespace {
// Streams n16 16-byte words once: each wave reads kReadLoads consecutive 1 KiB
// pieces (lane-contiguous 16-byte loads with the nontemporal hint, all issued
// before any is consumed), as the expert kernels read weight rows.  Of the
// shapes tried for one 50 MB launch (128-1024 threads per block, 4-16 loads per
// lane), 256 threads x 4 loads read fastest (8.42 us against 8.57 us for 8
// loads), so it sets the practical ceiling.
constexpr int kReadLoads = 4;
__global__ __launch_bounds__(kBlock) void hbm_read_kernel(const uint8_t *__restrict__ buf, size_t n16,
                                                          float *__restrict__ sink) {
    const int lane = threadIdx.x & (kWave - 1);
    const size_t wave = size_t(blockIdx.x) * (kBlock / kWave) + threadIdx.x / kWave;
    const size_t first = wave * (kReadLoads * kWave) + lane;
    uint4 v[kReadLoads];
#pragma unroll
    for (int i = 0; i < kReadLoads; ++i) {
        const size_t w = first + size_t(i) * kWave;
        v[i] = w < n16 ? load16_stream(buf + w * 16) : make_uint4(0u, 0u, 0u, 0u);
    }
    uint32_t acc = 0;
#pragma unroll
    for (int i = 0; i < kReadLoads; ++i) acc ^= v[i].x ^ v[i].y ^ v[i].z ^ v[i].w;
    if (acc == 0x7fc00001u) sink[0] = __uint_as_float(acc);  // keeps the loads; a benign race if it fires
}
}  // namespace

hipError_t launch_hbm_read(const void *buf, size_t bytes, float *sink, hipStream_t s) {
    const size_t n16 = bytes / 16;
    if (n16 == 0) return hipSuccess;
    const size_t per_block = size_t(kReadLoads) * kBlock;  // 16-byte words per block
    const size_t blocks = (n16 + per_block - 1) / per_block;
    if (blocks >= (size_t(1) << 31)) return hipErrorInvalidValue;
    hbm_read_kernel<<<unsigned(blocks), kBlock, 0, s>>>(static_cast<const uint8_t *>(buf), n16, sink);
    return hipGetLastError();
}

hipError_t launch_fill_slots(const FillBatch &b, hipStream_t s) {
    if (b.n < 1 || b.n > kMaxFillBatch || b.n_tab < 0 || b.n_tab > 2 * kMaxFillBatch || b.bytes <= 0 || b.bytes % 16)
        return hipErrorInvalidValue;
    long long bpf = b.bytes / (64 << 10);  // 32 blocks for a 9 MiB blob; smaller blobs take fewer
    bpf = bpf < 4 ? 4 : (bpf > 32 ? 32 : bpf);
    const int ny = b.n < kHostFillsInFlight ? b.n : kHostFillsInFlight;
    fill_slots_kernel<<<dim3(unsigned(bpf), unsigned(ny)), kBlock, 0, s>>>(b);
    return hipGetLastError();
}

hipError_t launch_slot_update(int32_t *table, const int32_t *index, const int32_t *value, int n,
                              hipStream_t s) {
    for (int b = 0; b < n; b += kSlotBatch) {
        SlotUpdates u;
        u.n = n - b < kSlotBatch ? n - b : kSlotBatch;
        for (int i = 0; i < u.n; ++i) {
            u.index[i] = index[b + i];
            u.value[i] = value[b + i];
        }
        slot_update_kernel<<<1, kWave, 0, s>>>(table, u);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace moe
