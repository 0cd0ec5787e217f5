// kernels.hip -- gfx950 kernels of the MoE decode step.
//
// Every kernel streams weight rows with 16-byte loads per lane, so one wave
// instruction moves 1 KiB of a row; dot products reduce across the 64-wide
// wave with cross-lane shuffles.  fp32 accumulation throughout; bf16 and int4
// weights widen to fp32 exactly in registers.
#include <limits.h>
#include <math.h>

#include "internal.h"
#include "../../include/moe_budget.h"

namespace moe {
namespace {

constexpr int kWave = 64;
constexpr int kBlock = 256;  // 4 waves per workgroup
constexpr int kDownRows = 2; // output rows per wave in the down projection
constexpr int kDownSlots = 4; // 16-byte chunks per lane per pass of the down projection
constexpr float kRmsEps = 1e-6f;

enum : int { F32 = MOE_F32, BF16 = MOE_BF16, INT4 = MOE_INT4G128 };

// Elements held by one 16-byte chunk, and bytes per element of the dense types.
template <int DT> struct Fmt;
template <> struct Fmt<F32> { static constexpr int EPC = 4; };
template <> struct Fmt<BF16> { static constexpr int EPC = 8; };
template <> struct Fmt<INT4> { static constexpr int EPC = 32; };

__host__ __device__ constexpr size_t row_bytes_of(int DT, int cols) {
    return DT == INT4 ? size_t(cols) / 2 : size_t(cols) * (DT == F32 ? 4 : 2);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

__device__ __forceinline__ float bf16_bits_to_float(uint32_t b16) { return __uint_as_float(b16 << 16); }

__device__ __forceinline__ uint4 load16(const uint8_t *p) { return *reinterpret_cast<const uint4 *>(p); }

// EPC consecutive fp32 values of x starting at col0 (16-byte aligned).
template <int DT>
__device__ __forceinline__ void load_x(const float *__restrict__ x, int col0, float *xv) {
    const float4 *p = reinterpret_cast<const float4 *>(x + col0);
#pragma unroll
    for (int i = 0; i < Fmt<DT>::EPC / 4; ++i) {
        float4 v = p[i];
        xv[4 * i + 0] = v.x;
        xv[4 * i + 1] = v.y;
        xv[4 * i + 2] = v.z;
        xv[4 * i + 3] = v.w;
    }
}

// Dot product of one 16-byte weight chunk with EPC fp32 values.  int4 returns
// the unscaled sum of q * x (the caller applies the group scale).
template <int DT>
__device__ __forceinline__ float chunk_dot(uint4 w, const float *xv) {
    const uint32_t d[4] = {w.x, w.y, w.z, w.w};
    float acc = 0.f;
    if constexpr (DT == F32) {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc = fmaf(__uint_as_float(d[i]), xv[i], acc);
    } else if constexpr (DT == BF16) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            acc = fmaf(__uint_as_float(d[i] << 16), xv[2 * i], acc);
            acc = fmaf(__uint_as_float(d[i] & 0xffff0000u), xv[2 * i + 1], acc);
        }
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                int q = __builtin_amdgcn_sbfe(d[i], 4 * e, 4);  // signed nibble e, low nibble first
                acc = fmaf(float(q), xv[8 * i + e], acc);
            }
    }
    return acc;
}

// --------------------------------------------------------------- router ---
// z[t, e] = W_r[e, :] . h_t (+ bias[t, e]) with h_t = x_t, or with NORM
// h_t = x_t / sqrt(mean(x_t^2) + eps); one wave per (token, expert row).  Each
// wave holds the whole token row (one 16-byte column chunk per lane and
// pass), so it forms the norm itself; wave 0 of the token's first block
// stores h_t for the expert FFN.
template <int DT, int NCH, bool NORM>
__global__ __launch_bounds__(kBlock) void router_logits_kernel(const float *__restrict__ x,
                                                               const uint8_t *__restrict__ w, int H,
                                                               int E, const float *__restrict__ bias,
                                                               float *__restrict__ logits,
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
    for (int c = 0; c < NCH; ++c) {
        const int col0 = (c * kWave + lane) * EPC;
        wv[c] = (col0 < H && e < E) ? load16(row + row_bytes_of(DT, col0)) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int col0 = (c * kWave + lane) * EPC;
        if (col0 < H) {
            load_x<DT>(xt, col0, xv[c]);
        } else {
#pragma unroll
            for (int q = 0; q < EPC; ++q) xv[c][q] = 0.f;
        }
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
                if (col0 < H) {
                    float4 *o = reinterpret_cast<float4 *>(h_out + size_t(t) * H + col0);
#pragma unroll
                    for (int q = 0; q < EPC / 4; ++q)
                        o[q] = make_float4(xv[c][4 * q], xv[c][4 * q + 1], xv[c][4 * q + 2], xv[c][4 * q + 3]);
                }
            }
        }
    }
    if (e >= E) return;
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) acc += chunk_dot<DT>(wv[c], xv[c]);
    acc = wave_sum(acc);
    if (lane == 0) logits[size_t(t) * E + e] = acc + (bias ? bias[size_t(t) * E + e] : 0.f);
}

// ---------------------------------------------------------------- top-k ---
// One wave per token: each lane holds up to 4 logits (E <= 256); k rounds of a
// wave-wide arg-max ordered by (value desc, id asc), then softmax over the k.
__global__ __launch_bounds__(kBlock) void topk_softmax_kernel(const float *__restrict__ logits, int T,
                                                              int E, int k, int32_t *__restrict__ ids,
                                                              float *__restrict__ wout, int *err) {
    const int lane = threadIdx.x & (kWave - 1);
    const int t = blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave);
    if (t >= T) return;
    const float *z = logits + size_t(t) * E;
    float v[4];
    bool live[4];
    bool bad = false;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const int e = lane + kWave * m;
        live[m] = e < E;
        v[m] = live[m] ? z[e] : 0.f;
        if (live[m] && !isfinite(v[m])) bad = true;
    }
    if (__any(bad)) {
        if (lane < k) {
            ids[size_t(t) * k + lane] = -1;
            wout[size_t(t) * k + lane] = 0.f;
        }
        if (lane == 0) atomicOr(err, kErrNonfinite);
        return;
    }
    int my_id = -1;
    float my_v = 0.f, z0 = 0.f;
    for (int j = 0; j < k; ++j) {
        // lane-local best; ids grow with m, so strict '>' keeps the lower id on ties
        float bv = -INFINITY;
        int bi = INT_MAX;
#pragma unroll
        for (int m = 0; m < 4; ++m)
            if (live[m] && (bi == INT_MAX || v[m] > bv)) {
                bv = v[m];
                bi = lane + kWave * m;
            }
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) {
            const float ov = __shfl_xor(bv, off, kWave);
            const int oi = __shfl_xor(bi, off, kWave);
            if (ov > bv || (ov == bv && oi < bi)) {
                bv = ov;
                bi = oi;
            }
        }
#pragma unroll
        for (int m = 0; m < 4; ++m)
            if (bi == lane + kWave * m) live[m] = false;
        if (lane == j) {
            my_id = bi;
            my_v = bv;
        }
        if (j == 0) z0 = bv;
    }
    const float s = lane < k ? expf(my_v - z0) : 0.f;
    const float sum = wave_sum(s);
    if (lane < k) {
        ids[size_t(t) * k + lane] = my_id;
        wout[size_t(t) * k + lane] = s / sum;
    }
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

// -------------------------------------------------------------- gate/up ---
// act[p, i] = silu(W_g[i] . x_t) * (W_u[i] . x_t) for every pair p of one
// expert group.  One wave per row pair (gate row 2i, up row 2i+1): the pair's
// weights are loaded once into registers and applied to each token of the
// group.  ONE_TOKEN: T == 1, groups are the k ranks (+ shared), no table.
template <int DT, int NCH, bool ONE_TOKEN>
__global__ __launch_bounds__(kBlock) void gateup_kernel(
    const float *__restrict__ x, int T, int H, int I, int E, int k, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ slot_of, const uint8_t *__restrict__ pool, size_t expert_bytes,
    const uint8_t *__restrict__ shared_w, int *groups, float *__restrict__ act, int *err) {
    constexpr int EPC = Fmt<DT>::EPC;
    const int lane = threadIdx.x & (kWave - 1);
    const int g = blockIdx.y;
    const uint8_t *blob;
    int pstart = 0, pcount = 1, single = 0;
    const int *pairs = nullptr;
    if constexpr (ONE_TOKEN) {
        if (g < k) {
            const int e = ids[g];
            if (e < 0 || e >= E) {
                if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(err, kErrRange);
                return;
            }
            const int s = slot_of ? slot_of[e] : e;
            if (s < 0) {
                if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(err, kErrNotResident);
                return;
            }
            blob = pool + size_t(s) * expert_bytes;
        } else {
            blob = shared_w;
        }
        single = g;  // pair index: rank g, or T*k + 0 = k for the shared expert
    } else {
        if (g >= groups[0]) return;
        const int s = group_slot(groups, T, k)[g];
        pstart = group_start(groups, T, k)[g];
        pcount = group_count(groups, T, k)[g];
        pairs = group_pairs(groups, T, k);
        blob = s == -2 ? shared_w : pool + size_t(s) * expert_bytes;
    }
    const int i = blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave);
    if (i >= I) return;
    const size_t rb = row_bytes_of(DT, H);
    const uint8_t *gate = blob + size_t(2 * i) * rb;
    const uint8_t *up = gate + rb;
    uint4 wg[NCH], wu[NCH];
    float sg[NCH], su[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int col0 = (c * kWave + lane) * EPC;
        const bool in = col0 < H;
        wg[c] = in ? load16(gate + row_bytes_of(DT, col0)) : make_uint4(0, 0, 0, 0);
        wu[c] = in ? load16(up + row_bytes_of(DT, col0)) : make_uint4(0, 0, 0, 0);
        if constexpr (DT == INT4) {
            const uint16_t *sc = reinterpret_cast<const uint16_t *>(blob + size_t(I) * H);
            const int groups_per_row = H / 128;
            sg[c] = in ? bf16_bits_to_float(sc[size_t(2 * i) * groups_per_row + col0 / 128]) : 0.f;
            su[c] = in ? bf16_bits_to_float(sc[size_t(2 * i + 1) * groups_per_row + col0 / 128]) : 0.f;
        }
    }
    const int P = T * k;
    for (int q = 0; q < pcount; ++q) {
        const int p = ONE_TOKEN ? single : pairs[pstart + q];
        const int t = p < P ? p / k : p - P;
        const float *xt = x + size_t(t) * H;
        float ga = 0.f, ua = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int col0 = (c * kWave + lane) * EPC;
            if (col0 < H) {
                float xv[EPC];
                load_x<DT>(xt, col0, xv);
                float dg = chunk_dot<DT>(wg[c], xv), du = chunk_dot<DT>(wu[c], xv);
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
        if (lane == 0) act[size_t(p) * I + i] = ga / (1.f + expf(-ga)) * ua;
    }
}

// ------------------------------------------------------ down + combine ---
// y[t, h] (+)= sum_j w[t,j] * (W_d^{e_tj}[h, :] . act[t*k + j]) + W_d^shared[h, :] . act[T*k + t].
// One block per (row tile, token); the token's k (+1) down rows for output h
// form one virtual row of (k+1) * I elements that the wave streams in 16-byte
// chunks; the combine weight is folded into the activations held in registers,
// which every output row of the wave reuses.
template <int DT>
__global__ __launch_bounds__(kBlock) void down_combine_kernel(
    int T, int H, int I, int E, int k, const int32_t *__restrict__ ids,
    const float *__restrict__ weights, const int32_t *__restrict__ slot_of,
    const uint8_t *__restrict__ pool, size_t expert_bytes, const uint8_t *__restrict__ shared_w,
    size_t d_off, const float *__restrict__ act, float *__restrict__ y, int accumulate) {
    constexpr int EPC = Fmt<DT>::EPC;
    __shared__ const uint8_t *ent_ptr[MOE_MAX_TOPK + 1];
    __shared__ float ent_w[MOE_MAX_TOPK + 1];
    __shared__ int ent_p[MOE_MAX_TOPK + 1];
    const int t = blockIdx.y;
    const int NE = k + (shared_w != nullptr);
    if (threadIdx.x < NE) {
        const int j = threadIdx.x;
        const uint8_t *ptr = nullptr;
        float wj = 0.f;
        int p;
        if (j < k) {
            p = t * k + j;
            const int e = ids[p];
            if (e >= 0 && e < E) {
                const int s = slot_of ? slot_of[e] : e;
                if (s >= 0) {
                    ptr = pool + size_t(s) * expert_bytes;
                    wj = weights[p];
                }
            }
        } else {
            p = T * k + t;
            ptr = shared_w;
            wj = 1.f;
        }
        ent_ptr[j] = ptr;
        ent_w[j] = wj;
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
            rp[s] = nullptr;
            sp[s] = nullptr;
            if (gch < total) {
                const int j = gch / cpr, c = gch - j * cpr;
                const uint8_t *blob = ent_ptr[j];
                if (blob) {
                    ok[s] = true;
                    rp[s] = blob + d_off + size_t(c) * 16;
                    if constexpr (DT == INT4)
                        sp[s] = reinterpret_cast<const uint16_t *>(blob + d_sc) + (c * EPC) / 128;
                    load_x<DT>(act + size_t(ent_p[j]) * I, c * EPC, av[s]);
                    const float wj = ent_w[j];
#pragma unroll
                    for (int q = 0; q < EPC; ++q) av[s][q] *= wj;
                }
            }
        }
        uint4 wv[kDownRows][kDownSlots];
#pragma unroll
        for (int r = 0; r < kDownRows; ++r)
#pragma unroll
            for (int s = 0; s < kDownSlots; ++s)
                wv[r][s] = (ok[s] && h0 + r < H) ? load16(rp[s] + size_t(h0 + r) * rb) : make_uint4(0, 0, 0, 0);
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

int chunks_per_row(int H, int dtype) {
    const int epc = dtype == F32 ? 4 : dtype == BF16 ? 8 : 32;
    const int need = (H + kWave * epc - 1) / (kWave * epc);
    for (int n : {1, 2, 4, 8})
        if (need <= n) return n;
    return -1;
}

}  // namespace

// ===================================================================== host

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
    const dim3 grid((E + 3) / 4, T);
    const auto *wp = static_cast<const uint8_t *>(w);
    const int nch = chunks_per_row(H, w_dtype);
#define ROUTER_CASE(DT, N)                                                                          \
    if (w_dtype == DT && nch == N) {                                                                \
        if (norm)                                                                                   \
            router_logits_kernel<DT, N, true><<<grid, kBlock, 0, s>>>(x, wp, H, E, bias, logits, h_out); \
        else                                                                                        \
            router_logits_kernel<DT, N, false><<<grid, kBlock, 0, s>>>(x, wp, H, E, bias, logits, nullptr); \
        return hipGetLastError();                                                                   \
    }
    ROUTER_CASE(F32, 1) ROUTER_CASE(F32, 2) ROUTER_CASE(F32, 4) ROUTER_CASE(F32, 8)
    ROUTER_CASE(BF16, 1) ROUTER_CASE(BF16, 2) ROUTER_CASE(BF16, 4) ROUTER_CASE(BF16, 8)
#undef ROUTER_CASE
    return hipErrorInvalidValue;
}

hipError_t launch_topk_softmax(const float *logits, int T, int E, int k, int32_t *ids, float *weights,
                               int *err_flags, hipStream_t s) {
    if (T == 0) return hipSuccess;
    topk_softmax_kernel<<<(T + 3) / 4, kBlock, 0, s>>>(logits, T, E, k, ids, weights, err_flags);
    return hipGetLastError();
}

hipError_t launch_expert_ffn(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                             const float *weights, const int32_t *slot_of, const void *pool,
                             size_t expert_bytes, int dtype, const void *shared_w, float *y,
                             bool accumulate, const FfnWorkspace &ws, int *err_flags, hipStream_t s,
                             const FfnEvents *ev) {
    if (T == 0) return hipSuccess;
    const bool one = T == 1;
    const int has_shared = shared_w != nullptr;
    const auto *pl = static_cast<const uint8_t *>(pool);
    const auto *sw = static_cast<const uint8_t *>(shared_w);
    if (!one) {
        group_pairs_kernel<<<1, kBlock, 0, s>>>(ids, T, k, E, slot_of, has_shared, ws.groups, err_flags);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (ev) (void)hipEventRecord(ev->gu_begin, s);
    const int groups = one ? k + has_shared : (T * k < E ? T * k : E) + has_shared;
    const dim3 ggrid((I + 3) / 4, groups);
    const int nch = chunks_per_row(H, dtype);
    bool launched = false;
#define GU_CASE(DT, N)                                                                              \
    if (!launched && dtype == DT && nch == N) {                                                     \
        if (one)                                                                                    \
            gateup_kernel<DT, N, true><<<ggrid, kBlock, 0, s>>>(x, T, H, I, E, k, ids, slot_of, pl,  \
                                                                expert_bytes, sw, ws.groups,        \
                                                                ws.act, err_flags);                 \
        else                                                                                        \
            gateup_kernel<DT, N, false><<<ggrid, kBlock, 0, s>>>(x, T, H, I, E, k, ids, slot_of, pl, \
                                                                 expert_bytes, sw, ws.groups,       \
                                                                 ws.act, err_flags);                \
        launched = true;                                                                            \
    }
    GU_CASE(F32, 1) GU_CASE(F32, 2) GU_CASE(F32, 4) GU_CASE(F32, 8)
    GU_CASE(BF16, 1) GU_CASE(BF16, 2) GU_CASE(BF16, 4) GU_CASE(BF16, 8)
    GU_CASE(INT4, 1) GU_CASE(INT4, 2) GU_CASE(INT4, 4) GU_CASE(INT4, 8)
#undef GU_CASE
    if (!launched) return hipErrorInvalidValue;
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (ev) (void)hipEventRecord(ev->gu_end, s);
    const dim3 dgrid((H + 4 * kDownRows - 1) / (4 * kDownRows), T);
    const size_t doff = down_offset(H, I, dtype);
    const int acc = accumulate ? 1 : 0;
    if (dtype == F32)
        down_combine_kernel<F32><<<dgrid, kBlock, 0, s>>>(T, H, I, E, k, ids, weights, slot_of, pl,
                                                           expert_bytes, sw, doff, ws.act, y, acc);
    else if (dtype == BF16)
        down_combine_kernel<BF16><<<dgrid, kBlock, 0, s>>>(T, H, I, E, k, ids, weights, slot_of, pl,
                                                            expert_bytes, sw, doff, ws.act, y, acc);
    else
        down_combine_kernel<INT4><<<dgrid, kBlock, 0, s>>>(T, H, I, E, k, ids, weights, slot_of, pl,
                                                            expert_bytes, sw, doff, ws.act, y, acc);
    e = hipGetLastError();
    if (ev) (void)hipEventRecord(ev->dn_end, s);
    return e;
}

hipError_t launch_combine(const float *y_partial, const float *weights, const float *y_shared, int T,
                          int k, int H, float *y, bool accumulate, hipStream_t s) {
    const size_t n = size_t(T) * H;
    if (n == 0) return hipSuccess;
    combine_kernel<<<unsigned((n + kBlock - 1) / kBlock), kBlock, 0, s>>>(y_partial, weights, y_shared, T,
                                                                          k, H, y, accumulate ? 1 : 0);
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
