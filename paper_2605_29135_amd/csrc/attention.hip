// attention.hip -- the decoder self-attention block of one decode token.
//
// The paper runs its model with a 4096-token context and attention on the
// accelerator (sec. 6); the block is a Qwen3-class reading: RMS pre-norm, one
// fused QKV projection, grouped-query heads with per-head RMS norm and the
// rotary position embedding (rotate-half form), a bf16 KV cache, softmax
// attention over positions 0..p, the output projection added to the residual.
//
//   1. QKV projection with the pre-norm: the router GEMV (one wave per row).
//   2. attn_heads_kernel: one wave per query head and per key head: RMS norm over
//      the head, rotation of the pairs (i, i + d/2) held by lane i, the query
//      written back in place, key and value appended to the caches at p.
//   3. attn_partial_kernel: one wave per (key/value head, 64 positions): lane j
//      scores position j against every query head of the group (queries read as
//      LDS broadcasts, keys as one 1 KiB contiguous load per 8 dimensions from
//      the [d/8][position][8] key layout), per-head max and sum over the wave,
//      then lanes switch to dimensions for the probability-weighted sum of the
//      value rows (row-major value layout); partial (max, sum, output) per
//      (query head, chunk).
//   4. attn_combine_kernel: per query head, the chunks merged by log-sum-exp.
//   5. Output projection: the same GEMV with the residual as its bias, in place.
#include "device_common.h"
#include "internal.h"

namespace moe {
namespace {

using dev::kBlock;
using dev::kWave;
using dev::wave_sum;
using dev::BF16;

constexpr int kAttnChunk = 64;     // positions per wave in the partial kernel
constexpr int kAttnMaxGroup = 16;  // query heads per key/value head

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
    return v;
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Waves 0..n_heads-1: query heads (normalised and rotated in place in qkv);
// waves n_heads..n_heads+n_kv-1: key heads, appended with their value heads.
__global__ __launch_bounds__(kBlock) void attn_heads_kernel(float *__restrict__ qkv, int n_heads, int n_kv, int d,
                                                            uint16_t *__restrict__ k_cache,
                                                            uint16_t *__restrict__ v_cache, int max_pos, int p,
                                                            float theta) {
    const int lane = threadIdx.x & (kWave - 1);
    const int w = blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
    if (w >= n_heads + n_kv) return;
    const int half = d / 2;
    float *head = qkv + size_t(w) * d;  // keys follow the queries in qkv
    const bool on = lane < half;
    float a = on ? head[lane] : 0.f, b = on ? head[lane + half] : 0.f;
    const float inv = rsqrtf(wave_sum(a * a + b * b) / float(d) + 1e-6f);
    a *= inv;
    b *= inv;
    // angle p * theta^(-2i/d), reduced in double so that positions up to thousands keep full precision
    const double ang = double(p) * pow(double(theta), -2.0 * double(lane) / double(d));
    double sd, cd;
    sincos(ang, &sd, &cd);
    const float c = float(cd), s = float(sd);
    const float ra = a * c - b * s, rb = b * c + a * s;
    if (!on) return;
    if (w < n_heads) {
        head[lane] = ra;
        head[lane + half] = rb;
        return;
    }
    const int g = w - n_heads;
    const float *vh = qkv + size_t(n_heads + n_kv + g) * d;
    // key layout [g][d/8][max_pos][8]; value layout [g][max_pos][d]
    auto kidx = [&](int i) { return ((size_t(g) * (d / 8) + i / 8) * max_pos + p) * 8 + (i % 8); };
    k_cache[kidx(lane)] = f32_to_bf16_rne(ra);
    k_cache[kidx(lane + half)] = f32_to_bf16_rne(rb);
    v_cache[(size_t(g) * max_pos + p) * d + lane] = f32_to_bf16_rne(vh[lane]);
    v_cache[(size_t(g) * max_pos + p) * d + lane + half] = f32_to_bf16_rne(vh[lane + half]);
}

// Block = 4 waves = 4 chunks of 64 positions of one key/value head g (blockIdx.y).  part layout:
// [query head][chunk][d + 2] (unnormalised output, then max, then sum).  d is a multiple of 8, at most 128.
__global__ __launch_bounds__(kBlock) void attn_partial_kernel(const float *__restrict__ q, int n_heads, int n_kv,
                                                              int d, const uint16_t *__restrict__ k_cache,
                                                              const uint16_t *__restrict__ v_cache, int max_pos,
                                                              int n_pos, int n_chunks, float *__restrict__ part) {
    __shared__ float qs[kAttnMaxGroup * 128];                       // the group's queries
    __shared__ float prob[kBlock / kWave][kAttnMaxGroup][kAttnChunk];  // per wave: probabilities by head, position
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int g = blockIdx.y, group = n_heads / n_kv;
    for (int i = threadIdx.x; i < group * d; i += kBlock) qs[i] = q[size_t(g) * group * d + i];
    __syncthreads();
    const int chunk = blockIdx.x * (kBlock / kWave) + wave;
    if (chunk >= n_chunks) return;
    const int pos = chunk * kAttnChunk + lane;
    const bool live = pos < n_pos;
    const int pc = live ? pos : n_pos - 1;  // clamped: loads stay in bounds, the score is discarded
    // scores of this lane's position against every query head of the group
    float sc[kAttnMaxGroup];
#pragma unroll
    for (int h = 0; h < kAttnMaxGroup; ++h) sc[h] = 0.f;
    const uint16_t *kb = k_cache + (size_t(g) * (d / 8) * max_pos + pc) * 8;
    for (int c = 0; c < d / 8; ++c) {
        const uint4 kw4 = dev::load16(reinterpret_cast<const uint8_t *>(kb + size_t(c) * max_pos * 8));
        const uint32_t kw[4] = {kw4.x, kw4.y, kw4.z, kw4.w};
        float kv[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {  // dims 8c + 2i (low half) and 8c + 2i + 1 (high half)
            kv[2 * i] = __uint_as_float(kw[i] << 16);
            kv[2 * i + 1] = __uint_as_float(kw[i] & 0xffff0000u);
        }
#pragma unroll
        for (int h = 0; h < kAttnMaxGroup; ++h) {
            if (h < group) {
                const float *qh = qs + h * d + c * 8;
#pragma unroll
                for (int i = 0; i < 8; ++i) sc[h] = fmaf(qh[i], kv[i], sc[h]);
            }
        }
    }
    const float scale = rsqrtf(float(d));
    float mx[kAttnMaxGroup], sm[kAttnMaxGroup];
#pragma unroll
    for (int h = 0; h < kAttnMaxGroup; ++h) {
        if (h < group) {
            const float s = live ? sc[h] * scale : -INFINITY;
            mx[h] = wave_max(s);
            const float e = live ? __expf(s - mx[h]) : 0.f;
            sm[h] = wave_sum(e);
            prob[wave][h][lane] = e;
        }
    }
    // the probabilities are this wave's own (waves past the last chunk have left): a wave-level LDS sync
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    // output: lanes over dimensions (2 per lane), the chunk's value rows weighted by each head's probabilities
    float o0[kAttnMaxGroup], o1[kAttnMaxGroup];
#pragma unroll
    for (int h = 0; h < kAttnMaxGroup; ++h) o0[h] = o1[h] = 0.f;
    const int dim = 2 * lane;
    const bool dlive = dim < d;
    const int n_here = min(kAttnChunk, n_pos - chunk * kAttnChunk);
    const uint16_t *vb = v_cache + (size_t(g) * max_pos + size_t(chunk) * kAttnChunk) * d + (dlive ? dim : 0);
    for (int j0 = 0; j0 < n_here; j0 += 8) {
        uint32_t vv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)  // 8 rows in flight; rows past n_here repeat the last live one (weight 0)
            vv[u] = *reinterpret_cast<const uint32_t *>(vb + size_t(min(j0 + u, n_here - 1)) * d);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const float v0 = __uint_as_float(vv[u] << 16), v1 = __uint_as_float(vv[u] & 0xffff0000u);
            const int j = j0 + u;
#pragma unroll
            for (int h = 0; h < kAttnMaxGroup; ++h) {
                if (h < group) {
                    const float pr = j < n_here ? prob[wave][h][j] : 0.f;
                    o0[h] = fmaf(pr, v0, o0[h]);
                    o1[h] = fmaf(pr, v1, o1[h]);
                }
            }
        }
    }
#pragma unroll
    for (int h = 0; h < kAttnMaxGroup; ++h) {
        if (h < group) {
            float *pp = part + (size_t(g * group + h) * n_chunks + chunk) * (d + 2);
            if (dlive) {
                pp[dim] = o0[h];
                pp[dim + 1] = o1[h];
            }
            if (lane == 0) {
                pp[d] = mx[h];
                pp[d + 1] = sm[h];
            }
        }
    }
}

// One block per query head: att[h][i] = sum_c e^(m_c - M) o_c[i] / sum_c e^(m_c - M) s_c.
__global__ __launch_bounds__(kBlock) void attn_combine_kernel(const float *__restrict__ part, int d, int n_chunks,
                                                              float *__restrict__ att) {
    const int h = blockIdx.x;
    const float *ph = part + size_t(h) * n_chunks * (d + 2);
    float M = -INFINITY;
    for (int c = 0; c < n_chunks; ++c) M = fmaxf(M, ph[size_t(c) * (d + 2) + d]);
    float S = 0.f;
    for (int c = 0; c < n_chunks; ++c) S += __expf(ph[size_t(c) * (d + 2) + d] - M) * ph[size_t(c) * (d + 2) + d + 1];
    for (int i = threadIdx.x; i < d; i += kBlock) {
        float acc = 0.f;
        for (int c = 0; c < n_chunks; ++c) acc += __expf(ph[size_t(c) * (d + 2) + d] - M) * ph[size_t(c) * (d + 2) + i];
        att[size_t(h) * d + i] = acc / S;
    }
}

}  // namespace

using dev::BF16;

bool attention_shape_supported(int H, int n_heads, int n_kv, int d, int max_pos) {
    return H > 0 && H % 128 == 0 && n_heads > 0 && n_kv > 0 && n_heads % n_kv == 0 &&
           n_heads / n_kv <= kAttnMaxGroup && d >= 8 && d <= 128 && d % 8 == 0 && (n_heads * d) % 128 == 0 &&
           max_pos > 0 && ffn_shape_supported(H, 128, BF16) && router_shape_supported(n_heads * d, BF16);
}

static size_t align256a(size_t n) { return (n + 255) & ~size_t(255); }

size_t attention_workspace_bytes(int n_heads, int n_kv, int d, int max_pos) {
    const size_t chunks = size_t((max_pos + kAttnChunk - 1) / kAttnChunk);
    return align256a(sizeof(float) * size_t(n_heads + 2 * n_kv) * d) + align256a(sizeof(float) * size_t(n_heads) * d) +
           align256a(sizeof(float) * size_t(n_heads) * chunks * (d + 2));
}

hipError_t launch_attention_decode(float *x, int H, int n_heads, int n_kv, int d, const void *w_qkv, const void *w_o,
                                   uint16_t *k_cache, uint16_t *v_cache, int max_pos, int p, float theta,
                                   void *workspace, hipStream_t s) {
    const int rows = (n_heads + 2 * n_kv) * d, n_pos = p + 1;
    const int n_chunks = (n_pos + kAttnChunk - 1) / kAttnChunk;
    const size_t max_chunks = size_t((max_pos + kAttnChunk - 1) / kAttnChunk);
    char *ws = static_cast<char *>(workspace);
    float *qkv = reinterpret_cast<float *>(ws);
    float *att = reinterpret_cast<float *>(ws + align256a(sizeof(float) * size_t(rows)));
    float *part = reinterpret_cast<float *>(ws + align256a(sizeof(float) * size_t(rows)) +
                                            align256a(sizeof(float) * size_t(n_heads) * d));
    (void)max_chunks;
    hipError_t e = launch_router_logits(x, w_qkv, BF16, 1, H, rows, nullptr, qkv, true, nullptr, s);
    if (e != hipSuccess) return e;
    attn_heads_kernel<<<(n_heads + n_kv + 3) / 4, kBlock, 0, s>>>(qkv, n_heads, n_kv, d, k_cache, v_cache, max_pos, p,
                                                                   theta);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    attn_partial_kernel<<<dim3((n_chunks + 3) / 4, n_kv), kBlock, 0, s>>>(qkv, n_heads, n_kv, d, k_cache, v_cache,
                                                                         max_pos, n_pos, n_chunks, part);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    attn_combine_kernel<<<n_heads, kBlock, 0, s>>>(part, d, n_chunks, att);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_router_logits(att, w_o, BF16, 1, n_heads * d, H, x, x, false, nullptr, s);
}

}  // namespace moe
