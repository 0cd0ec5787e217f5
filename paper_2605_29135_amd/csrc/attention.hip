// attention.hip -- the decoder self-attention block of one decode token.
//
// The paper runs its model with a 4096-token context and attention on the
// accelerator (sec. 6); the block is a Qwen3-class reading: RMS pre-norm, one
// fused QKV projection, grouped-query heads with per-head RMS norm and the
// rotary position embedding (rotate-half form), a bf16 KV cache, softmax
// attention over positions 0..p, the output projection added to the residual.
//
//   1. QKV projection with the pre-norm: the router GEMV (one wave per row).
//   2. attn_partial_kernel: one block per (key/value head, 64 positions), 8 waves
//      of 8 positions.  The block normalises and rotates its group's queries into
//      LDS (the block of the last chunk also forms the key and value of p and
//      appends them to the caches); lanes (dimension slice, position) score the
//      positions against every query head of the group (queries read as LDS
//      broadcasts, keys from the [d/8][position][8] layout), per-head max and sum
//      over the wave's positions, then lanes switch to dimensions for the
//      probability-weighted sum of the value rows (row-major value layout); the 8
//      waves merge into one partial (max, sum, output) per (query head, chunk).
//   3. attn_combine_kernel: per query head, the chunks merged by log-sum-exp.
//   4. Output projection: the same GEMV with the residual as its bias, in place.
#include "device_common.h"
#include "internal.h"

namespace moe {
namespace {

using dev::kBlock;
using dev::kWave;
using dev::wave_sum;
using dev::BF16;
using dev::dpp;

constexpr int kAttnChunk = 64;  // positions per block (one partial per query head) in the partial kernel

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

// Rotation of dimension pair (i, i + d/2) at position p: angle p * theta^(-2i/d).  The angle is formed and
// reduced to [-pi, pi] in double, so thousands of positions keep full single precision in cos and sin.
__device__ __forceinline__ void rope_cs(int p, int i, int d, float theta, float &c, float &s) {
    const double inv_freq = exp2(-2.0 * double(i) / double(d) * log2(double(theta)));
    const double ang = double(p) * inv_freq;
    constexpr double kTwoPi = 6.283185307179586;
    const double r = fma(-rint(ang * (1.0 / kTwoPi)), kTwoPi, ang);
    double sd, cd;
    sincos(r, &sd, &cd);
    c = float(cd);
    s = float(sd);
}

// Block = one chunk of 64 positions of key/value head g (blockIdx.y), 8 waves of 8 positions.  The block first
// brings its group's queries to their final form (RMS norm over each head, rotation at p), and the block of the
// last chunk also the key and value of position p, which it appends to the caches and uses from LDS.  part layout:
// [query head][chunk][d + 4] (unnormalised output, then max, then sum; rows padded to 16 bytes).  d is a
// multiple of 8, at most 128.  Every load of a wave -- its positions' key pieces and their value rows, which
// do not depend on the scores -- is issued before any is used: one memory round trip per wave.
constexpr int kAttnWaves = 8;
constexpr int kAttnBlock = kAttnWaves * kWave;      // threads of a partial block
constexpr int kPosW = kAttnChunk / kAttnWaves;      // positions per wave
constexpr int kSlices = kWave / kPosW;              // lanes per position in the scores (dimension slices)
constexpr int kMaxDC = 16;                          // key pieces of 8 dims per position (d <= 128)
constexpr int kPPS = kMaxDC / kSlices;              // key pieces per slice
static_assert(kPosW == 8 && kSlices == 8, "lane layout of the partial kernel");

// Max and sum over the 8 lanes of a half-row (DPP quad swaps and the half-row mirror).
__device__ __forceinline__ float lanes8_max(float v) {
    v = fmaxf(v, dpp<0xB1>(v));
    v = fmaxf(v, dpp<0x4E>(v));
    return fmaxf(v, dpp<0x141>(v));
}
__device__ __forceinline__ float lanes8_sum(float v) {
    v += dpp<0xB1>(v);
    v += dpp<0x4E>(v);
    return v + dpp<0x141>(v);
}

// GROUP = query heads per key/value head; FULL = (d == 128).  Both compile time, so every loop over heads
// and key pieces is static.
//   heads:   job j = wave, wave + 8, ...: query head j of the group, job GROUP (last chunk only) the key and
//            value heads; lane i holds the pair (i, i + d/2);
//   scores: lane = slice * 8 + position; slice s dots key pieces s and s + 8 (8 dims each) with every query
//           head of the group (queries read from LDS as float4 broadcasts), then the 8 slices are summed
//           (row rotation by 8, then two cross-row swaps);
//   softmax: per head, max and sum over the wave's 8 positions;
//   output:  lane = dimension pair, the 8 value rows weighted by each head's probabilities (from LDS);
//   merge:   the 8 waves' (max, sum, output) per head merged through LDS into the chunk's partial, at most
//            8 heads per pass.
template <int GROUP, bool FULL>
__global__ __launch_bounds__(kAttnBlock) void attn_partial_kernel(const float *__restrict__ qkv, int d_arg,
                                                                  uint16_t *__restrict__ k_cache,
                                                                  uint16_t *__restrict__ v_cache, int max_pos,
                                                                  int n_pos, float theta, int n_chunks,
                                                                  float *__restrict__ part) {
    constexpr int HB = GROUP < 8 ? GROUP : 8;  // heads per merge pass
    __shared__ float4 qs4[GROUP * 128 / 4];                    // the group's queries, [head][d]
    __shared__ float4 prob4[kAttnWaves][GROUP][kPosW / 4];     // per wave: probabilities [head][position]
    __shared__ float wm[kAttnWaves][GROUP], ws[kAttnWaves][GROUP];
    __shared__ float wo[kAttnWaves][HB][128];
    __shared__ uint4 knew4[128 / 8], vnew4[128 / 8];  // bf16 key and value of position p (last chunk)
    float *qs = reinterpret_cast<float *>(qs4);
    uint16_t *knew = reinterpret_cast<uint16_t *>(knew4), *vnew = reinterpret_cast<uint16_t *>(vnew4);
    const int d = FULL ? 128 : d_arg, dc = d / 8;
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int g = blockIdx.y, chunk = blockIdx.x, n_kv = gridDim.y, p = n_pos - 1;
    const bool last = chunk == n_chunks - 1;  // holds position p
    const int pl = lane % kPosW, slice = lane / kPosW;
    const int pos0 = chunk * kAttnChunk + wave * kPosW;
    const int n_here = max(0, min(kPosW, n_pos - pos0));  // live positions of this wave (wave 0 has >= 1)
    const bool live = pl < n_here;
    // 1. all loads, clamped to the last position: keys (lanes = slice, position), values (lanes = dimensions)
    uint4 kw[kPPS];
    const uint16_t *kb = k_cache + (size_t(g) * dc * max_pos + min(pos0 + pl, n_pos - 1)) * 8;
#pragma unroll
    for (int i = 0; i < kPPS; ++i) {
        const int c = FULL ? slice + kSlices * i : min(slice + kSlices * i, dc - 1);
        kw[i] = dev::load16(reinterpret_cast<const uint8_t *>(kb + size_t(c) * max_pos * 8));
    }
    const int dim = 2 * lane;
    const bool dlive = FULL || dim < d;
    uint32_t vv[kPosW];
    const uint16_t *vb = v_cache + size_t(g) * max_pos * d + (dlive ? dim : 0);
#pragma unroll
    for (int j = 0; j < kPosW; ++j)
        vv[j] = *reinterpret_cast<const uint32_t *>(vb + size_t(min(pos0 + j, n_pos - 1)) * d);
    // 2. heads: queries normalised and rotated into LDS; the new key and value (last chunk)
    {
        const int half = d / 2;
        const bool on = lane < half;
        float rc = 0.f, rs = 0.f;
        rope_cs(p, lane, d, theta, rc, rs);
        for (int j = wave; j < GROUP + (last ? 1 : 0); j += kAttnWaves) {
            const int row = j < GROUP ? g * GROUP + j : GROUP * n_kv + g;  // query head, else key head
            const float *src = qkv + size_t(row) * d;
            float a = on ? src[lane] : 0.f, b = on ? src[lane + half] : 0.f;
            const float inv = rsqrtf(wave_sum(a * a + b * b) / float(d) + 1e-6f);
            a *= inv;
            b *= inv;
            const float ra = a * rc - b * rs, rb = b * rc + a * rs;
            if (!on) continue;
            if (j < GROUP) {
                qs[j * d + lane] = ra;
                qs[j * d + lane + half] = rb;
                continue;
            }
            // key layout [g][d/8][max_pos][8]; value layout [g][max_pos][d]
            const float *vsrc = qkv + size_t(GROUP * n_kv + n_kv + g) * d;
            const uint16_t k0 = f32_to_bf16_rne(ra), k1 = f32_to_bf16_rne(rb);
            const uint16_t v0 = f32_to_bf16_rne(vsrc[lane]), v1 = f32_to_bf16_rne(vsrc[lane + half]);
            knew[lane] = k0;
            knew[lane + half] = k1;
            vnew[lane] = v0;
            vnew[lane + half] = v1;
            auto kidx = [&](int i) { return ((size_t(g) * dc + i / 8) * max_pos + p) * 8 + (i % 8); };
            k_cache[kidx(lane)] = k0;
            k_cache[kidx(lane + half)] = k1;
            v_cache[(size_t(g) * max_pos + p) * d + lane] = v0;
            v_cache[(size_t(g) * max_pos + p) * d + lane + half] = v1;
        }
    }
    __syncthreads();
    // Position p: the key and value just formed, not the cache's previous content.  Loads clamped to p (past
    // the last position) take them too: their weight is 0, and 0 times a stale NaN would not be.
    if (last) {
        if (pos0 + pl >= p) {
#pragma unroll
            for (int i = 0; i < kPPS; ++i) {
                const int c = slice + kSlices * i;
                if (FULL || c < dc) kw[i] = knew4[c];
            }
        }
        if (dlive) {
            const uint32_t vp = *reinterpret_cast<const uint32_t *>(vnew + dim);
#pragma unroll
            for (int j = 0; j < kPosW; ++j)
                if (pos0 + j >= p) vv[j] = vp;
        }
    }
    // 3. scores
    float sc[GROUP];
#pragma unroll
    for (int h = 0; h < GROUP; ++h) sc[h] = 0.f;
#pragma unroll
    for (int i = 0; i < kPPS; ++i) {
        const int c = slice + kSlices * i;
        if (FULL || c < dc) {
            const uint32_t kwv[4] = {kw[i].x, kw[i].y, kw[i].z, kw[i].w};
            float kv[8];
#pragma unroll
            for (int u = 0; u < 4; ++u) {  // dims 8c + 2u (low half) and 8c + 2u + 1 (high half)
                kv[2 * u] = __uint_as_float(kwv[u] << 16);
                kv[2 * u + 1] = __uint_as_float(kwv[u] & 0xffff0000u);
            }
#pragma unroll
            for (int h = 0; h < GROUP; ++h) {
                const float4 qa = qs4[(h * d + c * 8) / 4], qb = qs4[(h * d + c * 8) / 4 + 1];
                float t = sc[h];
                t = fmaf(qa.x, kv[0], t);
                t = fmaf(qa.y, kv[1], t);
                t = fmaf(qa.z, kv[2], t);
                t = fmaf(qa.w, kv[3], t);
                t = fmaf(qb.x, kv[4], t);
                t = fmaf(qb.y, kv[5], t);
                t = fmaf(qb.z, kv[6], t);
                sc[h] = fmaf(qb.w, kv[7], t);
            }
        }
    }
    // 4. softmax over the wave's positions; slice 0's lanes keep the probabilities in LDS
    const float scale = rsqrtf(float(d));
    float mx[GROUP], sm[GROUP];
    float *pw = reinterpret_cast<float *>(prob4[wave]);
#pragma unroll
    for (int h = 0; h < GROUP; ++h) {
        float t = sc[h];
        t += dpp<0x128>(t);  // row rotation by 8: slices 2r and 2r + 1
        t += __shfl_xor(t, 16);
        t += __shfl_xor(t, 32);
        const float s = live ? t * scale : -INFINITY;
        mx[h] = lanes8_max(s);
        const float e = live ? __expf(s - mx[h]) : 0.f;
        sm[h] = lanes8_sum(e);
        if (slice == 0) pw[h * kPosW + pl] = e;
    }
    // the probabilities are this wave's own: a wave-level LDS sync
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    // 5. output: lanes over dimensions (2 per lane); probabilities are 0 past the live positions
    float o0[GROUP], o1[GROUP];
#pragma unroll
    for (int h = 0; h < GROUP; ++h) o0[h] = o1[h] = 0.f;
#pragma unroll
    for (int j4 = 0; j4 < kPosW / 4; ++j4) {
        float v0[4], v1[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            v0[u] = __uint_as_float(vv[4 * j4 + u] << 16);
            v1[u] = __uint_as_float(vv[4 * j4 + u] & 0xffff0000u);
        }
#pragma unroll
        for (int h = 0; h < GROUP; ++h) {
            const float4 pr = prob4[wave][h][j4];
            o0[h] = fmaf(pr.w, v0[3], fmaf(pr.z, v0[2], fmaf(pr.y, v0[1], fmaf(pr.x, v0[0], o0[h]))));
            o1[h] = fmaf(pr.w, v1[3], fmaf(pr.z, v1[2], fmaf(pr.y, v1[1], fmaf(pr.x, v1[0], o1[h]))));
        }
    }
    // 6. merge the 8 waves (a wave with no live position has max -inf, sum 0, output 0)
    if (lane == 0) {
#pragma unroll
        for (int h = 0; h < GROUP; ++h) {
            wm[wave][h] = mx[h];
            ws[wave][h] = sm[h];
        }
    }
#pragma unroll
    for (int hb = 0; hb < GROUP / HB; ++hb) {
        if (dlive) {
#pragma unroll
            for (int hh = 0; hh < HB; ++hh) {
                wo[wave][hh][dim] = o0[hb * HB + hh];
                wo[wave][hh][dim + 1] = o1[hb * HB + hh];
            }
        }
        __syncthreads();
        for (int idx = threadIdx.x; idx < HB * d; idx += kAttnBlock) {
            const int hh = idx / d, i = idx - hh * d, h = hb * HB + hh;
            float M = wm[0][h];
#pragma unroll
            for (int w = 1; w < kAttnWaves; ++w) M = fmaxf(M, wm[w][h]);  // finite: wave 0 has a live position
            float o = 0.f, S = 0.f;
#pragma unroll
            for (int w = 0; w < kAttnWaves; ++w) {
                const float f = __expf(wm[w][h] - M);
                o = fmaf(f, wo[w][hh][i], o);
                S = fmaf(f, ws[w][h], S);
            }
            float *pp = part + (size_t(g * GROUP + h) * n_chunks + chunk) * (d + 4);
            pp[i] = o;
            if (i == 0) {
                pp[d] = M;
                pp[d + 1] = S;
            }
        }
        if (hb + 1 < GROUP / HB) __syncthreads();  // before the next pass overwrites wo
    }
}

// One block per query head: att[h][i] = sum_c e^(m_c - M) o_c[i] / sum_c e^(m_c - M) s_c.  Thread t first
// issues the loads of its share of the outputs (4 dimensions as one float4, chunks t/32, t/32 + 8, ...),
// then reads chunk t's max and sum (n_chunks <= kBlock) and the block reduces those to the weights.
constexpr int kCombineBatch = 8;  // outputs loaded per thread per round trip
__global__ __launch_bounds__(kBlock) void attn_combine_kernel(const float *__restrict__ part, int d, int n_chunks,
                                                              float *__restrict__ att) {
    __shared__ float red[kBlock / kWave];
    __shared__ float wgt[kBlock];
    __shared__ float4 acc_sh[kBlock / 32][32];
    const int h = blockIdx.x, tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int stride = d + 4;
    const float *ph = part + size_t(h) * n_chunks * stride;
    const int i4 = tid % 32, cs = tid / 32;  // dimensions 4*i4..4*i4+3, chunks cs + 8k
    const bool ilive = 4 * i4 < d;
    float4 v[kCombineBatch];
#pragma unroll
    for (int k = 0; k < kCombineBatch; ++k) {
        const int c = cs + (kBlock / 32) * k;
        v[k] = (ilive && c < n_chunks) ? *reinterpret_cast<const float4 *>(ph + size_t(c) * stride + 4 * i4)
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    const bool live = tid < n_chunks;
    const float m = live ? ph[size_t(tid) * stride + d] : -INFINITY;
    const float sv = live ? ph[size_t(tid) * stride + d + 1] : 0.f;
    float M = wave_max(m);
    if (lane == 0) red[wave] = M;
    __syncthreads();
    M = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    const float e = live ? __expf(m - M) : 0.f;
    float S = wave_sum(e * sv);
    if (lane == 0) red[wave] = S;
    __syncthreads();
    S = red[0] + red[1] + red[2] + red[3];
    wgt[tid] = e / S;
    __syncthreads();
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int base = 0;; base += kCombineBatch * (kBlock / 32)) {
#pragma unroll
        for (int k = 0; k < kCombineBatch; ++k) {
            const int c = base + cs + (kBlock / 32) * k;
            const float w = c < n_chunks ? wgt[c] : 0.f;
            acc.x = fmaf(w, v[k].x, acc.x);
            acc.y = fmaf(w, v[k].y, acc.y);
            acc.z = fmaf(w, v[k].z, acc.z);
            acc.w = fmaf(w, v[k].w, acc.w);
        }
        const int next = base + kCombineBatch * (kBlock / 32);
        if (next >= n_chunks) break;
#pragma unroll
        for (int k = 0; k < kCombineBatch; ++k) {
            const int c = next + cs + (kBlock / 32) * k;
            v[k] = (ilive && c < n_chunks) ? *reinterpret_cast<const float4 *>(ph + size_t(c) * stride + 4 * i4)
                                           : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
    acc_sh[cs][i4] = acc;
    __syncthreads();
    if (tid < 32 && ilive) {
        float4 r = acc_sh[0][tid];
#pragma unroll
        for (int k = 1; k < kBlock / 32; ++k) {
            const float4 t = acc_sh[k][tid];
            r.x += t.x;
            r.y += t.y;
            r.z += t.z;
            r.w += t.w;
        }
        *reinterpret_cast<float4 *>(att + size_t(h) * d + 4 * tid) = r;
    }
}

}  // namespace

using dev::BF16;

bool attention_shape_supported(int H, int n_heads, int n_kv, int d, int max_pos) {
    const int grp = n_kv > 0 ? n_heads / n_kv : 0;
    return H > 0 && H % 128 == 0 && n_heads > 0 && n_kv > 0 && n_heads % n_kv == 0 &&
           (grp == 1 || grp == 2 || grp == 4 || grp == 8 || grp == 16) && d >= 8 && d <= 128 && d % 8 == 0 && (n_heads * d) % 128 == 0 &&
           max_pos > 0 && max_pos <= kBlock * kAttnChunk && ffn_shape_supported(H, 128, BF16) &&
           router_shape_supported(n_heads * d, BF16);
}

static size_t align256a(size_t n) { return (n + 255) & ~size_t(255); }

size_t attention_workspace_bytes(int n_heads, int n_kv, int d, int max_pos) {
    const size_t chunks = size_t((max_pos + kAttnChunk - 1) / kAttnChunk);
    return align256a(sizeof(float) * size_t(n_heads + 2 * n_kv) * d) + align256a(sizeof(float) * size_t(n_heads) * d) +
           align256a(sizeof(float) * size_t(n_heads) * chunks * (d + 4));
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
    const dim3 pgrid(n_chunks, n_kv);
    const bool full = d == 128;
    switch (n_heads / n_kv) {
#define ATTN_GROUP(G)                                                                                            \
    case G:                                                                                                      \
        if (full)                                                                                                \
            attn_partial_kernel<G, true>                                                                         \
                <<<pgrid, kAttnBlock, 0, s>>>(qkv, d, k_cache, v_cache, max_pos, n_pos, theta, n_chunks, part); \
        else                                                                                                     \
            attn_partial_kernel<G, false>                                                                        \
                <<<pgrid, kAttnBlock, 0, s>>>(qkv, d, k_cache, v_cache, max_pos, n_pos, theta, n_chunks, part); \
        break;
        ATTN_GROUP(1) ATTN_GROUP(2) ATTN_GROUP(4) ATTN_GROUP(8) ATTN_GROUP(16)
#undef ATTN_GROUP
    default:
        return hipErrorInvalidValue;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    attn_combine_kernel<<<n_heads, kBlock, 0, s>>>(part, d, n_chunks, att);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_router_logits(att, w_o, BF16, 1, n_heads * d, H, x, x, false, nullptr, s);
}

}  // namespace moe
