// prefill.hip -- MoE FFN over a prefill chunk on gfx950: the (token, rank)
// pairs are grouped by expert, then each expert's tokens run through grouped
// GEMMs on bf16 MFMA (v_mfma_f32_16x16x32_bf16, fp32 accumulation).
//
// An expert sees ~T*k/E tokens of a chunk (64 at T = 2048, k = 8, E = 256), so
// its weights are read once for all of them: this is the one place in the path
// that is a dense contraction.  Activations are rounded to bf16 as they are
// staged in LDS; int4 weights are dequantised to bf16 there.
#include "internal.h"
#include "device_common.h"

namespace moe {
namespace {

using namespace dev;

constexpr int kTileM = 64;      // pair rows per tile
constexpr int kTileN = 64;      // output columns per tile (gate/up: W_gu rows; down: output h)
constexpr int kTileK = 64;      // reduction elements staged per LDS round
constexpr int kLdsStride = 72;  // bf16 per LDS row (64 + 8 padding: 16-lane reads hit distinct banks)
constexpr int kAlignThreads = 1024;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) { return bf16_rne(lo) | (bf16_rne(hi) << 16); }

// Sixteen consecutive fp32 values of a row -> eight packed bf16 pairs.
__device__ __forceinline__ void f32x16_to_bf16(const float *p, uint4 out[2]) {
    const float4 *q = reinterpret_cast<const float4 *>(p);
    const float4 a = q[0], b = q[1], c = q[2], d = q[3];
    out[0] = make_uint4(pack_bf16(a.x, a.y), pack_bf16(a.z, a.w), pack_bf16(b.x, b.y), pack_bf16(b.z, b.w));
    out[1] = make_uint4(pack_bf16(c.x, c.y), pack_bf16(c.z, c.w), pack_bf16(d.x, d.y), pack_bf16(d.z, d.w));
}

// Sixteen consecutive weights of row r, columns col .. col+15, of a dense
// [rows x K] matrix at `m` -> eight packed bf16 pairs (bf16 copied, f32 rounded).
template <int DT>
__device__ __forceinline__ void weights16_to_bf16(const uint8_t *m, int K, int r, int col, uint4 out[2]) {
    static_assert(DT == BF16 || DT == F32, "int4 rows are dequantised by dequant16");
    if constexpr (DT == BF16) {
        const uint4 *q = reinterpret_cast<const uint4 *>(m + (size_t(r) * K + col) * 2);
        out[0] = q[0];
        out[1] = q[1];
    } else {
        f32x16_to_bf16(reinterpret_cast<const float *>(m) + size_t(r) * K + col, out);
    }
}

// Raw 16 nibbles (two dwords) times one scale -> eight packed bf16 pairs.
__device__ __forceinline__ void dequant16(uint2 nib, float s, uint4 out[2]) {
    uint32_t w[8];
#pragma unroll
    for (int d = 0; d < 2; ++d) {
        const uint32_t v = d == 0 ? nib.x : nib.y;
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
            const float lo = float(int(__builtin_amdgcn_sbfe(v, 4 * e, 4))) * s;  // builtin returns the source's (unsigned) type
            const float hi = float(int(__builtin_amdgcn_sbfe(v, 4 * e + 4, 4))) * s;
            w[d * 4 + e / 2] = pack_bf16(lo, hi);
        }
    }
    out[0] = make_uint4(w[0], w[1], w[2], w[3]);
    out[1] = make_uint4(w[4], w[5], w[6], w[7]);
}

// ------------------------------------------------------------------ align ---
// Groups: 0..E-1 routed experts, E the shared expert (all T tokens).  Output:
// hdr[0] = tiles; g_slot[g]; g_off[g] (start of group g in `sorted`);
// tiles (group, first row) of up to 64 rows; sorted pair ids (routed pair
// p = t*k + j, shared pair T*k + t).  Pairs with a bad id or no slot raise
// the flag and their partial output rows are zeroed.
__global__ __launch_bounds__(kAlignThreads) void prefill_align_kernel(const int32_t *__restrict__ ids, int T,
                                                                      int k, int E, const int32_t *__restrict__ slot_of,
                                                                      int has_shared, PrefillWorkspace ws, int H,
                                                                      int *err) {
    __shared__ int cnt[MOE_MAX_EXPERTS + 1], cur[MOE_MAX_EXPERTS + 1], off[MOE_MAX_EXPERTS + 2];
    __shared__ int slot[MOE_MAX_EXPERTS + 1];
    const int P = T * k, G = E + 1;
    for (int g = threadIdx.x; g < G; g += kAlignThreads) {
        cnt[g] = 0;
        cur[g] = 0;
        slot[g] = g == E ? -2 : (slot_of ? slot_of[g] : g);
    }
    __syncthreads();
    for (int p = threadIdx.x; p < P; p += kAlignThreads) {
        const int e = ids[p];
        const bool in = e >= 0 && e < E;
        if (!in || slot[e] < 0) {
            atomicOr(err, in ? kErrNotResident : kErrRange);
            for (int h = 0; h < H; ++h) ws.y_part[size_t(p) * H + h] = 0.f;
            continue;
        }
        atomicAdd(&cnt[e], 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        cnt[E] = has_shared ? T : 0;
        off[0] = 0;
        int nt = 0;
        for (int g = 0; g < G; ++g) {
            off[g + 1] = off[g] + cnt[g];
            for (int r0 = 0; r0 < cnt[g]; r0 += kTileM) {
                ws.tile_g[nt] = g;
                ws.tile_r0[nt] = r0;
                ++nt;
            }
        }
        ws.hdr[0] = nt;
    }
    __syncthreads();
    for (int g = threadIdx.x; g <= G; g += kAlignThreads) {
        ws.g_off[g] = off[g];
        if (g < G) ws.g_slot[g] = slot[g];
    }
    for (int p = threadIdx.x; p < P; p += kAlignThreads) {
        const int e = ids[p];
        if (e < 0 || e >= E || slot[e] < 0) continue;
        ws.sorted[off[e] + atomicAdd(&cur[e], 1)] = p;
    }
    if (has_shared)
        for (int t = threadIdx.x; t < T; t += kAlignThreads) ws.sorted[off[E] + t] = P + t;
}

// ------------------------------------------------------------ grouped GEMM ---
// One 64 x 64 output tile per block of 4 waves (2 x 2 waves of 32 x 32, each
// 2 x 2 MFMA 16x16 blocks).  Rows are pairs of one group; the A operand is
// the pair's input row (gate/up: x of its token; down: its SwiGLU activation),
// the B operand rows of the group's expert matrix.  Global loads of the next
// K round are issued before the MFMAs of the current one.
//   DOWN = false: C = x W_gu^T, epilogue act[p, i] = silu(C[:, 2i]) * C[:, 2i+1]
//   DOWN = true:  C = act W_d^T, epilogue y_part[p, h] (routed) / y_shared[t, h]
template <int DT, bool DOWN>
__global__ __launch_bounds__(kBlock) void prefill_gemm_kernel(const float *__restrict__ x, int T, int H, int I, int k,
                                                              const uint8_t *__restrict__ pool, size_t expert_bytes,
                                                              const uint8_t *__restrict__ shared_w, size_t d_off,
                                                              PrefillWorkspace ws) {
    __shared__ __align__(16) uint16_t As[kTileM * kLdsStride];
    __shared__ __align__(16) uint16_t Bs[kTileN * kLdsStride];
    __shared__ int arow[kTileM];  // pair id of each tile row (-1 = padding)
    const int tile = blockIdx.y;
    if (tile >= ws.hdr[0]) return;
    const int P = T * k;
    const int g = ws.tile_g[tile];
    const int base = ws.g_off[g] + ws.tile_r0[tile];
    const int rows = min(kTileM, ws.g_off[g + 1] - base);
    const int sl = ws.g_slot[g];
    const uint8_t *blob = sl == -2 ? shared_w : pool + size_t(sl) * expert_bytes;
    // B matrix: gate/up [2I x H] at the blob start; down [H x I] at d_off
    const int K = DOWN ? I : H;
    const uint8_t *bmat = DOWN ? blob + d_off : blob;
    const int brows = DOWN ? H : 2 * I;
    const uint16_t *bscale = reinterpret_cast<const uint16_t *>(bmat + size_t(brows) * K / 2);  // int4 only
    const int n0 = blockIdx.x * kTileN;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    if (tid < kTileM) arow[tid] = tid < rows ? ws.sorted[base + tid] : -1;
    __syncthreads();
    // staging assignment: thread -> row tid/4, 16 columns at (tid%4)*16
    const int sr = tid / 4, sc = (tid % 4) * 16;
    const int p_s = arow[sr];
    const float *arow_ptr = nullptr;
    if (p_s >= 0) {
        if (DOWN)
            arow_ptr = ws.act + size_t(p_s) * I;
        else
            arow_ptr = x + size_t(p_s < P ? p_s / k : p_s - P) * H;
    }
    uint4 ra[2], rb[2];
    uint2 rnib = make_uint2(0u, 0u);
    float rscale = 0.f;
    auto fetch = [&](int k0) {
        if (arow_ptr)
            f32x16_to_bf16(arow_ptr + k0 + sc, ra);
        else
            ra[0] = ra[1] = make_uint4(0u, 0u, 0u, 0u);
        const int br = n0 + sr;
        if constexpr (DT == INT4) {
            rnib = *reinterpret_cast<const uint2 *>(bmat + (size_t(br) * K + k0 + sc) / 2);
            rscale = bf16_bits_to_float(bscale[size_t(br) * (K / 128) + (k0 + sc) / 128]);
        } else {
            weights16_to_bf16<DT>(bmat, K, br, k0 + sc, rb);
        }
    };
    floatx4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int wm = wave / 2, wn = wave % 2;
    fetch(0);
    for (int k0 = 0; k0 < K; k0 += kTileK) {
        if constexpr (DT == INT4) dequant16(rnib, rscale, rb);
        uint4 *as = reinterpret_cast<uint4 *>(As + sr * kLdsStride + sc);
        uint4 *bs = reinterpret_cast<uint4 *>(Bs + sr * kLdsStride + sc);
        as[0] = ra[0];
        as[1] = ra[1];
        bs[0] = rb[0];
        bs[1] = rb[1];
        __syncthreads();
        if (k0 + kTileK < K) fetch(k0 + kTileK);  // next round's loads overlap the MFMAs
#pragma unroll
        for (int ks = 0; ks < kTileK; ks += 32) {
            bf16x8 a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                a[i] = *reinterpret_cast<const bf16x8 *>(As + (wm * 32 + i * 16 + lane % 16) * kLdsStride + ks + (lane / 16) * 8);
                b[i] = *reinterpret_cast<const bf16x8 *>(Bs + (wn * 32 + i * 16 + lane % 16) * kLdsStride + ks + (lane / 16) * 8);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }
    // epilogue: lane holds C[m = (lane/16)*4 + q][n = lane%16] of each 16x16 block
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int m = wm * 32 + i * 16 + (lane / 16) * 4 + q;
                const int n = n0 + wn * 32 + j * 16 + lane % 16;
                const float v = acc[i][j][q];
                const int p = arow[m];
                if constexpr (DOWN) {
                    if (p >= 0) {
                        float *o = p < P ? ws.y_part + size_t(p) * H : ws.y_shared + size_t(p - P) * H;
                        o[n] = v;
                    }
                } else {
                    // W_gu rows 2i (gate) and 2i+1 (up) sit in neighbouring lanes
                    const float partner = dpp<0xB1>(v);
                    if ((n & 1) == 0 && p >= 0) {
                        const float gte = v, up = partner;
                        ws.act[size_t(p) * I + n / 2] = gte / (1.f + expf(-gte)) * up;
                    }
                }
            }
}

template <typename... Params, typename... Args>
hipError_t launch(void (*kernel)(Params...), dim3 grid, dim3 block, size_t shmem, hipStream_t s, Args... args) {
    kernel<<<grid, block, shmem, s>>>(static_cast<Params>(args)...);
    return hipGetLastError();
}

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

int max_tiles(int T, int k, int E) { return (T * k + T + kTileM - 1) / kTileM + E + 1; }

}  // namespace

size_t prefill_workspace_bytes(int T, int k, int E, int H, int I) {
    const size_t P = size_t(T) * k, mt = size_t(max_tiles(T, k, E));
    return align256(sizeof(int) * 16) + align256(sizeof(int) * (E + 1)) + align256(sizeof(int) * (E + 2)) +
           2 * align256(sizeof(int) * mt) + align256(sizeof(int) * (P + T)) + align256(sizeof(float) * (P + T) * I) +
           align256(sizeof(float) * P * H) + align256(sizeof(float) * size_t(T) * H);
}

PrefillWorkspace prefill_workspace(void *base, int T, int k, int E, int H, int I) {
    const size_t P = size_t(T) * k, mt = size_t(max_tiles(T, k, E));
    char *c = static_cast<char *>(base);
    PrefillWorkspace w;
    auto take = [&](size_t n) {
        char *r = c;
        c += align256(n);
        return r;
    };
    w.hdr = reinterpret_cast<int *>(take(sizeof(int) * 16));
    w.g_slot = reinterpret_cast<int *>(take(sizeof(int) * (E + 1)));
    w.g_off = reinterpret_cast<int *>(take(sizeof(int) * (E + 2)));
    w.tile_g = reinterpret_cast<int *>(take(sizeof(int) * mt));
    w.tile_r0 = reinterpret_cast<int *>(take(sizeof(int) * mt));
    w.sorted = reinterpret_cast<int *>(take(sizeof(int) * (P + T)));
    w.act = reinterpret_cast<float *>(take(sizeof(float) * (P + T) * I));
    w.y_part = reinterpret_cast<float *>(take(sizeof(float) * P * H));
    w.y_shared = reinterpret_cast<float *>(take(sizeof(float) * size_t(T) * H));
    return w;
}

hipError_t launch_prefill_ffn(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                              const float *weights, const int32_t *slot_of, const void *pool, size_t expert_bytes,
                              int dtype, const void *shared_w, float *y, bool accumulate, const PrefillWorkspace &ws,
                              int *err_flags, hipStream_t s) {
    if (T == 0) return hipSuccess;
    const auto *pl = static_cast<const uint8_t *>(pool);
    const auto *sw = static_cast<const uint8_t *>(shared_w);
    const int has_shared = sw != nullptr;
    hipError_t e = launch(prefill_align_kernel, dim3(1), dim3(kAlignThreads), 0, s, ids, T, k, E, slot_of, has_shared,
                          ws, H, err_flags);
    if (e != hipSuccess) return e;
    const int mt = max_tiles(T, k, E);
    const size_t doff = down_offset(H, I, dtype);
    const dim3 g1(2 * I / kTileN, mt), g2(H / kTileN, mt);
#define PF_CASE(DT)                                                                                          \
    if (dtype == DT) {                                                                                       \
        e = launch(prefill_gemm_kernel<DT, false>, g1, dim3(kBlock), 0, s, x, T, H, I, k, pl, expert_bytes, sw, \
                   doff, ws);                                                                                \
        if (e == hipSuccess)                                                                                 \
            e = launch(prefill_gemm_kernel<DT, true>, g2, dim3(kBlock), 0, s, x, T, H, I, k, pl, expert_bytes, sw, \
                       doff, ws);                                                                            \
    }
    PF_CASE(F32) PF_CASE(BF16) PF_CASE(INT4)
#undef PF_CASE
    if (e != hipSuccess) return e;
    return launch_combine(ws.y_part, weights, has_shared ? ws.y_shared : nullptr, T, k, H, y, accumulate, s);
}

}  // namespace moe
