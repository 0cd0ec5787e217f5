// prefill.hip -- MoE FFN over a prefill chunk on gfx950: the (token, rank)
// pairs are grouped by expert, then each expert's rows run through grouped
// GEMMs on bf16 MFMA (v_mfma_f32_16x16x32_bf16, fp32 accumulation).
//
// An expert sees ~T*k/E rows of a chunk (64 at T = 2048, k = 8, E = 256), so
// its weights are read once for all of them: this is the one place in the path
// that is a dense contraction.  Layout of the work:
//   plan    one block groups the pairs by expert (histogram, scan, 64-row
//           tiles, scatter); the other blocks round x to bf16 once.
//   gate/up C = x W_gu^T per 64 x 256 tile; the epilogue writes the bf16
//           SwiGLU activation in grouped row order.
//   down    C = act W_d^T per 64 x 256 tile; one fp32 output row per pair.
//   combine each token's rows summed in rank order with its weights.
// In both GEMMs the A rows (activations, shared by the block's four waves)
// are staged through double-buffered LDS, while each wave loads its own 64
// weight rows straight into registers in the matrix-core lane layout and
// dequantises int4 there: a weight is used by exactly one wave, so staging it
// in LDS would only add traffic.
#include "internal.h"
#include "device_common.h"

#include <algorithm>
#include <type_traits>

namespace moe {
namespace {

using namespace dev;

constexpr int kTileM = 64;        // pair rows per tile
constexpr int kWaveN = 64;        // output columns per wave
constexpr int kTileN = 4 * kWaveN;  // output columns per block
constexpr int kPlanThreads = 1024;
constexpr int kXcds = 8;          // gfx950 dispatches consecutive workgroups round-robin over 8 XCDs

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Two floats -> packed bf16 pair (round to nearest even; one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{lo, hi}, bf16x2));
}

// int4 -> bf16 with the offset form used by the grouped GEMM: for the eight
// nibbles of one dword (element e in bits 4e..4e+3, two's complement q), the
// bf16 pattern 0x4300 | (r ^ 8) is exactly 128 + (q + 8) = 136 + q.  Two bit
// operations give a pair: ((v >> 4e) & 0x000F000F) ^ 0x43084308 holds elements
// e and e + 4, so the eight values come out in the order 0,4,1,5,2,6,3,7 (the
// A operand is stored in the same order).  The scale and the -136 offset are
// applied to the fp32 MFMA result of the whole quantisation group.
__device__ __forceinline__ bf16x8 int4_offset8(uint32_t v) {
    const uint32_t w0 = v & 0x000F000Fu, w1 = (v >> 4) & 0x000F000Fu, w2 = (v >> 8) & 0x000F000Fu,
                   w3 = (v >> 12) & 0x000F000Fu;
    return __builtin_bit_cast(bf16x8, make_uint4(w0 ^ 0x43084308u, w1 ^ 0x43084308u, w2 ^ 0x43084308u,
                                                 w3 ^ 0x43084308u));
}

// Position of element e (0..7) of an 8-element group in the order 0,4,1,5,2,6,3,7.
__device__ __forceinline__ int perm8_pos(int e) { return e < 4 ? 2 * e : 2 * e - 7; }

// ------------------------------------------------------------------- plan ---
// Groups: 0..E-1 routed experts, E the shared expert (all T tokens).  Output:
// hdr[0] = tiles; g_slot[g]; g_off[g] (start of group g in `sorted`); tiles
// (group, first row) of up to 64 rows; sorted pair ids (routed pair p = t*k+j,
// shared pair T*k + t).  Pairs with a bad id or no slot raise the flag and
// their output rows are zeroed.  Blocks 1.. write xb = bf16(x).
__global__ __launch_bounds__(kPlanThreads) void prefill_plan_kernel(const int32_t *__restrict__ ids, int T, int k,
                                                                    int E, const int32_t *__restrict__ slot_of,
                                                                    int has_shared, const float *__restrict__ x,
                                                                    int H, int offset_form, PrefillWorkspace ws,
                                                                    int *err) {
    if (blockIdx.x > 0) {
        // 8 elements per thread; 16 consecutive threads hold one 128-element group (H % 128 == 0)
        const size_t n8 = size_t(T) * H / 8;
        const size_t stride = size_t(gridDim.x - 1) * kPlanThreads;
        for (size_t i = size_t(blockIdx.x - 1) * kPlanThreads + threadIdx.x; i < n8; i += stride) {
            const float4 a = reinterpret_cast<const float4 *>(x)[2 * i];
            const float4 b = reinterpret_cast<const float4 *>(x)[2 * i + 1];
            if (offset_form) {
                const uint32_t p0 = pack2(a.x, b.x), p1 = pack2(a.y, b.y), p2 = pack2(a.z, b.z), p3 = pack2(a.w, b.w);
                reinterpret_cast<uint4 *>(ws.xb)[i] = make_uint4(p0, p1, p2, p3);
                // group sum of the bf16 values the matrix cores see
                float sum = 0.f;
                const uint32_t pk[4] = {p0, p1, p2, p3};
#pragma unroll
                for (int e = 0; e < 4; ++e) sum += __uint_as_float(pk[e] << 16) + __uint_as_float(pk[e] & 0xffff0000u);
#pragma unroll
                for (int d = 1; d < 16; d <<= 1) sum += __shfl_xor(sum, d);
                if ((threadIdx.x & 15) == 0) ws.sx[i / 16] = sum;
            } else {
                reinterpret_cast<uint4 *>(ws.xb)[i] =
                    make_uint4(pack2(a.x, a.y), pack2(a.z, a.w), pack2(b.x, b.y), pack2(b.z, b.w));
            }
        }
        return;
    }
    __shared__ int cnt[MOE_MAX_EXPERTS + 1], cur[MOE_MAX_EXPERTS + 1], slot[MOE_MAX_EXPERTS + 1];
    __shared__ int off[MOE_MAX_EXPERTS + 2], toff[MOE_MAX_EXPERTS + 2];
    const int P = T * k, G = E + 1, tid = threadIdx.x;
    for (int g = tid; g < G; g += kPlanThreads) {
        cnt[g] = 0;
        cur[g] = 0;
        slot[g] = g == E ? -2 : (slot_of ? slot_of[g] : g);
    }
    __syncthreads();
    for (int p = tid; p < P; p += kPlanThreads) {
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
    if (tid == 0) cnt[E] = has_shared ? T : 0;
    __syncthreads();
    // exclusive scans of the group sizes and of their tile counts, by wave 0 in chunks of 64
    if (tid < kWave) {
        int carry = 0, tcarry = 0;
        for (int g0 = 0; g0 < G; g0 += kWave) {
            const int g = g0 + tid;
            const int c = g < G ? cnt[g] : 0;
            int v = c, tv = (c + kTileM - 1) / kTileM;
            const int c_t = tv;
            for (int d = 1; d < kWave; d <<= 1) {
                const int y = __shfl_up(v, d), ty = __shfl_up(tv, d);
                if (tid >= d) {
                    v += y;
                    tv += ty;
                }
            }
            if (g < G) {
                off[g] = carry + v - c;
                toff[g] = tcarry + tv - c_t;
            }
            carry += __shfl(v, kWave - 1);
            tcarry += __shfl(tv, kWave - 1);
        }
        if (tid == 0) {
            off[G] = carry;
            toff[G] = tcarry;
            ws.hdr[0] = tcarry;
        }
    }
    __syncthreads();
    for (int g = tid; g <= G; g += kPlanThreads) {
        ws.g_off[g] = off[g];
        if (g < G) {
            ws.g_slot[g] = slot[g];
            for (int i = 0, t = toff[g]; t < toff[g + 1]; ++i, ++t) {
                ws.tile_g[t] = g;
                ws.tile_r0[t] = i * kTileM;
            }
        }
    }
    for (int p = tid; p < P; p += kPlanThreads) {
        const int e = ids[p];
        if (e < 0 || e >= E || slot[e] < 0) continue;
        ws.sorted[off[e] + atomicAdd(&cur[e], 1)] = p;
    }
    if (has_shared)
        for (int t = tid; t < T; t += kPlanThreads) ws.sorted[off[E] + t] = P + t;
}

// ------------------------------------------------------------ grouped GEMM ---
// Reduction depth per round: int4 takes one quantisation group (128), so a
// column's weights of a round share one scale; bf16 takes 64.  Lane l of a
// wave owns output column (l % 16) of each of its four 16-column blocks and the
// k range [SEG*(l/16), SEG*(l/16) + SEG) of the round; MFMA step s uses the
// eight k at offset 8s of that range, from A and B alike.
template <int DT>
struct Round {
    static constexpr int BK = DT == INT4 ? 128 : 64;
    static constexpr int SEG = BK / 4;        // k per lane group, and per staging thread of A
    static constexpr int STEPS = BK / 32;     // MFMA k-steps per round
    static constexpr int LDS = BK + 8;        // bf16 per LDS row: 16 rows read at one offset hit distinct banks
    static constexpr int A16 = SEG / 8;       // 16-byte A loads per staging thread
    static constexpr int B16 = DT == INT4 ? 1 : SEG / 8;  // 16-byte weight loads per lane and column block
};

// int4: per round, tmp = A (136 + Q)^T on the matrix cores, then
//   acc += s_n * (tmp - 136 * S_m)
// with s_n the column's scale and S_m the row's sum of A over the group (read
// from ws.sx for x, ws.sa for the activations).  bf16: acc += A W^T directly.
template <int DT, bool DOWN>
__global__ __launch_bounds__(kBlock, 2) void prefill_gemm_kernel(int T, int H, int I, int k,
                                                              const uint8_t *__restrict__ pool, size_t expert_bytes,
                                                              const uint8_t *__restrict__ shared_w, size_t d_off,
                                                              int nblk_n, PrefillWorkspace ws) {
    using R = Round<DT>;
    constexpr bool kOffset = DT == INT4;
    __shared__ __align__(16) uint16_t As[2][kTileM * R::LDS];
    __shared__ __align__(16) float Ss[2][kTileM];  // int4: group sums of the tile rows
    __shared__ float Sred[4][kTileM];              // int4 gate/up epilogue: per-wave activation sums
    __shared__ int arow[kTileM];                   // pair id of each tile row (-1 = padding)
    // XCD-aware order: the blocks of one tile (and neighbouring tiles of a group) share an XCD's L2
    const int nwork = ws.hdr[0] * nblk_n;
    const int chunk = (nwork + kXcds - 1) / kXcds;
    const int idx = blockIdx.x / kXcds;
    if (idx >= chunk) return;
    const int work = (blockIdx.x % kXcds) * chunk + idx;
    if (work >= nwork) return;
    const int tile = work / nblk_n, nb = work % nblk_n;

    const int P = T * k;
    const int g = ws.tile_g[tile];
    const int base = ws.g_off[g] + ws.tile_r0[tile];
    const int rows = min(kTileM, ws.g_off[g + 1] - base);
    const int sl = ws.g_slot[g];
    const uint8_t *blob = sl == -2 ? shared_w : pool + size_t(sl) * expert_bytes;
    const int K = DOWN ? I : H, N = DOWN ? H : 2 * I;
    const int KG = K / 128;                            // quantisation groups per row
    const uint8_t *bmat = DOWN ? blob + d_off : blob;  // gate/up [2I x H] at the blob start, down [H x I]
    const uint16_t *bscale = reinterpret_cast<const uint16_t *>(bmat + size_t(N) * K / 2);  // int4 only
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int lr = lane % 16, lg = lane / 16;
    const int wn0 = nb * kTileN + wave * kWaveN;
    const bool active = wn0 < N;  // N is a multiple of 64: a wave's columns are all in range or all out
    // The main loop has no branches: padding rows load row 0 of the tile and an out-of-range wave
    // loads weight row N-1; neither result is stored.  (A branch around a load leaves the compiler
    // unable to count outstanding loads, and it then waits for all of them.)

    if (tid < kTileM) arow[tid] = tid < rows ? ws.sorted[base + tid] : -1;
    __syncthreads();

    // A staging: thread -> row tid / 4, SEG columns at (tid % 4) * SEG of each round
    const int sr = tid / 4, sc = (tid % 4) * R::SEG;
    const int ar = sr < rows ? sr : 0;
    const uint16_t *asrc;
    if constexpr (DOWN) {
        asrc = ws.act + size_t(base + ar) * I;
    } else {
        const int p = arow[ar];
        asrc = ws.xb + size_t(p < P ? p / k : p - P) * H;
    }
    // group sums: thread tid < 64 stages row tid's sum of the next round
    const float *ssrc = nullptr;
    if constexpr (kOffset) {
        const int rr = tid < rows ? tid : 0;
        if constexpr (DOWN) {
            ssrc = ws.sa + size_t(base + rr) * KG;
        } else {
            const int p = arow[tid < kTileM ? rr : 0];
            ssrc = ws.sx + size_t(p < P ? p / k : p - P) * KG;
        }
    }

    // The main loop and the epilogue are instantiated for 1..4 live 16-row blocks: 16-row blocks that
    // are all padding take no MFMA, A read or fold (a group of 70 rows has a second tile of 6 rows).
    auto body = [&](auto mb_tag) __attribute__((always_inline)) {
        constexpr int MB = decltype(mb_tag)::value;
        floatx4 acc[MB][4];
    #pragma unroll
        for (int i = 0; i < MB; ++i)
    #pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

        u32x4 ra[R::A16];       // next round's A segment of this thread
        uint4 rb[4][R::B16];    // next round's weights of this lane, one entry per 16-column block
        uint32_t rsb[4] = {0u, 0u, 0u, 0u};  // their raw bf16 scale bits (widened at use: no wait after the load)
        float rS = 0.f;         // next round's group sum of row tid (int4, tid < 64)
        // 32-bit byte offsets of this lane's weight rows (and scale rows) within the expert matrix
        uint32_t boff[4], soff[4];
    #pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t n = uint32_t(min(wn0 + 16 * j + lr, N - 1));
            boff[j] = DT == INT4 ? n * uint32_t(K / 2) + uint32_t(R::SEG * lg / 2) : (n * uint32_t(K) + uint32_t(R::SEG * lg)) * 2u;
            soff[j] = n * uint32_t(KG);
        }
        const int rounds = K / R::BK;
        // Software pipeline: iteration r issues round r+1's loads, multiplies round r out of LDS and
        // registers, then stores round r+1's A into the other LDS buffer.
        for (int r = -1; r < rounds; ++r) {
            uint4 cb[4][R::B16];
            float cs[4];
    #pragma unroll
            for (int j = 0; j < 4; ++j) {
                cs[j] = bf16_bits_to_float(rsb[j]);
    #pragma unroll
                for (int i = 0; i < R::B16; ++i) cb[j][i] = rb[j][i];
            }
            if (r + 1 < rounds) {
                const int k0 = (r + 1) * R::BK;
    #pragma unroll
                for (int i = 0; i < R::A16; ++i) ra[i] = *reinterpret_cast<const u32x4 *>(asrc + k0 + sc + 8 * i);
                if constexpr (kOffset) {
                    if (tid < kTileM) rS = ssrc[r + 1];
                }
    #pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if constexpr (DT == INT4) {
                        rb[j][0] = *reinterpret_cast<const uint4 *>(bmat + boff[j] + uint32_t(k0 / 2));
                        rsb[j] = bscale[soff[j] + uint32_t(k0 / 128)];
                    } else {
    #pragma unroll
                        for (int i = 0; i < R::B16; ++i)
                            rb[j][i] = *reinterpret_cast<const uint4 *>(bmat + boff[j] + uint32_t(k0 * 2 + 16 * i));
                    }
                }
            }
            if (r >= 0) {
                const int buf = r & 1;
                floatx4 tmp[MB][4];
    #pragma unroll
                for (int s = 0; s < R::STEPS; ++s) {
                    bf16x8 a[MB];
    #pragma unroll
                    for (int i = 0; i < MB; ++i)
                        a[i] = *reinterpret_cast<const bf16x8 *>(&As[buf][(16 * i + lr) * R::LDS + R::SEG * lg + 8 * s]);
    #pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if constexpr (kOffset) {
                            const uint32_t d = s == 0 ? cb[j][0].x : s == 1 ? cb[j][0].y : s == 2 ? cb[j][0].z : cb[j][0].w;
                            const bf16x8 b = int4_offset8(d);
    #pragma unroll
                            for (int i = 0; i < MB; ++i)
                                tmp[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    a[i], b, s == 0 ? floatx4{0.f, 0.f, 0.f, 0.f} : tmp[i][j], 0, 0, 0);
                        } else {
                            const bf16x8 b = __builtin_bit_cast(bf16x8, cb[j][s]);
    #pragma unroll
                            for (int i = 0; i < MB; ++i)
                                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b, acc[i][j], 0, 0, 0);
                        }
                    }
                }
                if constexpr (kOffset) {
                    // rows of this lane: m = 16i + 4lg + q
    #pragma unroll
                    for (int i = 0; i < MB; ++i) {
                        const float4 sv = *reinterpret_cast<const float4 *>(&Ss[buf][16 * i + 4 * lg]);
                        const float svq[4] = {sv.x, sv.y, sv.z, sv.w};
    #pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const float off = -136.f * cs[j];
    #pragma unroll
                            for (int q = 0; q < 4; ++q) acc[i][j][q] = fmaf(cs[j], tmp[i][j][q], fmaf(off, svq[q], acc[i][j][q]));
                        }
                    }
                }
            }
            if (r + 1 < rounds) {
                u32x4 *dst = reinterpret_cast<u32x4 *>(&As[(r + 1) & 1][sr * R::LDS + sc]);
    #pragma unroll
                for (int i = 0; i < R::A16; ++i) dst[i] = ra[i];
                if constexpr (kOffset) {
                    if (tid < kTileM) Ss[(r + 1) & 1][tid] = rS;
                }
            }
            __syncthreads();
        }

        // epilogue: lane holds C[m = 16i + 4*lg + q][n = wn0 + 16j + lr]
        float rowsum[MB][4];  // int4 gate/up: this lane's bf16 activations summed per row
    #pragma unroll
        for (int i = 0; i < MB; ++i)
    #pragma unroll
            for (int q = 0; q < 4; ++q) {
                rowsum[i][q] = 0.f;
                const int m = 16 * i + 4 * lg + q;
                const int p = arow[m];
    #pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int n = wn0 + 16 * j + lr;
                    const float v = acc[i][j][q];
                    if constexpr (DOWN) {
                        if (active && p >= 0) {
                            float *o = p < P ? ws.y_part + size_t(p) * H : ws.y_shared + size_t(p - P) * H;
                            o[n] = v;
                        }
                    } else {
                        // W_gu rows 2i (gate) and 2i+1 (up) sit in neighbouring lanes
                        const float partner = dpp<0xB1>(v);
                        if ((lr & 1) == 0 && active && p >= 0) {
                            const float a = v * __builtin_amdgcn_rcpf(1.f + __expf(-v)) * partner;
                            const uint32_t ab = pack2(a, 0.f) & 0xffffu;
                            const int c = n / 2;
                            const int pos = kOffset ? (c & ~7) + perm8_pos(c & 7) : c;
                            ws.act[size_t(base + m) * I + pos] = uint16_t(ab);
                            rowsum[i][q] += __uint_as_float(ab << 16);
                        }
                    }
                }
            }
        if constexpr (kOffset && !DOWN) {
            // group sums of the activations for the down GEMM: this block's 256 gate/up columns are
            // the 128 activation columns of down group nb
    #pragma unroll
            for (int i = 0; i < MB; ++i)
    #pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float v = rowsum[i][q];
                    v += __shfl_xor(v, 1);
                    v += __shfl_xor(v, 2);
                    v += __shfl_xor(v, 4);
                    v += __shfl_xor(v, 8);
                    if (lr == 0) Sred[wave][16 * i + 4 * lg + q] = v;
                }
            __syncthreads();
            if (tid < rows) ws.sa[size_t(base + tid) * (I / 128) + nb] = Sred[0][tid] + Sred[1][tid] + Sred[2][tid] + Sred[3][tid];
        }
    };
    switch ((rows + 15) / 16) {
        case 1: body(std::integral_constant<int, 1>{}); break;
        case 2: body(std::integral_constant<int, 2>{}); break;
        case 3: body(std::integral_constant<int, 3>{}); break;
        default: body(std::integral_constant<int, 4>{}); break;
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

bool prefill_dtype_supported(int dtype) { return dtype == BF16 || dtype == INT4; }

size_t prefill_workspace_bytes(int T, int k, int E, int H, int I) {
    const size_t P = size_t(T) * k, R = P + T, mt = size_t(max_tiles(T, k, E));
    return align256(sizeof(int) * 16) + align256(sizeof(int) * (E + 1)) + align256(sizeof(int) * (E + 2)) +
           2 * align256(sizeof(int) * mt) + align256(sizeof(int) * R) + align256(2 * size_t(T) * H) +
           align256(2 * R * I) + align256(sizeof(float) * P * H) + align256(sizeof(float) * size_t(T) * H) +
           align256(sizeof(float) * size_t(T) * (H / 128)) + align256(sizeof(float) * R * (I / 128));
}

PrefillWorkspace prefill_workspace(void *base, int T, int k, int E, int H, int I) {
    const size_t P = size_t(T) * k, R = P + T, mt = size_t(max_tiles(T, k, E));
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
    w.sorted = reinterpret_cast<int *>(take(sizeof(int) * R));
    w.xb = reinterpret_cast<uint16_t *>(take(2 * size_t(T) * H));
    w.act = reinterpret_cast<uint16_t *>(take(2 * R * I));
    w.y_part = reinterpret_cast<float *>(take(sizeof(float) * P * H));
    w.y_shared = reinterpret_cast<float *>(take(sizeof(float) * size_t(T) * H));
    w.sx = reinterpret_cast<float *>(take(sizeof(float) * size_t(T) * (H / 128)));
    w.sa = reinterpret_cast<float *>(take(sizeof(float) * R * (I / 128)));
    return w;
}

hipError_t launch_prefill_ffn(const float *x, int T, int H, int I, int E, int k, const int32_t *ids,
                              const float *weights, const int32_t *slot_of, const void *pool, size_t expert_bytes,
                              int dtype, const void *shared_w, float *y, bool accumulate, const PrefillWorkspace &ws,
                              int *err_flags, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (!prefill_dtype_supported(dtype)) return hipErrorInvalidValue;
    const auto *pl = static_cast<const uint8_t *>(pool);
    const auto *sw = static_cast<const uint8_t *>(shared_w);
    const int has_shared = sw != nullptr;
    const size_t n8 = size_t(T) * H / 8;
    const size_t cvt_blocks = std::min<size_t>(1024, (n8 + kPlanThreads - 1) / kPlanThreads);
    hipError_t e = launch(prefill_plan_kernel, dim3(unsigned(1 + cvt_blocks)), dim3(kPlanThreads), 0, s, ids, T, k,
                          E, slot_of, has_shared, x, H, dtype == INT4 ? 1 : 0, ws, err_flags);
    if (e != hipSuccess) return e;
    const int mt = max_tiles(T, k, E);
    const int nb1 = (2 * I + kTileN - 1) / kTileN, nb2 = (H + kTileN - 1) / kTileN;
    const size_t doff = down_offset(H, I, dtype);
    // grids rounded up to whole XCD rounds: the block -> work map needs 8 * ceil(work / 8) blocks
    const unsigned g1 = unsigned((mt * nb1 + kXcds - 1) / kXcds * kXcds), g2 = unsigned((mt * nb2 + kXcds - 1) / kXcds * kXcds);
    if (dtype == INT4) {
        e = launch(prefill_gemm_kernel<INT4, false>, dim3(g1), dim3(kBlock), 0, s, T, H, I, k, pl,
                   expert_bytes, sw, doff, nb1, ws);
        if (e == hipSuccess)
            e = launch(prefill_gemm_kernel<INT4, true>, dim3(g2), dim3(kBlock), 0, s, T, H, I, k, pl,
                       expert_bytes, sw, doff, nb2, ws);
    } else {
        e = launch(prefill_gemm_kernel<BF16, false>, dim3(g1), dim3(kBlock), 0, s, T, H, I, k, pl,
                   expert_bytes, sw, doff, nb1, ws);
        if (e == hipSuccess)
            e = launch(prefill_gemm_kernel<BF16, true>, dim3(g2), dim3(kBlock), 0, s, T, H, I, k, pl,
                       expert_bytes, sw, doff, nb2, ws);
    }
    if (e != hipSuccess) return e;
    return launch_combine(ws.y_part, weights, has_shared ? ws.y_shared : nullptr, T, k, H, y, accumulate, s);
}

}  // namespace moe
