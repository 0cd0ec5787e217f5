// device_common.h -- device helpers shared by the library's kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/moe_budget.h"

namespace moe {
namespace dev {

constexpr int kWave = 64;
constexpr int kBlock = 256;  // 4 waves per workgroup

enum : int { F32 = MOE_F32, BF16 = MOE_BF16, INT4 = MOE_INT4G128 };

// Elements held by one 16-byte chunk, and bytes per element of the dense types.
template <int DT> struct Fmt;
template <> struct Fmt<F32> { static constexpr int EPC = 4; };
template <> struct Fmt<BF16> { static constexpr int EPC = 8; };
template <> struct Fmt<INT4> { static constexpr int EPC = 32; };

__host__ __device__ constexpr size_t row_bytes_of(int DT, int cols) {
    return DT == INT4 ? size_t(cols) / 2 : size_t(cols) * (DT == F32 ? 4 : 2);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the 64 lanes, returned in every lane: DPP quad swaps (xor 1, xor 2),
// half-row and row mirrors give each 16-lane row its total; four readlanes add the rows.
__device__ __forceinline__ float wave_sum(float v) {
    v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp<0x141>(v);  // row_half_mirror
    v += dpp<0x140>(v);  // row_mirror
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0)) +
           __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16)) +
           __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32)) +
           __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
}

// Maximum (MAX) or minimum of a 32-bit unsigned value over the 64 lanes, returned in every lane (the same
// DPP pattern as wave_reduce_u64 below).
template <bool MAX>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v) {
    auto pick = [](uint32_t a, uint32_t b) { return MAX ? (b > a ? b : a) : (b < a ? b : a); };
#define MOE_DPP32(CTRL, ROWS) uint32_t(__builtin_amdgcn_update_dpp(int(v), int(v), CTRL, ROWS, 0xF, false))
    v = pick(v, MOE_DPP32(0xB1, 0xF));
    v = pick(v, MOE_DPP32(0x4E, 0xF));
    v = pick(v, MOE_DPP32(0x141, 0xF));
    v = pick(v, MOE_DPP32(0x140, 0xF));
    v = pick(v, MOE_DPP32(0x142, 0xA));
    v = pick(v, MOE_DPP32(0x143, 0xC));
#undef MOE_DPP32
    return uint32_t(__builtin_amdgcn_readlane(int(v), 63));
}

// Maximum (MAX) or minimum of a 64-bit value over the 64 lanes, returned in every lane: DPP quad swaps and
// half-row / row mirrors reduce each row of 16; row broadcasts 15 and 31 carry the rows' results to lane 63.
template <bool MAX>
__device__ __forceinline__ uint64_t wave_reduce_u64(uint64_t v) {
    auto pick = [](uint64_t a, uint64_t b) { return MAX ? (b > a ? b : a) : (b < a ? b : a); };
    auto lo = [](uint64_t a) { return int(uint32_t(a)); };
    auto hi = [](uint64_t a) { return int(uint32_t(a >> 32)); };
    auto join = [](int l, int h) { return uint64_t(uint32_t(l)) | (uint64_t(uint32_t(h)) << 32); };
#define MOE_DPP64(CTRL, ROWS) \
    join(__builtin_amdgcn_update_dpp(lo(v), lo(v), CTRL, ROWS, 0xF, false), \
         __builtin_amdgcn_update_dpp(hi(v), hi(v), CTRL, ROWS, 0xF, false))
    v = pick(v, MOE_DPP64(0xB1, 0xF));   // quad_perm [1,0,3,2]
    v = pick(v, MOE_DPP64(0x4E, 0xF));   // quad_perm [2,3,0,1]
    v = pick(v, MOE_DPP64(0x141, 0xF));  // row_half_mirror
    v = pick(v, MOE_DPP64(0x140, 0xF));  // row_mirror
    v = pick(v, MOE_DPP64(0x142, 0xA));  // row_bcast:15 into rows 1 and 3
    v = pick(v, MOE_DPP64(0x143, 0xC));  // row_bcast:31 into rows 2 and 3
#undef MOE_DPP64
    return join(__builtin_amdgcn_readlane(lo(v), 63), __builtin_amdgcn_readlane(hi(v), 63));
}

__device__ __forceinline__ float bf16_bits_to_float(uint32_t b16) { return __uint_as_float(b16 << 16); }

__device__ __forceinline__ uint4 load16(const uint8_t *p) { return *reinterpret_cast<const uint4 *>(p); }

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load with the nontemporal hint, for expert weights that are read once
// per call: a streamed read of tens of MB then does not displace what the next
// kernels reuse, and reaches a higher fraction of HBM bandwidth.
// A word that an earlier kernel on the stream wrote, loaded through a vector register even when the address is
// uniform: the pointer passes through an empty asm (in the global address space, so the load stays a global
// load), which keeps the compiler from issuing it through the scalar cache.
__device__ __forceinline__ int load_stream_word(const int32_t *p) {
    typedef const __attribute__((address_space(1))) int32_t gword;
    gword *q = (gword *)p;
    asm volatile("" : "+v"(q));
    return *q;
}

// One float4 read as a native vector (a float4 copied as an aggregate can end up in private memory).
__device__ __forceinline__ float4 load_f4(const float4 *p) {
    const u32x4 v = *reinterpret_cast<const u32x4 *>(p);
    return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
}

__device__ __forceinline__ uint4 load16_stream(const uint8_t *p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

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
                const int q = int(__builtin_amdgcn_sbfe(d[i], 4 * e, 4));  // signed nibble e, low nibble first
                acc = fmaf(float(q), xv[8 * i + e], acc);
            }
    }
    return acc;
}

// ---- int4 x fp16 dot products (the one-token int4 kernels) ----
// The activations of a 32-element chunk (one lane's 16 bytes of nibbles) are held as fp16 pairs, scaled by
// a power of two 2^sh that puts the chunk's largest magnitude in [2^13, 2^14): fp16 then keeps 11
// significant bits of every element (elements below 2^-27 of the chunk's largest become subnormal), and
// no element can overflow.  Dword i of the chunk (elements 8i .. 8i+7, nibble e at bits 4e) pairs with
// the 16-byte word {(x0, x4), (x1, x5), (x2, x6), (x3, x7)} of those elements.
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ half2_t as_half2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }

// A signed nibble q becomes the fp16 value bias + q with one three-input bit operation: its sign bit is
// flipped (q + 8 as an unsigned nibble) and the result is dropped into the mantissa of 1024 (nibble at
// bits 0-3 of a half: 1024 + q + 8) or of 64 (bits 4-7, sixteen times the weight of a mantissa step:
// 64 + q + 8).  So every nibble is exact, and the sum carries sum_x (1032 x) over the elements at even
// nibble positions and sum_x (72 x) over the odd ones: stage8_i4h forms that bias term for the chunk when
// it stages the activations, and the caller subtracts it once per chunk and row.
constexpr uint32_t kNibLo = 0x000F000Fu, kMagicLo = 0x64086408u;  // 1024 + (q ^ 8) per half
constexpr uint32_t kNibHi = 0x00F000F0u, kMagicHi = 0x54805480u;  // 64 + (q ^ 8) per half
constexpr float kBiasLo = 1032.f, kBiasHi = 72.f;

// sum of (q + bias) * x over the eight nibbles of d, added to acc (x pairs as above).
__device__ __forceinline__ float dot8_i4h(uint32_t d, uint4 xq, float acc) {
    const uint32_t t = d >> 8;
    acc = __builtin_amdgcn_fdot2(as_half2((d & kNibLo) ^ kMagicLo), as_half2(xq.x), acc, false);
    acc = __builtin_amdgcn_fdot2(as_half2((d & kNibHi) ^ kMagicHi), as_half2(xq.y), acc, false);
    acc = __builtin_amdgcn_fdot2(as_half2((t & kNibLo) ^ kMagicLo), as_half2(xq.z), acc, false);
    acc = __builtin_amdgcn_fdot2(as_half2((t & kNibHi) ^ kMagicHi), as_half2(xq.w), acc, false);
    return acc;
}

// One 16-byte chunk of 32 nibbles against its four words of fp16 pairs: sum of (q + bias) * x.
__device__ __forceinline__ float chunk_dot_i4h(uint4 w, const uint4 *xq) {
    float acc = dot8_i4h(w.x, xq[0], 0.f);
    acc = dot8_i4h(w.y, xq[1], acc);
    acc = dot8_i4h(w.z, xq[2], acc);
    return dot8_i4h(w.w, xq[3], acc);
}

// The staging side, run by the four consecutive lanes (a quad) that hold one chunk's four dwords of
// activations, v[0..7] each: returns this lane's word of fp16 pairs; sh_out gets the chunk's exponent
// shift (the dot's result is scaled back by 2^-sh) and bias_out the chunk's bias term (same in the four
// lanes).  Every lane of the wave must call it (quad DPP exchanges).
__device__ __forceinline__ uint4 stage8_i4h(const float *v, int &sh_out, float &bias_out) {
    float m = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(v[e]));
    m = fmaxf(m, dpp<0xB1>(m));  // quad_perm [1,0,3,2]
    m = fmaxf(m, dpp<0x4E>(m));  // quad_perm [2,3,0,1]
    int ex;
    (void)frexpf(m, &ex);  // m = f * 2^ex, f in [0.5, 1) (ex = 0 for m = 0)
    const int sh = 14 - ex;
    uint32_t p[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const half2_t h = {(_Float16)ldexpf(v[e], sh), (_Float16)ldexpf(v[e + 4], sh)};
        p[e] = __builtin_bit_cast(uint32_t, h);
    }
    const half2_t lo = {(_Float16)kBiasLo, (_Float16)kBiasLo}, hi = {(_Float16)kBiasHi, (_Float16)kBiasHi};
    float b = __builtin_amdgcn_fdot2(as_half2(p[0]), lo, 0.f, false);
    b = __builtin_amdgcn_fdot2(as_half2(p[1]), hi, b, false);
    b = __builtin_amdgcn_fdot2(as_half2(p[2]), lo, b, false);
    b = __builtin_amdgcn_fdot2(as_half2(p[3]), hi, b, false);
    b += dpp<0xB1>(b);
    b += dpp<0x4E>(b);
    sh_out = sh;
    bias_out = b;
    return make_uint4(p[0], p[1], p[2], p[3]);
}

}  // namespace dev
}  // namespace moe
