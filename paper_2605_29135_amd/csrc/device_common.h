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


}  // namespace dev
}  // namespace moe
