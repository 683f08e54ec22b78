// Shared device helpers for the libpresto kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "presto.h"

namespace presto {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Orderable encodings.  ord32(x) is monotone in x as an unsigned integer,
// with -0.0 mapped onto +0.0; NaN patterns never come out of valid inputs.

__device__ __forceinline__ uint32_t ord32(float x) {
    uint32_t u = __float_as_uint(x);
    u = (u == 0x80000000u) ? 0u : u;  // -0.0 == +0.0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float unord32(uint32_t o) {
    uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
    return __uint_as_float(u);
}

// Candidate key: larger key = larger value, then lower id.
__device__ __forceinline__ uint64_t vocab_key(float x, uint32_t id) {
    return ((uint64_t)ord32(x) << 32) | (uint64_t)(0xffffffffu - id);
}
__device__ __forceinline__ uint32_t key_id(uint64_t k) { return 0xffffffffu - (uint32_t)k; }
__device__ __forceinline__ float key_value(uint64_t k) { return unord32((uint32_t)(k >> 32)); }

// bf16 <-> fp32 on raw bit patterns.
__device__ __forceinline__ float bf16lo(uint32_t packed) { return __uint_as_float(packed << 16); }
__device__ __forceinline__ float bf16hi(uint32_t packed) { return __uint_as_float(packed & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ uint16_t f_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// 16-byte streaming load (read once: do not keep in the caches).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream16(const void* p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v[0], v[1], v[2], v[3]);
}

// ---------------------------------------------------------------------------
// Wave-wide reductions (butterfly: every lane ends with the result).

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        uint32_t w = __shfl_xor(v, o, kWave);
        v = w > v ? w : v;
    }
    return v;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
    uint32_t lo = __shfl_xor((uint32_t)v, o, kWave);
    uint32_t hi = __shfl_xor((uint32_t)(v >> 32), o, kWave);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        uint64_t w = shfl_xor_u64(v, o);
        v = w > v ? w : v;
    }
    return v;
}

__device__ __forceinline__ int wave_sum_i32(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// ---------------------------------------------------------------------------
// DPP reductions (no LDS traffic).  `old` is the identity, returned by lanes
// whose DPP source is out of range or masked off.
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROW_MASK, 0xf, false);
}

// Unsigned max over the whole wave (result returned to every lane).
__device__ __forceinline__ uint32_t wave_max_u32_dpp(uint32_t v) {
    v = max(v, dpp_u32<0xb1>(0u, v));        // quad_perm [1,0,3,2]
    v = max(v, dpp_u32<0x4e>(0u, v));        // quad_perm [2,3,0,1]
    v = max(v, dpp_u32<0x114>(0u, v));       // row_shr:4
    v = max(v, dpp_u32<0x118>(0u, v));       // row_shr:8
    v = max(v, dpp_u32<0x142, 0xa>(0u, v));  // row_bcast:15
    v = max(v, dpp_u32<0x143, 0xc>(0u, v));  // row_bcast:31
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t old, uint64_t v) {
    const uint32_t lo = dpp_u32<CTRL, ROW_MASK>((uint32_t)old, (uint32_t)v);
    const uint32_t hi = dpp_u32<CTRL, ROW_MASK>((uint32_t)(old >> 32), (uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ float dpp_f32(float old, float v) {
    return __uint_as_float(dpp_u32<CTRL, ROW_MASK>(__float_as_uint(old), __float_as_uint(v)));
}

// Float max / sum over the whole wave (result returned to every lane).
__device__ __forceinline__ float wave_max_f32_dpp(float v) {
    v = fmaxf(v, dpp_f32<0xb1>(-INFINITY, v));
    v = fmaxf(v, dpp_f32<0x4e>(-INFINITY, v));
    v = fmaxf(v, dpp_f32<0x114>(-INFINITY, v));
    v = fmaxf(v, dpp_f32<0x118>(-INFINITY, v));
    v = fmaxf(v, dpp_f32<0x142, 0xa>(-INFINITY, v));
    v = fmaxf(v, dpp_f32<0x143, 0xc>(-INFINITY, v));
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ float wave_sum_f32_dpp(float v) {
    v += dpp_f32<0xb1>(0.f, v);
    v += dpp_f32<0x4e>(0.f, v);
    v += dpp_f32<0x114>(0.f, v);
    v += dpp_f32<0x118>(0.f, v);
    v += dpp_f32<0x142, 0xa>(0.f, v);
    v += dpp_f32<0x143, 0xc>(0.f, v);
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ uint32_t wave_min_u32_dpp(uint32_t v) {
    v = min(v, dpp_u32<0xb1>(~0u, v));
    v = min(v, dpp_u32<0x4e>(~0u, v));
    v = min(v, dpp_u32<0x114>(~0u, v));
    v = min(v, dpp_u32<0x118>(~0u, v));
    v = min(v, dpp_u32<0x142, 0xa>(~0u, v));
    v = min(v, dpp_u32<0x143, 0xc>(~0u, v));
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Inclusive prefix sum over the lanes of a wave.
__device__ __forceinline__ int wave_prefix_sum_i32(int v) {
    const int lane = lane_id();
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const int t = __shfl_up(v, d);
        if (lane >= d) v += t;
    }
    return v;
}

// Unsigned 64-bit max / min over the whole wave, as two 32-bit reductions:
// the high words first, then the low words of the lanes holding that high
// word (each stage is one fused DPP max/min per step).
__device__ __forceinline__ uint64_t wave_max_u64_dpp(uint64_t v) {
    const uint32_t hi = (uint32_t)(v >> 32);
    const uint32_t H = wave_max_u32_dpp(hi);
    const uint32_t L = wave_max_u32_dpp(hi == H ? (uint32_t)v : 0u);
    return ((uint64_t)H << 32) | L;
}

__device__ __forceinline__ uint64_t wave_min_u64_dpp(uint64_t v) {
    const uint32_t hi = (uint32_t)(v >> 32);
    const uint32_t H = wave_min_u32_dpp(hi);
    const uint32_t L = wave_min_u32_dpp(hi == H ? (uint32_t)v : ~0u);
    return ((uint64_t)H << 32) | L;
}

// Unsigned 64-bit max over lanes 0..15 (row 0), returned to every lane.
__device__ __forceinline__ uint64_t row0_max_u64_dpp(uint64_t v) {
    uint64_t t;
    t = dpp_u64<0xb1>(0ull, v); v = t > v ? t : v;
    t = dpp_u64<0x4e>(0ull, v); v = t > v ? t : v;
    t = dpp_u64<0x114>(0ull, v); v = t > v ? t : v;
    t = dpp_u64<0x118>(0ull, v); v = t > v ? t : v;
    return readlane_u64(v, 15);
}

// Flags word: OR a bit from one lane (vector atomic).
__device__ __forceinline__ void raise_flag(int32_t* flags, int32_t bit) {
    if (flags) atomicOr(flags, bit);
}

}  // namespace presto

// Host-side launch helpers shared by the translation units.
namespace presto_host {
presto_status set_error(presto_status s, const char* fmt, ...);
presto_status check_launch(const char* what);
}  // namespace presto_host
