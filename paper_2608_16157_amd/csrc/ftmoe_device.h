// Device-side helpers shared by the gfx950 kernels of libftmoe (internal header).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ftmoe {

constexpr int kWave = 64;

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float floatx4_t __attribute__((__vector_size__(4 * sizeof(float))));
typedef float floatx16_t __attribute__((__vector_size__(16 * sizeof(float))));
typedef float floatx2_t __attribute__((__vector_size__(2 * sizeof(float))));
typedef uint32_t u32x4_t __attribute__((__vector_size__(4 * sizeof(uint32_t))));

// ---------------------------------------------------------------- number formats

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float32 -> bfloat16, round to nearest even (inputs are finite)
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// pack the high halves of two exactly-representable floats into a bf16 pair (exact for fp8 values)
__device__ __forceinline__ uint32_t pack_bf16_trunc(float lo, float hi) {
    return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

// 8 fp8 e4m3fn codes (two 32-bit words, code 0 in the low byte) -> 8 bf16, exact
__device__ __forceinline__ u32x4_t fp8x8_to_bf16x8(uint32_t w0, uint32_t w1) {
    const floatx2_t a = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w0), false);
    const floatx2_t b = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w0), true);
    const floatx2_t c = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w1), false);
    const floatx2_t d = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w1), true);
    return u32x4_t{pack_bf16_trunc(a[0], a[1]), pack_bf16_trunc(b[0], b[1]),
                   pack_bf16_trunc(c[0], c[1]), pack_bf16_trunc(d[0], d[1])};
}

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) {
    return __builtin_bit_cast(bf16x8_t, v);
}

// ---------------------------------------------------------------- wave utilities

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
        uint64_t o = __shfl_xor(v, s, kWave);
        v = o > v ? o : v;
    }
    return v;
}

__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) v += __shfl_xor(v, s, kWave);
    return v;
}

// Lanes of the wave whose `v` equals this lane's, restricted to `active`.
__device__ __forceinline__ uint64_t match_lanes(uint32_t v, int nbits, uint64_t active) {
    uint64_t m = active;
    for (int b = 0; b < nbits; ++b) {
        const bool bit = (v >> b) & 1u;
        const uint64_t bal = __ballot(bit);
        m &= bit ? bal : ~bal;
    }
    return m;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int l = lane_id();
    return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// ---------------------------------------------------------------- top-k keys
// Order-preserving 64-bit key: larger logit first, then lower expert id; -0.0 == +0.0.
__device__ __forceinline__ uint64_t topk_key(float logit, uint32_t e) {
    uint32_t u = __float_as_uint(logit);
    if (u == 0x80000000u) u = 0u;
    const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return (static_cast<uint64_t>(ord) << 32) | static_cast<uint32_t>(~e);
}

__device__ __forceinline__ uint32_t key_expert(uint64_t key) {
    return ~static_cast<uint32_t>(key);
}

__device__ __forceinline__ float key_logit(uint64_t key) {
    const uint32_t ord = static_cast<uint32_t>(key >> 32);
    const uint32_t u = (ord & 0x80000000u) ? (ord & 0x7FFFFFFFu) : ~ord;
    return __uint_as_float(u);
}

__device__ __forceinline__ float silu_f32(float z) { return z / (1.0f + __expf(-z)); }

}  // namespace ftmoe
