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

// 8 fp8 e4m3fn codes (two 32-bit words, code 0 in the low byte) -> 8 bf16, exact.  gfx950's
// scaled conversion multiplies by a power of two taken from its scale operand's exponent; with
// scale 1.0 it is a plain widening, exact because every e4m3fn value (3 mantissa bits, exponents
// 2^-9 .. 2^8) is a bf16 value.  Element order is kept: the low half of each result holds the
// lower-addressed code.
typedef __bf16 bf16x2_vec_t __attribute__((ext_vector_type(2)));
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI));
}
__device__ __forceinline__ u32x4_t fp8x8_to_bf16x8(uint32_t w0, uint32_t w1) {
    return u32x4_t{fp8x2_to_bf16x2<false>(w0), fp8x2_to_bf16x2<true>(w0), fp8x2_to_bf16x2<false>(w1),
                   fp8x2_to_bf16x2<true>(w1)};
}

// Scale operand of the scaled fp4 conversion for an e8m0 scale byte e (2^(e - 127); e = 0 the
// subnormal 2^-127, e = 255 NaN).  The conversion reads only the exponent field of its float
// operand, as an e8m0 exponent, so the byte shifted into that field is the whole decode: measured
// bit-identical to passing the decoded float (2^-127 as a subnormal, NaN for 255) for every byte
// and every code pair, without the compares and selects the decode costs.
__device__ __forceinline__ float fp4_scale_operand(uint32_t e) {
    return __builtin_bit_cast(float, e << 23);
}

// 8 fp4 e2m1 codes (one 32-bit word, element 0 in the low nibble) times a power-of-two scale ->
// 8 bf16 (exact: an e2m1 value has two significant bits), element order preserved; s comes from
// fp4_scale_operand
__device__ __forceinline__ u32x4_t fp4x8_scaled_to_bf16x8(uint32_t w, float s) {
    auto pk = [](bf16x2_vec_t v) { return __builtin_bit_cast(uint32_t, v); };
    return u32x4_t{pk(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, s, 0)),
                   pk(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, s, 1)),
                   pk(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, s, 2)),
                   pk(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, s, 3))};
}

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) {
    return __builtin_bit_cast(bf16x8_t, v);
}

// fp8 activations (FT_ACT_FP8_1x128_POW2).  The scale exponent of a 128-value block with largest
// magnitude amax: the smallest e with 448 * 2^e >= amax (448 = 0.875 * 2^9), 0 for amax = 0,
// clamped to the e8m0 range [-127, 127].
__device__ __forceinline__ int act_scale_exp(float amax) {
    int ex;
    const float m = frexpf(amax, &ex);   // amax = m 2^ex, 0.5 <= m < 1
    const int e = amax > 0.0f ? ex - 9 + (m > 0.875f ? 1 : 0) : 0;
    return min(max(e, -127), 127);
}

// e4m3fn code nearest to v, ties to even, for |v| <= 448.  Below 2^-6 the values are the
// multiples of 2^-9 (subnormal codes 0..7; 8 is the smallest normal, 2^-6); above, 3 mantissa
// bits rounded from float32's 23.
__device__ __forceinline__ uint32_t e4m3_rne(float v) {
    const uint32_t bits = __float_as_uint(v), sign = (bits >> 24) & 0x80u;
    const float a = fabsf(v);
    if (a < 0.015625f) return sign | static_cast<uint32_t>(__builtin_rintf(a * 512.0f));
    const uint32_t ab = bits & 0x7FFFFFFFu, m = ab & 0x7FFFFFu;
    uint32_t q = m >> 20;
    const uint32_t rem = m & 0xFFFFFu;
    q += (rem > 0x80000u || (rem == 0x80000u && (q & 1u))) ? 1u : 0u;
    return sign | ((((ab >> 23) - 120u) << 3) + q);   // exponent field e + 7; q = 8 carries
}

// value of an e4m3fn code (no NaN codes reach it)
__device__ __forceinline__ float e4m3_value(uint32_t c) {
    const uint32_t e = (c >> 3) & 15u, m = c & 7u;
    const float v = e ? __uint_as_float(((e + 120u) << 23) | (m << 20)) : static_cast<float>(m) * 0.001953125f;
    return (c & 0x80u) ? -v : v;
}

// ---------------------------------------------------------------- wave utilities
// Cross-lane steps use DPP row rotations/shifts (within 16-lane rows) plus v_readlane of the
// four row results, so no reduction goes through the LDS crossbar (ds_bpermute).

__device__ __forceinline__ int lane_id() { return __lane_id(); }

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, 0xF, 0xF, true));
}
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppRowRor1 = 0x121, kDppRowRor2 = 0x122, kDppRowRor4 = 0x124, kDppRowRor8 = 0x128;

__device__ __forceinline__ uint32_t readlane_u32(uint32_t v, int l) {
    return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), l));
}

// max over the 16 lanes of this lane's row, in every lane of the row
__device__ __forceinline__ uint32_t row_max_u32(uint32_t v) {
    v = max(v, dpp_u32<kDppRowRor1>(v));
    v = max(v, dpp_u32<kDppRowRor2>(v));
    v = max(v, dpp_u32<kDppRowRor4>(v));
    return max(v, dpp_u32<kDppRowRor8>(v));
}

// max over the 64 lanes, result uniform
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = row_max_u32(v);
    return max(max(readlane_u32(v, 0), readlane_u32(v, 16)), max(readlane_u32(v, 32), readlane_u32(v, 48)));
}

// sum over the 64 lanes in a fixed order (deterministic), result uniform
__device__ __forceinline__ float wave_sum_f32(float x) {
    uint32_t v = __float_as_uint(x);
    v = __float_as_uint(__uint_as_float(v) + __uint_as_float(dpp_u32<kDppRowRor1>(v)));
    v = __float_as_uint(__uint_as_float(v) + __uint_as_float(dpp_u32<kDppRowRor2>(v)));
    v = __float_as_uint(__uint_as_float(v) + __uint_as_float(dpp_u32<kDppRowRor4>(v)));
    v = __float_as_uint(__uint_as_float(v) + __uint_as_float(dpp_u32<kDppRowRor8>(v)));
    const float a = __uint_as_float(readlane_u32(v, 0)), b = __uint_as_float(readlane_u32(v, 16));
    const float c = __uint_as_float(readlane_u32(v, 32)), d = __uint_as_float(readlane_u32(v, 48));
    return (a + b) + (c + d);
}

// inclusive prefix sum over the 64 lanes (lane order)
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) {
    v += dpp_u32<kDppRowShr1>(v);
    v += dpp_u32<kDppRowShr2>(v);
    v += dpp_u32<kDppRowShr4>(v);
    v += dpp_u32<kDppRowShr8>(v);
    const uint32_t r0 = readlane_u32(v, 15), r1 = readlane_u32(v, 31), r2 = readlane_u32(v, 47);
    const int row = lane_id() >> 4;
    return v + (row > 0 ? r0 : 0u) + (row > 1 ? r1 : 0u) + (row > 2 ? r2 : 0u);
}

// inclusive prefix maximum over the 64 lanes (lane order); 0 is the neutral value
__device__ __forceinline__ uint32_t wave_incl_max_u32(uint32_t v) {
    v = max(v, dpp_u32<kDppRowShr1>(v));
    v = max(v, dpp_u32<kDppRowShr2>(v));
    v = max(v, dpp_u32<kDppRowShr4>(v));
    v = max(v, dpp_u32<kDppRowShr8>(v));
    const uint32_t r0 = readlane_u32(v, 15), r1 = readlane_u32(v, 31), r2 = readlane_u32(v, 47);
    const int row = lane_id() >> 4;
    const uint32_t c = max(row > 0 ? r0 : 0u, max(row > 1 ? r1 : 0u, row > 2 ? r2 : 0u));
    return max(v, c);
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
// Order-preserving 32-bit key of a finite float (larger float -> larger key, -0.0 == +0.0);
// every finite float maps to a key >= 0x00800000, so 0 can mark an empty/removed entry.
__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_to_float(uint32_t ord) {
    const uint32_t u = (ord & 0x80000000u) ? (ord & 0x7FFFFFFFu) : ~ord;
    return __uint_as_float(u);
}

__device__ __forceinline__ float silu_f32(float z) { return z / (1.0f + __expf(-z)); }

}  // namespace ftmoe
