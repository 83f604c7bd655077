// Device helpers shared by the hook-step kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xmix {

constexpr int kWave = 64;

// ---------------------------------------------------------------- bf16 bits
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round-to-nearest-even of an fp32 value onto bf16, as bits.  Adding
// 0x7FFF plus the lowest kept bit and truncating rounds half to even; it
// carries into the exponent correctly, including the overflow to infinity.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0;  // NaN
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// Two bf16 packed in one dword: element 0 in the low half.
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
    return static_cast<uint32_t>(f32_to_bf16_rne(a)) |
           (static_cast<uint32_t>(f32_to_bf16_rne(b)) << 16);
}

// Round-to-nearest-even of an fp64 value onto bf16 without double
// rounding: first round to fp32 with round-to-odd (truncate, then set the
// last bit if anything was dropped), which keeps the information a later
// round-to-nearest needs because fp32 carries 16 more bits than bf16; then
// round that fp32 value to bf16.
__device__ __forceinline__ uint16_t f64_to_bf16_rne(double x) {
    float f = __double2float_rz(x);
    if (static_cast<double>(f) != x && x == x) f = __uint_as_float(__float_as_uint(f) | 1u);
    return f32_to_bf16_rne(f);
}
__device__ __forceinline__ uint32_t pack_bf16_from_f64(double a, double b) {
    return static_cast<uint32_t>(f64_to_bf16_rne(a)) |
           (static_cast<uint32_t>(f64_to_bf16_rne(b)) << 16);
}

// Order-preserving map of fp32 onto uint32: a < b  <=>  key(a) < key(b).
__device__ __forceinline__ uint32_t f32_key(float f) {
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_f32(uint32_t k) {
    uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(u);
}

// ----------------------------------------------------------- wave helpers
__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Number of lanes below this one whose bit is set in `ballot`.
__device__ __forceinline__ int lanes_below(uint64_t ballot) {
    return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(ballot >> 32),
                                     __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(ballot), 0));
}

__device__ __forceinline__ uint64_t wave_ballot(bool p) { return __ballot(p); }

// Butterfly sum over the 64 lanes; every lane receives the total.  The
// combination order is fixed, so the result is bit-reproducible.
// DPP lane moves (every source lane active): quad_perm [1,0,3,2] and
// [2,3,0,1], row_half_mirror and row_mirror inside each row of 16 lanes.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;
__device__ __forceinline__ float readlane_f(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// The sum over the 64 lanes of a wave, the same value in every lane (every
// lane active): DPP moves add within each row of 16 lanes, then the four row
// sums are added in a fixed order.
__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_f<kDppXor1>(v);
    v += dpp_f<kDppXor2>(v);
    v += dpp_f<kDppHalfMirror>(v);
    v += dpp_f<kDppMirror>(v);
    return (readlane_f(v, 0) + readlane_f(v, 16)) + (readlane_f(v, 32) + readlane_f(v, 48));
}

__device__ __forceinline__ float logistic(float x) { return 1.0f / (1.0f + expf(-x)); }

}  // namespace xmix
