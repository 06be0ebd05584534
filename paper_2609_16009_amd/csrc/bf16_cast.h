// fp32 -> bf16 conversions shared by the kernels (device code only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace nmm {

// Nearest, ties to even (the hardware conversion).
__device__ __forceinline__ uint16_t to_bf16_bits(float v) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}

// Nearest, ties away from zero: adding half of the dropped range to the magnitude bits carries
// into the kept bits exactly when the dropped part is at least one half (a carry out of the
// largest finite value ends at infinity, as it should).  NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t to_bf16_bits_away(float v) {
    const uint32_t u = __float_as_uint(v);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
    return static_cast<uint16_t>((u + 0x8000u) >> 16);
}

__device__ __forceinline__ uint16_t to_bf16_mode(float v, int away) {
    return away ? to_bf16_bits_away(v) : to_bf16_bits(v);
}

}  // namespace nmm
