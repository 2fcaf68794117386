// Final attention outputs in the caller's element type (device code only).
#pragma once

#include "kernels.h"

namespace ema {

// fp32 -> bf16 with round to nearest, ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float v) {
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x0040u);
  return uint16_t((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// out[idx] = v in a.out_dtype (fp16 conversion rounds to nearest even).
__device__ __forceinline__ void store_out(const AttnArgs& a, int64_t idx, float v) {
  if (a.out_dtype == kOutF32) {
    static_cast<float*>(a.out)[idx] = v;
  } else if (a.out_dtype == kOutBF16) {
    static_cast<uint16_t*>(a.out)[idx] = f32_to_bf16_rne(v);
  } else {
    static_cast<_Float16*>(a.out)[idx] = _Float16(v);
  }
}

}  // namespace ema
