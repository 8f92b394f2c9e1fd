// Device helpers of the FP8 (OCP e4m3fn) path: the fp32 RoPE rotation that
// the codes start from, and the fp32 -> e4m3fn conversions.
#pragma once
#include "frt_device.hpp"

namespace frt {

// The rotation and scaling of rotate8_apply, stopping at the float rounding:
// the eight fp32 values that its bf16 rounding would start from.
__device__ __forceinline__ void rotate8_f32(const Rope4 &t, u32x4 x, double mul, float y[8]) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const uint32_t lo = x[w] & 0xFFFFu, hi = x[w] >> 16;
    double y0, y1;
    if (t.on & (1u << w)) {
      rotate_pair_f64(lo, hi, t.cs[w].x, t.cs[w].y, y0, y1);
    } else {
      y0 = (double)bf16_bits_to_f32(lo);
      y1 = (double)bf16_bits_to_f32(hi);
    }
    y[2 * w] = (float)(y0 * mul);
    y[2 * w + 1] = (float)(y1 * mul);
  }
}

// Four fp32 values -> four OCP e4m3fn codes in one word (value j in byte j):
// clamped to +-448, then rounded to nearest, ties to even, by the hardware
// conversion (which leaves values beyond the range as NaN, hence the clamp).
constexpr float kE4m3Max = 448.f;
__device__ __forceinline__ uint32_t e4m3x4(float a, float b, float c, float d) {
  a = fminf(fmaxf(a, -kE4m3Max), kE4m3Max);
  b = fminf(fmaxf(b, -kE4m3Max), kE4m3Max);
  c = fminf(fmaxf(c, -kE4m3Max), kE4m3Max);
  d = fminf(fmaxf(d, -kE4m3Max), kE4m3Max);
  const uint32_t w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
}
// The same for values already known to lie within +-448 (no clamp needed).
__device__ __forceinline__ uint32_t e4m3x4_inrange(float a, float b, float c, float d) {
  const uint32_t w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
}

}  // namespace frt
