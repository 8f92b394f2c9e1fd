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
// The first conversion fills the low half of a word whose high half the
// second one overwrites, so its starting contents are free: a's own bits,
// which saves clearing a register.
__device__ __forceinline__ uint32_t e4m3x4_inrange(float a, float b, float c, float d) {
  const uint32_t w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)__float_as_uint(a), false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
}

// Codes of the 8 values v[0..7] / s (float division, nearest even).
__device__ __forceinline__ u32x2 code8(const float v[8], float s) {
  u32x2 w;
  w[0] = e4m3x4(__fdiv_rn(v[0], s), __fdiv_rn(v[1], s), __fdiv_rn(v[2], s), __fdiv_rn(v[3], s));
  w[1] = e4m3x4(__fdiv_rn(v[4], s), __fdiv_rn(v[5], s), __fdiv_rn(v[6], s), __fdiv_rn(v[7], s));
  return w;
}

__device__ __forceinline__ void bf16x8_to_f32(u32x4 x, float v[8]) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    v[2 * w] = bf16_bits_to_f32(x[w] & 0xFFFFu);
    v[2 * w + 1] = bf16_bits_to_f32(x[w] >> 16);
  }
}

// The power-of-two row scale of a query: the smallest e with mx <= 448 * 2^e
// (mx = max |a| over the row; 0 gives 0). mx = f * 2^k with f in [1, 2) and
// 448 = 1.75 * 2^8.
__device__ __forceinline__ int fp8_row_exponent(float mx) {
  if (!(mx > 0.f)) return 0;
  const uint32_t bits = __float_as_uint(mx);
  return (int)(bits >> 23) - 127 - 8 + ((bits & 0x7FFFFFu) > 0x600000u ? 1 : 0);
}


}  // namespace frt
