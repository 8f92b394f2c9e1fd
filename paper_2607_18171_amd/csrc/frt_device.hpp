// Device-side helpers shared by the libfrt kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace frt {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kMaskBlockCausal = 1;
constexpr int kMaskCausal = 2;
constexpr int kRopeNone = 0;
constexpr int kRope1D = 1;
constexpr int kRope3D = 2;

// Buffer resource word 3 for raw (untyped) buffer access on gfx9-family parts.
constexpr int kBufferWord3 = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                           kBufferWord3);
}

// 16-byte buffer load; byte offsets at or past `bytes` of the descriptor read 0.
__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, 0);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) {
  return __uint_as_float(b << 16);
}

// float -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// Rotary parameters as the kernels see them.
struct RopeDev {
  int mode;           // kRopeNone / kRope1D / kRope3D
  int npairs[3];      // pairs per axis (axis_dims / 2); 0 = axis absent
  int maxpos[3];      // table rows per axis
  int frame_h, frame_w;
  const float2 *tab[3];  // per axis: (cos, sin) at [pos][pair]
};

// Axis coordinates of token p.
__device__ __forceinline__ void rope_coords(const RopeDev &r, long long p, int c[3]) {
  if (r.mode == kRope3D) {
    long long hw = (long long)r.frame_h * r.frame_w;
    long long t = p / hw;
    long long rem = p - t * hw;
    c[0] = (int)t;
    c[1] = (int)(rem / r.frame_w);
    c[2] = (int)(rem - (long long)c[1] * r.frame_w);
  } else {
    c[0] = (int)p;
    c[1] = 0;
    c[2] = 0;
  }
}

// cos/sin of pair `j` of the head vector at coordinates c; returns false when
// the pair lies outside every rotated slice (identity).
__device__ __forceinline__ bool rope_pair(const RopeDev &r, const int c[3], int j, float &cs,
                                          float &sn) {
  if (r.mode == kRopeNone) return false;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    if (j < r.npairs[a]) {
      int pos = c[a];
      pos = pos < 0 ? 0 : (pos >= r.maxpos[a] ? r.maxpos[a] - 1 : pos);
      float2 v = r.tab[a][(size_t)pos * r.npairs[a] + j];
      cs = v.x;
      sn = v.y;
      return true;
    }
    j -= r.npairs[a];
  }
  return false;
}

// Rotate one pair of bf16 values in double precision. Each product of a bf16
// and a float is exact in double, so only the final add rounds; with or
// without contraction the double result is the same.
__device__ __forceinline__ void rotate_pair_f64(uint32_t x0b, uint32_t x1b, float cs, float sn,
                                                double &y0, double &y1) {
  double x0 = (double)bf16_bits_to_f32(x0b);
  double x1 = (double)bf16_bits_to_f32(x1b);
  double c = (double)cs, s = (double)sn;
  y0 = x0 * c - x1 * s;
  y1 = x0 * s + x1 * c;
}

// Rotate 8 consecutive bf16 values (4 pairs starting at pair `j0`) of a head
// vector at coordinates c, scale by `mul` in double, and round double ->
// float -> bf16 (nearest even at both steps). With mul = 1 this is exactly
// the value a ring slot stores for a key.
__device__ __forceinline__ u32x4 rotate8_round(const RopeDev &r, const int c[3], int j0, u32x4 x,
                                               double mul) {
  u32x4 y;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t lo = x[w] & 0xFFFFu, hi = x[w] >> 16;
    float cs, sn;
    double y0, y1;
    if (rope_pair(r, c, j0 + w, cs, sn)) {
      rotate_pair_f64(lo, hi, cs, sn, y0, y1);
    } else {
      y0 = (double)bf16_bits_to_f32(lo);
      y1 = (double)bf16_bits_to_f32(hi);
    }
    y0 *= mul;
    y1 *= mul;
    y[w] = f32_to_bf16_rne((float)y0) | (f32_to_bf16_rne((float)y1) << 16);
  }
  return y;
}

// Inclusive range [lo, hi] of key tokens visible to query token p.
__device__ __forceinline__ void visible_range(int kind, int block, int window, long long p,
                                              long long &lo, long long &hi) {
  if (kind == kMaskBlockCausal) {
    long long bp = p / block;
    lo = window ? (bp - window) * (long long)block : 0;
    hi = (bp + 1) * (long long)block - 1;
  } else {
    lo = window ? p - window + 1 : 0;
    hi = p;
  }
  if (lo < 0) lo = 0;
}

__device__ __forceinline__ int clamp_i32(long long v) {
  return v < -0x40000000LL ? -0x40000000 : (v > 0x40000000LL ? 0x40000000 : (int)v);
}

}  // namespace frt
