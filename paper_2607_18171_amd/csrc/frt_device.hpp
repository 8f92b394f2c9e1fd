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

// Selection between values, not lvalues: a conditional between two lvalues
// selects their addresses, which pushes the selected variables to memory.
template <class T>
__device__ __forceinline__ T pick(bool c, T a, T b) {
  return c ? a : b;
}

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

// V ring layout of one (stream, KV head): the C slots are kept in blocks of
// kVBlock slots, and block k stores its slots row by row of the head
// dimension, so a block of consecutive keys is one contiguous piece of memory.
// Element (slot s, row d) sits at kVBlock*D*k + w_k*d + s % kVBlock, where w_k
// is kVBlock for a full block and C % kVBlock for a partial last block (C is a
// multiple of 8, so an 8-slot group never leaves its block).
constexpr int kVBlock = 32;
// row length w_k of the block holding slot s (0 <= s)
__device__ __forceinline__ uint32_t vring_width(int s, int C) {
  const uint32_t k = (uint32_t)s / kVBlock, nfull = (uint32_t)C / kVBlock;
  return k < nfull ? kVBlock : (uint32_t)C - kVBlock * nfull;
}
__device__ __forceinline__ uint32_t vring_elem(int s, int d, int C, int D) {
  return kVBlock * (uint32_t)D * ((uint32_t)s / kVBlock) + vring_width(s, C) * (uint32_t)d +
         (uint32_t)s % kVBlock;
}

// Two packed bf16 values as a vector. Taking the word by value matters:
// __builtin_bit_cast applied directly to a subscripted vector element has
// been seen to read element 0 whatever the index.
__device__ __forceinline__ bf16x2 u32_as_bf16x2(uint32_t w) {
  return __builtin_bit_cast(bf16x2, w);
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

// Rotary parameters as the kernels receive them (a kernel argument). The
// (cos, sin) table holds the axes back to back, axis a from entry tab_off[a],
// each as [pos][pair].
struct RopeDev {
  int mode;           // kRopeNone / kRope1D / kRope3D
  int npairs[3];      // pairs per axis (axis_dims / 2); 0 = axis absent
  int maxpos[3];      // table rows per axis
  int tab_off[3];     // first entry of each axis
  int frame_h, frame_w;
  uint32_t tab_bytes;  // bytes of the whole table (< 2^31)
  const float2 *table;
};

// The same parameters held in scalar registers. Each field passes through
// readfirstlane once, and the table is read through a buffer descriptor, so
// choosing a lane's axis is a select between register values and a table
// read is an ordinary vector load that needs no wait of its own.
struct RopeReg {
  int n0, n1, n2;  // pairs per axis
  int m0, m1, m2;  // table rows per axis
  int o0, o1, o2;  // first entry per axis
  int mode, fh, fw;
  __amdgpu_buffer_rsrc_t tab;
};

__device__ __forceinline__ int uniform_i32(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ RopeReg rope_reg(const RopeDev &r) {
  RopeReg g;
  g.mode = uniform_i32(r.mode);
  g.n0 = uniform_i32(r.npairs[0]);
  g.n1 = uniform_i32(r.npairs[1]);
  g.n2 = uniform_i32(r.npairs[2]);
  g.m0 = uniform_i32(r.maxpos[0]);
  g.m1 = uniform_i32(r.maxpos[1]);
  g.m2 = uniform_i32(r.maxpos[2]);
  g.o0 = uniform_i32(r.tab_off[0]);
  g.o1 = uniform_i32(r.tab_off[1]);
  g.o2 = uniform_i32(r.tab_off[2]);
  g.fh = uniform_i32(r.frame_h);
  g.fw = uniform_i32(r.frame_w);
  g.tab = make_rsrc(r.table, r.tab_bytes);
  return g;
}

// Axis coordinates of token p.
__device__ __forceinline__ void rope_coords(const RopeReg &r, long long p, int c[3]) {
  if (r.mode == kRope3D) {
    const long long hw = (long long)r.fh * r.fw;
    const long long t = p / hw;
    const long long rem = p - t * hw;
    c[0] = (int)t;
    c[1] = (int)(rem / r.fw);
    c[2] = (int)(rem - (long long)c[1] * r.fw);
  } else {
    c[0] = (int)p;
    c[1] = 0;
    c[2] = 0;
  }
}

// (cos, sin) of pair j of the head vector at coordinates c; false when the
// pair lies outside every rotated slice (identity; cs is then (0, 0)). The
// load is issued either way, past the descriptor when not needed.
__device__ __forceinline__ bool rope_pair(const RopeReg &r, const int c[3], int j, float2 &cs) {
  const int e0 = r.n0, e1 = e0 + r.n1, e2 = e1 + r.n2;
  const bool on = j < e2;  // no axis when the mode is kRopeNone
  const bool in0 = j < e0, in1 = j < e1;
  const int np = pick(in0, r.n0, pick(in1, r.n1, r.n2));
  const int mp = pick(in0, r.m0, pick(in1, r.m1, r.m2));
  const int base = pick(in0, r.o0, pick(in1, r.o1 - e0, r.o2 - e1));
  int pos = pick(in0, c[0], pick(in1, c[1], c[2]));
  pos = pos < 0 ? 0 : (pos >= mp ? mp - 1 : pos);
  const uint32_t off = on ? (uint32_t)(base + pos * np + j) * 8u : 0x80000000u;
  const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r.tab, (int)off, 0, 0);
  cs = make_float2(__uint_as_float(v[0]), __uint_as_float(v[1]));
  return on;
}

// Table entries of the 4 pairs starting at pair j0; bit w of the result says
// whether pair j0 + w is rotated. Split from the arithmetic so that a kernel
// can issue these loads early.
struct Rope4 {
  float2 cs[4];
  uint32_t on;
};

__device__ __forceinline__ Rope4 rope_fetch4(const RopeReg &r, const int c[3], int j0) {
  Rope4 t;
  t.on = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w)
    if (rope_pair(r, c, j0 + w, t.cs[w])) t.on |= 1u << w;
  return t;
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

// Rotate 8 consecutive bf16 values (the 4 pairs of t) in double precision,
// scale by `mul` in double, and round double -> float -> bf16 (nearest even
// at both steps). With mul = 1 this is exactly the value a ring slot stores
// for a key. Pairs that are not rotated pass through unchanged before the
// scaling, which keeps the sign of a zero.
__device__ __forceinline__ u32x4 rotate8_apply(const Rope4 &t, u32x4 x, double mul) {
  u32x4 y;
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
    y0 *= mul;
    y1 *= mul;
    y[w] = f32_to_bf16_rne((float)y0) | (f32_to_bf16_rne((float)y1) << 16);
  }
  return y;
}

__device__ __forceinline__ u32x4 rotate8_round(const RopeReg &r, const int c[3], int j0, u32x4 x,
                                               double mul) {
  return rotate8_apply(rope_fetch4(r, c, j0), x, mul);
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
