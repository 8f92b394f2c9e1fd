// Measurement probes for the benchmark (not part of the attention library):
// the bf16 and FP8 (e4m3) MFMA rates this part sustains on random operands
// with no memory or vector work, at the occupancy of the chunk attention
// kernels (one block of eight waves per CU, two waves per SIMD); and the rate
// at which plain streaming reads of a given size come from HBM.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int kWaves = 8;
constexpr int kFrags = 4;  // operand fragments per wave, used in rotation
constexpr int kPadBytes = 96 * 1024;  // LDS that keeps a second block off the CU

// Each wave runs kFrags independent accumulator chains of 32x32 MFMAs;
// iteration i pairs A fragment c with B fragment (c + i) mod kFrags, so the
// operands change from one MFMA to the next as a real contraction's do.
__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma(i32x8 a, i32x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

template <class Frag>
__global__ __launch_bounds__(kWaves * 64) void mfma_loop_kernel(const Frag *frags, float *out,
                                                                int iters) {
  __shared__ float pad[kPadBytes / 4];
  const int lane = threadIdx.x & 63;
  Frag a[kFrags], b[kFrags];
#pragma unroll
  for (int c = 0; c < kFrags; ++c) {
    a[c] = frags[c * 64 + lane];
    b[c] = frags[(kFrags + c) * 64 + lane];
  }
  f32x16 acc[kFrags];
#pragma unroll
  for (int c = 0; c < kFrags; ++c) acc[c] = f32x16{};
  for (int i = 0; i < iters; i += kFrags) {
#pragma unroll
    for (int r = 0; r < kFrags; ++r)
#pragma unroll
      for (int c = 0; c < kFrags; ++c)
        acc[c] = mfma(a[c], b[(c + r) % kFrags], acc[c]);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kFrags; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  // every thread writes its own LDS word across the whole pad, so the pad is
  // allocated in full
  pad[threadIdx.x * (kPadBytes / 4 / (kWaves * 64))] = s;
  __syncthreads();
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] =
      pad[(threadIdx.x ^ 1) * (kPadBytes / 4 / (kWaves * 64))];
}

template <class Frag>
int launch(const void *frags, void *out, int blocks, int iters, void *stream) {
  if (frags == nullptr || out == nullptr || blocks <= 0 || iters <= 0 || iters % kFrags != 0)
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(mfma_loop_kernel<Frag>, dim3(blocks), dim3(kWaves * 64), 0,
                     (hipStream_t)stream, static_cast<const Frag *>(frags),
                     static_cast<float *>(out), iters);
  return (int)hipGetLastError();
}

// Streaming read: thread i of the grid reads the 16-byte words i, i + n, ...
// (n = threads in the grid), U independent loads in flight per thread, and
// folds them with xor; only a word that can never occur is stored, so the
// loads cannot be dropped and nothing is written.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

template <int U>
__global__ __launch_bounds__(256) void read_kernel(const u32x4 *__restrict__ src, size_t n16,
                                                   unsigned *sink) {
  const size_t nth = (size_t)gridDim.x * 256;
  u32x4 acc = {0, 0, 0, 0};
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += nth * U) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const size_t j = i + (size_t)u * nth;
      v[u] = j < n16 ? src[j] : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u];
  }
  if ((acc[0] ^ acc[1] ^ acc[2] ^ acc[3]) == 0x9e3779b9u && acc[0] == 0x7f4a7c15u)
    sink[blockIdx.x] = acc[1];
}

}  // namespace

extern "C" {

// frags: 2 * 4 * 64 operand fragments (device, random values): 16-byte
// bf16x8 fragments, or 32-byte fragments of 32 e4m3 codes for the FP8 probe.
// out: blocks * 512 floats (device). iters: MFMAs per chain, a multiple of 4.
// Work: blocks * 8 waves * 4 chains * iters MFMAs of 32*32*16*2 (bf16) or
// 32*32*64*2 (FP8) flops. Returns 0, or the HIP error of the launch.
int frt_probe_mfma_bf16(const void *frags, void *out, int blocks, int iters, void *stream) {
  return launch<bf16x8>(frags, out, blocks, iters, stream);
}

int frt_probe_mfma_fp8(const void *frags, void *out, int blocks, int iters, void *stream) {
  return launch<i32x8>(frags, out, blocks, iters, stream);
}

// src: `bytes` of device memory (a multiple of 16), read once. sink: `blocks`
// unsigned words (device), written only for a data pattern the caller never
// supplies. blocks: grid size (256 threads each); unroll: loads in flight per
// thread, 2, 4, 8 or 16. Returns 0, or hipErrorInvalidValue for bad arguments,
// or the HIP error of the launch.
int frt_probe_read(const void *src, size_t bytes, void *sink, int blocks, int unroll,
                   void *stream) {
  if (src == nullptr || sink == nullptr || bytes == 0 || bytes % 16 != 0 || blocks <= 0)
    return (int)hipErrorInvalidValue;
  const u32x4 *p = static_cast<const u32x4 *>(src);
  unsigned *k = static_cast<unsigned *>(sink);
  const hipStream_t st = (hipStream_t)stream;
  switch (unroll) {
    case 2: hipLaunchKernelGGL(read_kernel<2>, dim3(blocks), dim3(256), 0, st, p, bytes / 16, k); break;
    case 4: hipLaunchKernelGGL(read_kernel<4>, dim3(blocks), dim3(256), 0, st, p, bytes / 16, k); break;
    case 8: hipLaunchKernelGGL(read_kernel<8>, dim3(blocks), dim3(256), 0, st, p, bytes / 16, k); break;
    case 16: hipLaunchKernelGGL(read_kernel<16>, dim3(blocks), dim3(256), 0, st, p, bytes / 16, k); break;
    default: return (int)hipErrorInvalidValue;
  }
  return (int)hipGetLastError();
}

}  // extern "C"
