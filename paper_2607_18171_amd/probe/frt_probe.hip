// Measurement probes for the benchmark (not part of the attention library):
// the bf16 and FP8 (e4m3) MFMA rates this part sustains on random operands
// with no memory or vector work, at the occupancy of the chunk attention
// kernels (one block of eight waves per CU, two waves per SIMD).
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

}  // extern "C"
