// Kernel parameter blocks and launchers (internal to libfrt).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "frt_device.hpp"

namespace frt {

struct AppendParams {
  const uint16_t *k_new;  // [B][n][Hkv][D]
  const uint16_t *v_new;  // [B][n][Hkv][D]
  uint16_t *k_ring;       // [B][Hkv][C][D]
  uint16_t *v_ring;       // [B][Hkv][C*D]   32-slot blocks
  int64_t *seq_len;       // [B]
  int B, Hkv, D, C, n;
};

// Append of a prepared chunk: the rotated keys of the step workspace and the
// values v_new go to slots (L + i) mod C, L as the preparation pass recorded
// it; seq_len becomes L + n.
struct ChunkAppendParams {
  const uint16_t *kr;     // [B][Hkv][n_pad][D]
  const uint16_t *v_new;  // [B][n][Hkv][D]
  const int64_t *lrec;    // [B]  seq_len at the step's start
  uint16_t *k_ring, *v_ring;
  int64_t *seq_len;
  int B, Hkv, D, C, n, n_pad;
};

// FP8 (e4m3fn) ring: same layouts as the bf16 ring with one-byte elements;
// per-(stream, KV head) fp32 scales, a stored code standing for code * scale.
struct Fp8Scales {
  const float *k, *v;     // [B][Hkv]
};

struct AppendFp8Params {
  const uint16_t *k_new;  // [B][n][Hkv][D]  bf16
  const uint16_t *v_new;
  uint8_t *k_ring;        // [B][Hkv][C][D]
  uint8_t *v_ring;        // [B][Hkv][C*D]   32-slot blocks
  int64_t *seq_len;
  Fp8Scales sc;
  int B, Hkv, D, C, n;
};

struct PrepFp8Params {
  const uint16_t *q, *k_new, *v_new;
  const int64_t *seq_len;
  uint8_t *qr;            // [B][Hkv][n*G][D]  query codes
  float *qs;              // [B][Hkv][n*G]     their row scale 2^e
  uint8_t *kr;            // [B][Hkv][n_pad][D] own key codes (as the ring stores them)
  uint8_t *vt;            // [B][Hkv][n_pad*D]  own value codes, ring block layout
  int64_t *lrec;          // [B]  seq_len at the step's start (for the fused append)
  Fp8Scales sc;
  int B, Hq, Hkv, G, D, n, n_pad;
  double qmul;
};

// Fused-step append of the FP8 ring from the preparation pass's codes.
struct ChunkAppendFp8Params {
  const uint8_t *kr;      // [B][Hkv][n_pad][D] key codes
  const uint8_t *vt;      // [B][Hkv][n_pad*D] value codes in 32-token blocks [d][32]
  const int64_t *lrec;    // [B]  seq_len at the step's start
  uint8_t *k_ring, *v_ring;
  int64_t *seq_len;
  int B, Hkv, D, C, n, n_pad;
};

struct AttnFp8Params {
  const uint8_t *qr, *kr, *vt;
  const float *qs;
  const uint8_t *k_ring, *v_ring;
  const int64_t *seq_len;
  Fp8Scales sc;
  uint16_t *out;
  float *lse;
  int B, Hq, Hkv, G, n, n_pad, C;
  int mask_kind, mask_block, mask_window;
  int row_tiles;
};

struct PrepParams {
  const uint16_t *q;      // [B][n][Hq][D]
  const uint16_t *k_new;  // [B][n][Hkv][D]
  const uint16_t *v_new;  // [B][n][Hkv][D]
  const int64_t *seq_len;
  uint16_t *qr;           // [B][Hkv][n*G][D]    rotated, scaled by qmul
  uint16_t *kr;           // [B][Hkv][n_pad][D]  rotated (stored-key rounding)
  uint16_t *vt;           // [B][Hkv][n_pad*D]   V ring block layout
  int64_t *lrec;          // [B]  seq_len at the step's start, recorded
  int B, Hq, Hkv, G, D, n, n_pad;
  double qmul;            // softmax scale * log2(e)
};

struct AttnParams {
  const uint16_t *qr, *kr, *vt;         // prepared chunk (see PrepParams)
  const uint16_t *k_ring, *v_ring;
  const int64_t *seq_len;
  uint16_t *out;                        // [B][n][Hq][D]
  float *lse;                           // [B][Hq][n] or null
  int B, Hq, Hkv, G, n, n_pad, C;
  int mask_kind, mask_block, mask_window;
  int row_tiles;
};

struct DecodeParams {
  const uint16_t *q;       // [B][1][Hq][D]
  const uint16_t *k_new;   // [B][1][Hkv][D]
  const uint16_t *v_new;   // [B][1][Hkv][D]
  uint16_t *k_ring, *v_ring;  // written only by the combine pass, and only with append
  int64_t *seq_len;
  float *ws;               // partials: nwaves + B * Hkv
  uint16_t *out;           // [B][1][Hq][D]
  float *lse;              // [B][Hq][1] or null
  int B, Hq, Hkv, G, D, C;
  int nwaves;              // piece waves of the split pass (multiple of 4)
  int mask_kind, mask_block, mask_window;
  int append;              // combine pass also appends the token to the ring
  double qmul;
};

// One-token decode over an FP8 ring (head_dim 128).
struct DecodeFp8Params {
  const uint16_t *q;       // [B][1][Hq][D] bf16
  const uint16_t *k_new;   // [B][1][Hkv][D] bf16
  const uint16_t *v_new;   // [B][1][Hkv][D] bf16
  uint8_t *k_ring, *v_ring;  // written only by the combine pass, and only with append
  int64_t *seq_len;
  Fp8Scales sc;
  float *ws;               // partials: nwaves + B * Hkv
  uint16_t *out;           // [B][1][Hq][D]
  float *lse;              // [B][Hq][1] or null
  int B, Hq, Hkv, G, D, C;
  int nwaves;              // piece waves of the split pass (multiple of 4)
  int mask_kind, mask_block, mask_window;
  int append;              // combine pass also appends the token to the ring
  double qmul;
};

constexpr int kAppendTokens = 64;   // tokens per append / prep block
constexpr int kAppendSmall = 16;    // appends up to this many tokens take one launch
constexpr int kChunkBN = 64;        // keys per attention tile
#ifndef FRT_ATTN_WAVES
#define FRT_ATTN_WAVES 8
#endif
constexpr int kChunkWaves = FRT_ATTN_WAVES;  // waves per attention block
constexpr int kChunkRows = 32 * kChunkWaves;  // query rows per block (32 per wave)
constexpr int kDecWavesPerSimd = 2;  // decode split occupancy (register bound)
constexpr int kDecBufs = 2;          // decode split tiles in flight per wave
constexpr int kDecResident = 256 * 4 * kDecWavesPerSimd;  // split waves resident at once
constexpr int kDecChunk = 12;        // most 32-token tiles of one decode piece

// Piece waves of a decode call: enough for every split of the tiles
// (resident waves plus one per head, or pieces of kDecChunk tiles when the
// ring is long), rounded up to whole blocks of 4 waves.
__host__ __device__ inline int decode_piece_waves(int B, int Hkv, int C) {
  const long long heads = (long long)B * Hkv;
  const long long tiles_max = (long long)C / 32 + 1;
  const long long cap = heads * ((tiles_max + kDecChunk - 1) / kDecChunk) + heads;
  long long w = kDecResident + heads;
  w = w > cap ? w : cap;
  return (int)((w + 3) / 4 * 4);
}
// One decode partial (floats): max[G] at 0, sum[G] at G, out[G][D] from
// decode_out_off(G); the stride keeps every partial and its output rows
// 16-byte aligned.
__host__ __device__ inline int decode_out_off(int G) { return (2 * G + 3) / 4 * 4; }
__host__ __device__ inline size_t decode_split_floats(int G, int D) {
  return (size_t)decode_out_off(G) + (size_t)G * D;
}
// Floats of one FP8 decode partial: max[G], sum[G], out[G][D], then (in a
// head's own-token slot) 4 header words and the token's key and value codes.
__host__ __device__ inline size_t decode_fp8_split_floats(int G, int D) {
  return ((size_t)G * (2 + D) + 4 + (size_t)D / 2 + 3) / 4 * 4;
}

// Timing events for the next kernel dispatch of this host thread. The
// library's timing sets them; the dispatch then records its own start and end
// in them (HIP's event-carrying launch), so a timed interval holds the kernel
// alone and no extra packets go into the stream.
struct DispatchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
DispatchEvents &pending_dispatch_events();

// Every kernel of the library is launched through this.
template <typename F, typename... Args>
void dispatch(F kernel, dim3 grid, dim3 block, hipStream_t s, Args... args) {
  DispatchEvents &ev = pending_dispatch_events();
  const hipEvent_t a = ev.start, b = ev.stop;
  ev = DispatchEvents{};
  hipExtLaunchKernelGGL(kernel, grid, block, 0u, s, a, b, 0u, args...);
}

hipError_t launch_rope_append(const AppendParams &p, const RopeDev &r, hipStream_t s);
hipError_t launch_rope_append_small(const AppendParams &p, const RopeDev &r, hipStream_t s);
hipError_t launch_seq_advance(int64_t *seq_len, int B, int n, hipStream_t s);
hipError_t launch_chunk_prep(const PrepParams &p, const RopeDev &r, hipStream_t s);
hipError_t launch_chunk_attn(const AttnParams &p, int D, hipStream_t s);
hipError_t launch_chunk_append(const ChunkAppendParams &p, hipStream_t s);
hipError_t launch_rope_append_fp8(const AppendFp8Params &p, const RopeDev &r, hipStream_t s);
hipError_t launch_chunk_prep_fp8(const PrepFp8Params &p, const RopeDev &r, hipStream_t s);
hipError_t launch_chunk_attn_fp8(const AttnFp8Params &p, int D, hipStream_t s);
hipError_t launch_chunk_append_fp8(const ChunkAppendFp8Params &p, hipStream_t s);
hipError_t launch_decode_split_fp8(const DecodeFp8Params &p, const RopeDev &r, hipStream_t s);
hipError_t launch_decode_combine_fp8(const DecodeFp8Params &p, hipStream_t s);
hipError_t launch_decode_split(const DecodeParams &p, const RopeDev &r, hipStream_t s);
hipError_t launch_decode_combine(const DecodeParams &p, hipStream_t s);

}  // namespace frt
