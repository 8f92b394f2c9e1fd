// Ring append (RoPE'd K, transposed V, seq_len advance) and the per-step
// chunk preparation used by the attention kernel.
//
// Both kernels are HBM-bound copies with a rotation in double precision: each
// block owns 64 consecutive tokens of one (stream, KV head); rows are read and
// written as 16-byte vectors, and V is transposed through LDS so that the
// block layout of the V ring is written with consecutive lanes on consecutive
// slots.
#include "frt_launch.hpp"

namespace frt {

namespace {

template <int D>
__global__ __launch_bounds__(256) void rope_append_kernel(AppendParams p, RopeDev rope) {
  constexpr int CH = D / 8;           // 16-byte chunks per row
  constexpr int VS = D + 2;           // LDS row stride (elements), odd dword count
  __shared__ uint16_t vs[kAppendTokens * VS];
  const RopeReg rg = rope_reg(rope);
  const int tb = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const long long L = p.seq_len[b];
  const int t0 = tb * kAppendTokens;
  const int ntok = min(kAppendTokens, p.n - t0);
  const size_t head = (size_t)b * p.Hkv + kvh;

  for (int idx = threadIdx.x; idx < kAppendTokens * CH; idx += 256) {
    const int r = idx / CH, c = idx % CH;
    if (r >= ntok) continue;
    const int i = t0 + r;
    const size_t src = (((size_t)b * p.n + i) * p.Hkv + kvh) * D + c * 8;
    const long long pos = L + i;
    int co[3];
    rope_coords(rg, pos, co);
    const u32x4 x = *reinterpret_cast<const u32x4 *>(p.k_new + src);
    const u32x4 y = rotate8_round(rg, co, c * 4, x, 1.0);
    const long long slot = pos % p.C;
    *reinterpret_cast<u32x4 *>(p.k_ring + (head * p.C + slot) * D + c * 8) = y;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(p.v_new + src);
    uint32_t *dst = reinterpret_cast<uint32_t *>(vs + r * VS + c * 8);
    dst[0] = v[0];
    dst[1] = v[1];
    dst[2] = v[2];
    dst[3] = v[3];
  }
  __syncthreads();
  const int r = threadIdx.x & 63;
  if (r < ntok) {
    const int slot = (int)((L + t0 + r) % p.C);
    uint16_t *vdst = p.v_ring + head * (size_t)D * p.C + vring_elem(slot, 0, p.C, D);
    const uint32_t w = vring_width(slot, p.C);
    for (int dd = threadIdx.x >> 6; dd < D; dd += 4) vdst[dd * w] = vs[r * VS + dd];
  }
}

// Appends of a few tokens (n <= kAppendSmall, e.g. one decode token): one
// block per stream writes the slots of every KV head and then advances
// seq_len itself, once all of its threads are past their reads of it.
template <int D>
__global__ __launch_bounds__(256) void rope_append_small_kernel(AppendParams p, RopeDev rope) {
  constexpr int CH = D / 8;  // 16-byte chunks per row
  const RopeReg rg = rope_reg(rope);
  const int b = blockIdx.x;
  const long long L = p.seq_len[b];
  const int total = p.n * p.Hkv * CH;
  for (int idx = threadIdx.x; idx < total; idx += 256) {
    const int c = idx % CH, rest = idx / CH;
    const int kvh = rest % p.Hkv, i = rest / p.Hkv;
    const size_t src = (((size_t)b * p.n + i) * p.Hkv + kvh) * D + c * 8;
    const long long pos = L + i;
    int co[3];
    rope_coords(rg, pos, co);
    const u32x4 y = rotate8_round(rg, co, c * 4, *reinterpret_cast<const u32x4 *>(p.k_new + src),
                                  1.0);
    const long long slot = pos % p.C;
    const size_t head = (size_t)b * p.Hkv + kvh;
    *reinterpret_cast<u32x4 *>(p.k_ring + (head * p.C + slot) * D + c * 8) = y;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(p.v_new + src);
    uint16_t *vd = p.v_ring + head * (size_t)D * p.C + vring_elem((int)slot, c * 8, p.C, D);
    const uint32_t vw = vring_width((int)slot, p.C);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      vd[(2 * w) * vw] = (uint16_t)(v[w] & 0xFFFFu);
      vd[(2 * w + 1) * vw] = (uint16_t)(v[w] >> 16);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) p.seq_len[b] = L + p.n;
}

__global__ void seq_advance_kernel(int64_t *seq_len, int B, int n) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) seq_len[b] += n;
}

// T threads per block. A thread's items are independent, so their loads are
// issued together before any of them is rotated: the pass is a few memory
// round trips per block, and with GQA (G query rows per key) most of its
// work is queries, which a 1024-thread block spreads four items a thread.
template <int D, int T>
__global__ __launch_bounds__(T) void chunk_prep_kernel(PrepParams p, RopeDev rope) {
  constexpr int CH = D / 8;
  constexpr int VS = D + 2;
  constexpr int KU = (kAppendTokens * CH + T - 1) / T;  // own-token items per thread
  constexpr int QU = 4;                                   // query items per loop pass
  __shared__ uint16_t vs[kAppendTokens * VS];
  const RopeReg rg = rope_reg(rope);
  const int tb = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const long long L = p.seq_len[b];
  const int t0 = tb * kAppendTokens;
  const size_t head = (size_t)b * p.Hkv + kvh;
  if (tb == 0 && kvh == 0 && threadIdx.x == 0) p.lrec[b] = L;

  // own keys (stored-key rounding) and values into LDS; zero padding rows
  u32x4 kx[KU], vx[KU];
#pragma unroll
  for (int u = 0; u < KU; ++u) {
    const int idx = threadIdx.x + T * u;
    const int r = idx / CH, c = idx % CH;
    const int i = t0 + r;
    kx[u] = u32x4{0u, 0u, 0u, 0u};
    vx[u] = u32x4{0u, 0u, 0u, 0u};
    if (idx < kAppendTokens * CH && i < p.n) {
      const size_t src = (((size_t)b * p.n + i) * p.Hkv + kvh) * D + c * 8;
      kx[u] = *reinterpret_cast<const u32x4 *>(p.k_new + src);
      vx[u] = *reinterpret_cast<const u32x4 *>(p.v_new + src);
    }
  }
#pragma unroll
  for (int u = 0; u < KU; ++u) {
    const int idx = threadIdx.x + T * u;
    if (idx >= kAppendTokens * CH) break;
    const int r = idx / CH, c = idx % CH;
    const int i = t0 + r;
    u32x4 y = {0u, 0u, 0u, 0u};
    if (i < p.n) {
      int co[3];
      rope_coords(rg, L + i, co);
      y = rotate8_round(rg, co, c * 4, kx[u], 1.0);
    }
    if (i < p.n_pad)
      *reinterpret_cast<u32x4 *>(p.kr + (head * p.n_pad + i) * D + c * 8) = y;
    uint32_t *dst = reinterpret_cast<uint32_t *>(vs + r * VS + c * 8);
    dst[0] = vx[u][0];
    dst[1] = vx[u][1];
    dst[2] = vx[u][2];
    dst[3] = vx[u][3];
  }

  // queries: row i*G + g of this KV head, rotated and scaled
  const int G = p.G;
  const int items = max(0, min(kAppendTokens, p.n - t0)) * G * CH;
  for (int base = threadIdx.x; base < items; base += T * QU) {
    u32x4 qx[QU];
#pragma unroll
    for (int u = 0; u < QU; ++u) {
      const int idx = base + T * u;
      qx[u] = u32x4{0u, 0u, 0u, 0u};
      if (idx < items) {
        const int rr = idx / CH, c = idx % CH;
        const int i = t0 + rr / G, g = rr % G;
        qx[u] = *reinterpret_cast<const u32x4 *>(
            p.q + (((size_t)b * p.n + i) * p.Hq + kvh * G + g) * D + c * 8);
      }
    }
#pragma unroll
    for (int u = 0; u < QU; ++u) {
      const int idx = base + T * u;
      if (idx < items) {
        const int rr = idx / CH, c = idx % CH;
        const int i = t0 + rr / G, g = rr % G;
        int co[3];
        rope_coords(rg, L + i, co);
        const u32x4 y = rotate8_round(rg, co, c * 4, qx[u], p.qmul);
        *reinterpret_cast<u32x4 *>(p.qr + (head * p.n * G + (size_t)i * G + g) * D + c * 8) = y;
      }
    }
  }
  __syncthreads();

  // values in the V ring's block layout (n_pad is a multiple of the block, so
  // every block is full): token pairs (2 per thread) x D rows
  if (t0 < p.n_pad) {
    const int ip = threadIdx.x & 31;
    const int s = t0 + 2 * ip;
    uint16_t *vbase = p.vt + head * (size_t)D * p.n_pad + (size_t)(s / kVBlock) * kVBlock * D +
                      s % kVBlock;
    for (int dd = threadIdx.x >> 5; dd < D; dd += T / 32) {
      const uint32_t lo = vs[(2 * ip) * VS + dd], hi = vs[(2 * ip + 1) * VS + dd];
      *reinterpret_cast<uint32_t *>(vbase + dd * kVBlock) = lo | (hi << 16);
    }
  }
}

// The append half of a fused step: the chunk's keys are already rotated and
// rounded exactly as frt_kv_append stores them, so they are copied; values
// take the transposing path of rope_append_kernel. seq_len is read by no
// block of this kernel (L comes from the record the preparation pass left),
// so one block per stream can advance it.
template <int D>
__global__ __launch_bounds__(256) void chunk_append_kernel(ChunkAppendParams p) {
  constexpr int CH = D / 8;  // 16-byte chunks per row
  constexpr int VS = D + 2;  // LDS row stride (elements), odd dword count
  __shared__ uint16_t vs[kAppendTokens * VS];
  const int tb = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const long long L = p.lrec[b];
  const int t0 = tb * kAppendTokens;
  const int ntok = min(kAppendTokens, p.n - t0);
  const size_t head = (size_t)b * p.Hkv + kvh;
  const uint16_t *krh = p.kr + head * (size_t)p.n_pad * D;
  for (int idx = threadIdx.x; idx < kAppendTokens * CH; idx += 256) {
    const int r = idx / CH, c = idx % CH;
    if (r >= ntok) continue;
    const int i = t0 + r;
    const int slot = (int)((L + i) % p.C);
    *reinterpret_cast<u32x4 *>(p.k_ring + (head * p.C + slot) * D + c * 8) =
        *reinterpret_cast<const u32x4 *>(krh + (size_t)i * D + c * 8);
    const u32x4 v =
        *reinterpret_cast<const u32x4 *>(p.v_new + (((size_t)b * p.n + i) * p.Hkv + kvh) * D + c * 8);
    uint32_t *dst = reinterpret_cast<uint32_t *>(vs + r * VS + c * 8);
    dst[0] = v[0];
    dst[1] = v[1];
    dst[2] = v[2];
    dst[3] = v[3];
  }
  __syncthreads();
  const int r = threadIdx.x & 63;
  if (r < ntok) {
    const int slot = (int)((L + t0 + r) % p.C);
    uint16_t *vdst = p.v_ring + head * (size_t)D * p.C + vring_elem(slot, 0, p.C, D);
    const uint32_t w = vring_width(slot, p.C);
    for (int dd = threadIdx.x >> 6; dd < D; dd += 4) vdst[dd * w] = vs[r * VS + dd];
  }
  if (tb == 0 && kvh == 0 && threadIdx.x == 0) p.seq_len[b] = L + p.n;
}

}  // namespace

hipError_t launch_chunk_append(const ChunkAppendParams &p, hipStream_t s) {
  dim3 grid((p.n + kAppendTokens - 1) / kAppendTokens, p.Hkv, p.B);
  if (p.D == 128)
    dispatch(chunk_append_kernel<128>, grid, dim3(256), s, p);
  else
    dispatch(chunk_append_kernel<64>, grid, dim3(256), s, p);
  return hipGetLastError();
}

hipError_t launch_rope_append(const AppendParams &p, const RopeDev &r, hipStream_t s) {
  dim3 grid((p.n + kAppendTokens - 1) / kAppendTokens, p.Hkv, p.B);
  if (p.D == 128)
    dispatch(rope_append_kernel<128>, grid, dim3(256), s, p, r);
  else
    dispatch(rope_append_kernel<64>, grid, dim3(256), s, p, r);
  return hipGetLastError();
}

hipError_t launch_rope_append_small(const AppendParams &p, const RopeDev &r, hipStream_t s) {
  if (p.D == 128)
    dispatch(rope_append_small_kernel<128>, dim3(p.B), dim3(256), s, p, r);
  else
    dispatch(rope_append_small_kernel<64>, dim3(p.B), dim3(256), s, p, r);
  return hipGetLastError();
}

hipError_t launch_seq_advance(int64_t *seq_len, int B, int n, hipStream_t s) {
  dispatch(seq_advance_kernel, dim3((B + 255) / 256), dim3(256), s, seq_len, B, n);
  return hipGetLastError();
}

hipError_t launch_chunk_prep(const PrepParams &p, const RopeDev &r, hipStream_t s) {
  dim3 grid((p.n_pad + kAppendTokens - 1) / kAppendTokens, p.Hkv, p.B);
  // GQA steps carry G query rows per key: four waves per block would leave
  // the pass waiting on memory (prefill, G = 4: 22.7 against 12.9 us)
  const bool wide = p.G >= 4;
  if (p.D == 128) {
    if (wide) dispatch(chunk_prep_kernel<128, 1024>, grid, dim3(1024), s, p, r);
    else dispatch(chunk_prep_kernel<128, 256>, grid, dim3(256), s, p, r);
  } else {
    if (wide) dispatch(chunk_prep_kernel<64, 1024>, grid, dim3(1024), s, p, r);
    else dispatch(chunk_prep_kernel<64, 256>, grid, dim3(256), s, p, r);
  }
  return hipGetLastError();
}

}  // namespace frt
