// FP8 (OCP e4m3fn) ring append and the FP8 step's chunk preparation.
//
// Codes: clamp to +-448, round to nearest, ties to even (the hardware
// conversion after an explicit clamp). A ring slot holds the key rotated in
// double, rounded to float, divided by the head's key scale in float, then
// coded; values are divided by the value scale and coded. Queries are kept in
// base-2 score units (rotated and multiplied by scale*log2(e) in double,
// rounded to float) and coded with a power-of-two scale per query row, the
// smallest 2^e with max|a| <= 448 * 2^e, so that the division is exact.
#include "frt_fp8.hpp"
#include "frt_launch.hpp"

namespace frt {

namespace {

// One block per 64 tokens of one (stream, KV head); the value codes go
// through LDS so that the block layout is written token-contiguous.
template <int D>
__global__ __launch_bounds__(256) void rope_append_fp8_kernel(AppendFp8Params p, RopeDev rope) {
  constexpr int CH = D / 8;
  constexpr int VS = D + 4;  // LDS row stride in bytes
  __shared__ uint8_t vs[kAppendTokens * VS];
  const RopeReg rg = rope_reg(rope);
  const int tb = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const long long L = p.seq_len[b];
  const int t0 = tb * kAppendTokens;
  const int ntok = min(kAppendTokens, p.n - t0);
  const size_t head = (size_t)b * p.Hkv + kvh;
  const float sk = p.sc.k[head], sv = p.sc.v[head];
  for (int idx = threadIdx.x; idx < kAppendTokens * CH; idx += 256) {
    const int r = idx / CH, c = idx % CH;
    if (r >= ntok) continue;
    const int i = t0 + r;
    const size_t src = (((size_t)b * p.n + i) * p.Hkv + kvh) * D + c * 8;
    const long long pos = L + i;
    int co[3];
    rope_coords(rg, pos, co);
    float y[8];
    rotate8_f32(rope_fetch4(rg, co, c * 4), *reinterpret_cast<const u32x4 *>(p.k_new + src), 1.0,
                y);
    const long long slot = pos % p.C;
    *reinterpret_cast<u32x2 *>(p.k_ring + (head * p.C + slot) * D + c * 8) = code8(y, sk);
    float v[8];
    bf16x8_to_f32(*reinterpret_cast<const u32x4 *>(p.v_new + src), v);
    *reinterpret_cast<u32x2 *>(vs + r * VS + c * 8) = code8(v, sv);
  }
  __syncthreads();
  const int r = threadIdx.x & 63;
  if (r < ntok) {
    const int slot = (int)((L + t0 + r) % p.C);
    uint8_t *vdst = p.v_ring + head * (size_t)D * p.C + vring_elem(slot, 0, p.C, D);
    const uint32_t w = vring_width(slot, p.C);
    for (int dd = threadIdx.x >> 6; dd < D; dd += 4) vdst[dd * w] = vs[r * VS + dd];
  }
}

template <int D>
__global__ __launch_bounds__(256) void chunk_prep_fp8_kernel(PrepFp8Params p, RopeDev rope) {
  constexpr int CH = D / 8;
  constexpr int VS = D + 4;
  static_assert(CH == 16 || CH == 8, "a query row is 8 or 16 lanes");
  __shared__ uint8_t vs[kAppendTokens * VS];
  const RopeReg rg = rope_reg(rope);
  const int tb = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const long long L = p.seq_len[b];
  const int t0 = tb * kAppendTokens;
  const size_t head = (size_t)b * p.Hkv + kvh;
  const float sk = p.sc.k[head], sv = p.sc.v[head];
  if (tb == 0 && kvh == 0 && threadIdx.x == 0) p.lrec[b] = L;

  // own key codes (as the ring will hold them) and value codes; zero padding
  for (int idx = threadIdx.x; idx < kAppendTokens * CH; idx += 256) {
    const int r = idx / CH, c = idx % CH;
    const int i = t0 + r;
    u32x2 kc = {0u, 0u}, vc = {0u, 0u};
    if (i < p.n) {
      const size_t src = (((size_t)b * p.n + i) * p.Hkv + kvh) * D + c * 8;
      int co[3];
      rope_coords(rg, L + i, co);
      float y[8];
      rotate8_f32(rope_fetch4(rg, co, c * 4), *reinterpret_cast<const u32x4 *>(p.k_new + src),
                  1.0, y);
      kc = code8(y, sk);
      float v[8];
      bf16x8_to_f32(*reinterpret_cast<const u32x4 *>(p.v_new + src), v);
      vc = code8(v, sv);
    }
    if (i < p.n_pad) *reinterpret_cast<u32x2 *>(p.kr + (head * p.n_pad + i) * D + c * 8) = kc;
    *reinterpret_cast<u32x2 *>(vs + r * VS + c * 8) = vc;
  }

  // queries: row i*G + g of this KV head; the CH lanes of a row are adjacent
  // lanes of one wave (CH divides 64 and the loop steps whole waves)
  const int G = p.G;
  const int rows_here = max(0, min(kAppendTokens, p.n - t0)) * G;
  for (int idx = threadIdx.x; idx < rows_here * CH; idx += 256) {
    const int rr = idx / CH, c = idx % CH;
    const int i = t0 + rr / G, g = rr % G;
    const size_t src = (((size_t)b * p.n + i) * p.Hq + kvh * G + g) * D + c * 8;
    int co[3];
    rope_coords(rg, L + i, co);
    float a[8];
    rotate8_f32(rope_fetch4(rg, co, c * 4), *reinterpret_cast<const u32x4 *>(p.q + src), p.qmul,
                a);
    float mx = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) mx = fmaxf(mx, fabsf(a[j]));
#pragma unroll
    for (int off = 1; off < CH; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    const int e = fp8_row_exponent(mx);
    float sa[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) sa[j] = ldexpf(a[j], -e);
    const size_t row = head * (size_t)p.n * G + (size_t)i * G + g;
    u32x2 qc;  // |sa| <= 448 by the choice of e
    qc[0] = e4m3x4_inrange(sa[0], sa[1], sa[2], sa[3]);
    qc[1] = e4m3x4_inrange(sa[4], sa[5], sa[6], sa[7]);
    *reinterpret_cast<u32x2 *>(p.qr + row * D + c * 8) = qc;
    if (c == 0) p.qs[row] = ldexpf(1.f, e);
  }
  __syncthreads();

  // value codes in the ring's block layout: 4 tokens x one row d per thread
  if (t0 < p.n_pad) {
    uint8_t *vbase = p.vt + head * (size_t)D * p.n_pad + (size_t)(t0 / kVBlock) * kVBlock * D;
    for (int idx = threadIdx.x; idx < (kAppendTokens / 4) * D; idx += 256) {
      const int quad = idx % (kAppendTokens / 4), dd = idx / (kAppendTokens / 4);
      const int r = 4 * quad;  // token within the block of 64
      const uint32_t w = (uint32_t)vs[r * VS + dd] | ((uint32_t)vs[(r + 1) * VS + dd] << 8) |
                         ((uint32_t)vs[(r + 2) * VS + dd] << 16) |
                         ((uint32_t)vs[(r + 3) * VS + dd] << 24);
      *reinterpret_cast<uint32_t *>(vbase + (size_t)(r / kVBlock) * kVBlock * D + dd * kVBlock +
                                    r % kVBlock) = w;
    }
  }
}

// The fused step's append: key rows copied from the codes the preparation
// pass wrote (kr), value codes re-blocked from its 32-token blocks (vt) at the
// ring's slots through LDS. seq_len is read by no block of this kernel (L
// comes from the record the preparation pass left), so one block per stream
// can advance it.
template <int D>
__global__ __launch_bounds__(256) void chunk_append_fp8_kernel(ChunkAppendFp8Params p) {
  constexpr int CH = D / 16;                // 16-byte chunks per key row
  constexpr int TS = kAppendTokens + 16;    // LDS row stride (bytes) of the [d][token] tile
  static_assert(kAppendTokens == 2 * kVBlock, "an append block is two value blocks");
  __shared__ __attribute__((aligned(16))) uint8_t vs[D * TS];
  const int tb = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const long long L = p.lrec[b];
  const int t0 = tb * kAppendTokens;
  const int ntok = min(kAppendTokens, p.n - t0);
  const size_t head = (size_t)b * p.Hkv + kvh;
  const uint8_t *krh = p.kr + head * (size_t)p.n_pad * D;
  for (int idx = threadIdx.x; idx < kAppendTokens * CH; idx += 256) {
    const int r = idx / CH, c = idx % CH;
    if (r >= ntok) continue;
    const int i = t0 + r;
    const int slot = (int)((L + i) % p.C);
    *reinterpret_cast<u32x4 *>(p.k_ring + (head * p.C + slot) * D + c * 16) =
        *reinterpret_cast<const u32x4 *>(krh + (size_t)i * D + c * 16);
  }
  // value codes of tokens t0 .. t0+63: two blocks [d][32] (n_pad is a
  // multiple of 64, so both lie inside the preparation pass's output)
  const uint8_t *vth = p.vt + head * (size_t)D * p.n_pad + (size_t)t0 * D;
  for (int idx = threadIdx.x; idx < 2 * D * 2; idx += 256) {
    const int kb = idx / (2 * D), d = (idx / 2) % D, h = idx % 2;
    *reinterpret_cast<u32x4 *>(vs + d * TS + kVBlock * kb + 16 * h) =
        *reinterpret_cast<const u32x4 *>(vth + (size_t)kb * kVBlock * D + d * kVBlock + 16 * h);
  }
  __syncthreads();
  const int r = threadIdx.x & 63;
  if (r < ntok) {
    const int slot = (int)((L + t0 + r) % p.C);
    uint8_t *vdst = p.v_ring + head * (size_t)D * p.C + vring_elem(slot, 0, p.C, D);
    const uint32_t w = vring_width(slot, p.C);
    for (int dd = threadIdx.x >> 6; dd < D; dd += 4) vdst[dd * w] = vs[dd * TS + r];
  }
  if (tb == 0 && kvh == 0 && threadIdx.x == 0) p.seq_len[b] = L + p.n;
}

}  // namespace

hipError_t launch_chunk_append_fp8(const ChunkAppendFp8Params &p, hipStream_t s) {
  dim3 grid((p.n + kAppendTokens - 1) / kAppendTokens, p.Hkv, p.B);
  if (p.D == 128)
    dispatch(chunk_append_fp8_kernel<128>, grid, dim3(256), s, p);
  else
    dispatch(chunk_append_fp8_kernel<64>, grid, dim3(256), s, p);
  return hipGetLastError();
}

hipError_t launch_rope_append_fp8(const AppendFp8Params &p, const RopeDev &r, hipStream_t s) {
  dim3 grid((p.n + kAppendTokens - 1) / kAppendTokens, p.Hkv, p.B);
  if (p.D == 128)
    dispatch(rope_append_fp8_kernel<128>, grid, dim3(256), s, p, r);
  else
    dispatch(rope_append_fp8_kernel<64>, grid, dim3(256), s, p, r);
  return hipGetLastError();
}

hipError_t launch_chunk_prep_fp8(const PrepFp8Params &p, const RopeDev &r, hipStream_t s) {
  dim3 grid((p.n_pad + kAppendTokens - 1) / kAppendTokens, p.Hkv, p.B);
  if (p.D == 128)
    dispatch(chunk_prep_fp8_kernel<128>, grid, dim3(256), s, p, r);
  else
    dispatch(chunk_prep_fp8_kernel<64>, grid, dim3(256), s, p, r);
  return hipGetLastError();
}

}  // namespace frt
