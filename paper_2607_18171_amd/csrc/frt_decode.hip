// One-token decode over the ring: split-KV partials, then a combine pass.
//
// Split pass: one block (4 waves) per (stream, KV head, 256 ring slots); a
// wave streams 64 slots as two tiles of 32 keys straight from HBM into MFMA
// operand registers (no LDS on the K/V path). All G = Hq/Hkv query heads of
// the KV head are the columns of one 16x16x32 bf16 MFMA, so K and V are read
// once for the whole group. S^T = K Q^T puts one query per lane column; the
// K rows are loaded in the order that makes a lane's 8 scores 8 consecutive
// slots, so the V^T operand of O^T = V^T P^T is one 16-byte load.
// The four waves merge their (max, sum, output) in LDS and the block writes
// one partial. Combine pass: one block per (stream, KV head) rescales every
// non-empty partial to the common max and adds the step's own token.
#include "frt_launch.hpp"

namespace frt {

namespace {

constexpr int kDecWaves = 4;
constexpr float kNegInf = -__builtin_inff();

template <int D>
__global__ __launch_bounds__(256) void decode_split_kernel(DecodeParams p, RopeDev rope) {
  constexpr int NDB = D / 16;  // 16-row d blocks of O^T
  constexpr int NKS = D / 32;  // k-steps of S^T
  __shared__ float wm[kDecWaves][16], wl[kDecWaves][16];
  __shared__ float wo[kDecWaves][16][D + 1];

  const int sp = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c16 = lane & 15, g4 = lane >> 4;
  const int G = p.G, C = p.C;
  const long long L = p.seq_len[b];
  const size_t head = (size_t)b * p.Hkv + kvh;

  // visible ring tokens for the query token L, relative to L: [rlo, -1]
  long long vlo, vhi;
  visible_range(p.mask_kind, p.mask_block, p.mask_window, L, vlo, vhi);
  const int lc = (int)(L < C ? L : (long long)C);
  const int rlo = max(clamp_i32(vlo - L), -lc);
  const int hh = (int)(L % C);

  // query fragment (B operand): query c16 (< G), d chunk (D/4)*g4 + 8*ks
  bf16x8 qf[NKS];
  {
    int co[3];
    rope_coords(rope, L, co);
#pragma unroll
    for (int k = 0; k < NKS; ++k) {
      u32x4 y = {0u, 0u, 0u, 0u};
      if (c16 < G) {
        const int d0 = (D / 4) * g4 + 8 * k;
        const u32x4 x = *reinterpret_cast<const u32x4 *>(
            p.q + ((size_t)b * p.Hq + kvh * G + c16) * D + d0);
        y = rotate8_round(rope, co, d0 / 2, x, p.qmul);
      }
      qf[k] = __builtin_bit_cast(bf16x8, y);
    }
  }

  const __amdgpu_buffer_rsrc_t rk = make_rsrc(p.k_ring + head * (size_t)C * D,
                                              (uint32_t)((size_t)C * D * 2));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(p.v_ring + head * (size_t)D * C,
                                              (uint32_t)((size_t)D * C * 2));

  f32x4 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = kNegInf, lsum = 0.f;

  auto krel_of = [&](int s) { return s < hh ? s - hh : s - hh - C; };

#pragma unroll
  for (int st = 0; st < 2; ++st) {
    const int sb = sp * kDecodeSplit + wave * 64 + st * 32;
    // skip a tile with no visible slot (uniform)
    bool any = false;
    if (sb < C && rlo <= -1) {
      const int se = min(sb + 32, C) - 1;
      if (sb < hh && hh <= se) {
        any = true;  // straddles the newest/oldest boundary
      } else {
        const int k0 = krel_of(sb), k1 = krel_of(se);
        any = k1 >= rlo && k0 <= -1;
      }
    }
    if (!any) continue;

    // K rows: block kb, A-row rho = c16 -> slot sb + 8*(rho/4) + 4*kb + rho%4
    u32x4 kraw[2][NKS];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int slot = sb + 8 * (c16 >> 2) + 4 * kb + (c16 & 3);
#pragma unroll
      for (int k = 0; k < NKS; ++k)
        kraw[kb][k] =
            buf_load16(rk, (uint32_t)(((size_t)slot * D + (D / 4) * g4 + 8 * k) * 2));
    }
    // V^T rows: d = 16*db + c16, slots sb + 8*g4 .. +8
    u32x4 vraw[NDB];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      vraw[db] = buf_load16(rv, (uint32_t)(((size_t)(16 * db + c16) * C + sb + 8 * g4) * 2));

    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < NKS; ++k)
        sacc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, kraw[kb][k]), qf[k], sacc[kb], 0, 0, 0);
    }
    // mask: score (kb, r) of lane group g4 is slot sb + 8*g4 + 4*kb + r
    float mt = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int s = sb + 8 * g4 + 4 * kb + r;
        const int kr = krel_of(s);
        const bool ok = s < C && kr >= rlo && kr <= -1;
        if (!ok) sacc[kb][r] = kNegInf;
        mt = fmaxf(mt, sacc[kb][r]);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float mnew = fmaxf(m, mt);
    const float msafe = mnew == kNegInf ? 0.f : mnew;
    const float alpha = __builtin_amdgcn_exp2f(m - msafe);
    m = mnew;
    bf16x8 pf;
    float ts = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float e = __builtin_amdgcn_exp2f(sacc[kb][r] - msafe);
        ts += e;
        pf[4 * kb + r] = (__bf16)e;
      }
    lsum = lsum * alpha + ts;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      o[db] *= alpha;
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vraw[db]), pf,
                                                       o[db], 0, 0, 0);
    }
  }

  // wave partial: lane column c16 = query, O^T row (d) = 16*db + 4*g4 + r
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if (lane < 16) {
    wm[wave][lane] = m;
    wl[wave][lane] = lsum;
  }
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 4; ++r) wo[wave][c16][16 * db + 4 * g4 + r] = o[db][r];
  __syncthreads();

  float *part = p.ws + ((head * p.nsplit) + sp) * decode_split_floats(G, D);
  for (int idx = threadIdx.x; idx < G * D; idx += 256) {
    const int q = idx / D, d = idx % D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, wm[w][q]);
    float acc = 0.f, lt = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w) {
        if (wl[w][q] > 0.f) {
          const float f = __builtin_amdgcn_exp2f(wm[w][q] - M);
          acc += wo[w][q][d] * f;
          lt += wl[w][q] * f;
        }
      }
    }
    part[2 * G + q * D + d] = acc;
    if (d == 0) {
      part[q] = M;
      part[G + q] = lt;
    }
  }
}

template <int D>
__global__ __launch_bounds__(256) void decode_combine_kernel(DecodeParams p, RopeDev rope) {
  constexpr int CH = D / 8;
  __shared__ float sown[16];
  const int kvh = blockIdx.x, b = blockIdx.y;
  const int G = p.G;
  const long long L = p.seq_len[b];
  const size_t head = (size_t)b * p.Hkv + kvh;

  // own-token score per query head: rotated, scaled, bf16 q (as the split
  // pass sees it) against the key the append will store
  {
    const int q = threadIdx.x / CH, c = threadIdx.x % CH;
    float part = 0.f;
    if (q < G) {
      int co[3];
      rope_coords(rope, L, co);
      const u32x4 qx = *reinterpret_cast<const u32x4 *>(
          p.q + ((size_t)b * p.Hq + kvh * G + q) * D + 8 * c);
      const u32x4 kx = *reinterpret_cast<const u32x4 *>(p.k_new + head * D + 8 * c);
      const u32x4 qy = rotate8_round(rope, co, 4 * c, qx, p.qmul);
      const u32x4 ky = rotate8_round(rope, co, 4 * c, kx, 1.0);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        part += bf16_bits_to_f32(qy[w] & 0xFFFFu) * bf16_bits_to_f32(ky[w] & 0xFFFFu);
        part += bf16_bits_to_f32(qy[w] >> 16) * bf16_bits_to_f32(ky[w] >> 16);
      }
    }
#pragma unroll
    for (int off = CH / 2; off >= 1; off >>= 1) part += __shfl_xor(part, off);
    if (q < G && c == 0) sown[q] = part;
  }
  __syncthreads();

  const float *parts = p.ws + head * p.nsplit * decode_split_floats(G, D);
  const size_t pstride = decode_split_floats(G, D);
  for (int idx = threadIdx.x; idx < G * D; idx += 256) {
    const int q = idx / D, d = idx % D;
    const float so = sown[q];
    float M = so;
    for (int s = 0; s < p.nsplit; ++s) {
      const float *pp = parts + s * pstride;
      if (pp[G + q] > 0.f) M = fmaxf(M, pp[q]);
    }
    const float fo = __builtin_amdgcn_exp2f(so - M);
    float lt = fo;
    float acc = fo * bf16_bits_to_f32(p.v_new[head * D + d]);
    for (int s = 0; s < p.nsplit; ++s) {
      const float *pp = parts + s * pstride;
      const float ls = pp[G + q];
      if (ls > 0.f) {
        const float f = __builtin_amdgcn_exp2f(pp[q] - M);
        lt += ls * f;
        acc += pp[2 * G + q * D + d] * f;
      }
    }
    const int hq = kvh * G + q;
    p.out[((size_t)b * p.Hq + hq) * D + d] = (uint16_t)f32_to_bf16_rne(acc / lt);
    if (d == 0 && p.lse != nullptr)
      p.lse[(size_t)b * p.Hq + hq] = (M + __builtin_amdgcn_logf(lt)) * 0.6931471805599453f;
  }
}

}  // namespace

hipError_t launch_decode_split(const DecodeParams &p, const RopeDev &r, hipStream_t s) {
  dim3 grid(p.nsplit, p.Hkv, p.B);
  if (p.D == 128)
    hipLaunchKernelGGL(decode_split_kernel<128>, grid, dim3(256), 0, s, p, r);
  else
    hipLaunchKernelGGL(decode_split_kernel<64>, grid, dim3(256), 0, s, p, r);
  return hipGetLastError();
}

hipError_t launch_decode_combine(const DecodeParams &p, const RopeDev &r, hipStream_t s) {
  dim3 grid(p.Hkv, p.B);
  if (p.D == 128)
    hipLaunchKernelGGL(decode_combine_kernel<128>, grid, dim3(256), 0, s, p, r);
  else
    hipLaunchKernelGGL(decode_combine_kernel<64>, grid, dim3(256), 0, s, p, r);
  return hipGetLastError();
}

}  // namespace frt
