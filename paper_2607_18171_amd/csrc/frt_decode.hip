// One-token decode over the ring: split-KV partials, then a combine pass.
//
// Split pass: one block (4 waves) per (stream, KV head, 256 ring slots); a
// wave streams 64 slots as two tiles of 32 keys straight from HBM into MFMA
// operand registers (no LDS on the K/V path), issuing both tiles' loads
// before any arithmetic. All G = Hq/Hkv query heads of the KV head are the
// columns of one 16x16x32 bf16 MFMA, so K and V are read once for the whole
// group. S^T = K Q^T puts one query per lane column; the K rows are loaded in
// the order that makes a lane's 8 scores 8 consecutive slots, so the V^T
// operand of O^T = V^T P^T is one 16-byte load. The four waves merge their
// (max, sum, output) in LDS and the block writes one partial. Combine pass:
// one block per (query head, KV head, stream) rescales the live partials to
// the common max and adds the step's own token.
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

  const __amdgpu_buffer_rsrc_t rk = make_rsrc(p.k_ring + head * (size_t)C * D,
                                              (uint32_t)((size_t)C * D * 2));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(p.v_ring + head * (size_t)D * C,
                                              (uint32_t)((size_t)D * C * 2));

  auto krel_of = [&](int s) { return s < hh ? s - hh : s - hh - C; };
  // any visible slot in [s0, s1)? (uniform)
  auto any_visible = [&](int s0, int s1) {
    if (s0 >= C || rlo > -1) return false;
    const int se = min(s1, C) - 1;
    if (s0 < hh && hh <= se) return true;  // straddles the newest/oldest boundary
    return krel_of(se) >= rlo && krel_of(s0) <= -1;
  };

  float *part = p.ws + ((head * p.nsplit) + sp) * decode_split_floats(G, D);
  if (!any_visible(sp * kDecodeSplit, sp * kDecodeSplit + kDecodeSplit)) {
    // empty split: only the header, which the combine pass reads first
    if (threadIdx.x < G) {
      part[threadIdx.x] = kNegInf;
      part[G + threadIdx.x] = 0.f;
    }
    return;
  }

  // Query fragment (B operand): query c16 (< G), d chunk 32*ks + 8*g4, so that
  // the four lane groups of one K load cover 64 contiguous bytes of a row.
  // Its raw values and rotary table entries are loaded first: vector loads
  // retire in order, so anything issued after the K/V stream would wait for it.
  const RopeReg rg = rope_reg(rope);
  // Columns c16 >= G read past the group's descriptor and get zeros.
  u32x4 qraw[NKS];
  Rope4 qrot[NKS];
  {
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(p.q + ((size_t)b * p.Hq + kvh * G) * D, (uint32_t)(G * D * 2));
    int co[3];
    rope_coords(rg, L, co);
#pragma unroll
    for (int k = 0; k < NKS; ++k) {
      const int d0 = 32 * k + 8 * g4;
      qraw[k] = buf_load16(rq, (uint32_t)((c16 * D + d0) * 2));
      qrot[k] = rope_fetch4(rg, co, d0 / 2);
    }
  }

  // Issue every K/V load of the wave's two tiles before any arithmetic, so
  // 32 KB per wave are in flight while the query is rotated. A tile with no
  // visible slot (uniform per wave) gets an offset past the descriptor: its
  // loads return zeros without touching memory and its compute is skipped.
  constexpr uint32_t kOob = 0x80000000u;  // >= every descriptor size (< 2^31)
  bool live[2];
  u32x4 kraw[2][2][NKS];
  u32x4 vraw[2][NDB];
#pragma unroll
  for (int st = 0; st < 2; ++st) {
    const int sb = sp * kDecodeSplit + wave * 64 + st * 32;
    const bool any = any_visible(sb, sb + 32);
    live[st] = any;
    // K rows: block kb, A-row rho = c16 -> slot sb + 8*(rho/4) + 4*kb + rho%4
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int slot = sb + 8 * (c16 >> 2) + 4 * kb + (c16 & 3);
#pragma unroll
      for (int k = 0; k < NKS; ++k) {
        const uint32_t off = (uint32_t)(((size_t)slot * D + 32 * k + 8 * g4) * 2);
        kraw[st][kb][k] = buf_load16(rk, any ? off : kOob);
      }
    }
    // V^T rows: d = 16*db + c16, slots sb + 8*g4 .. +8
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const uint32_t off = (uint32_t)(((size_t)(16 * db + c16) * C + sb + 8 * g4) * 2);
      vraw[st][db] = buf_load16(rv, any ? off : kOob);
    }
  }

  bf16x8 qf[NKS];
#pragma unroll
  for (int k = 0; k < NKS; ++k)
    qf[k] = __builtin_bit_cast(bf16x8, rotate8_apply(qrot[k], qraw[k], p.qmul));

  f32x4 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = kNegInf, lsum = 0.f;

#pragma unroll
  for (int st = 0; st < 2; ++st) {
    if (!live[st]) continue;
    const int sb = sp * kDecodeSplit + wave * 64 + st * 32;
    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < NKS; ++k)
        sacc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, kraw[st][kb][k]), qf[k], sacc[kb], 0, 0, 0);
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
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vraw[st][db]),
                                                       pf, o[db], 0, 0, 0);
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
    // a split with no visible slot leaves its output rows unwritten: the
    // combine pass reads a row only when its sum is positive
    if (lt > 0.f) part[2 * G + q * D + d] = acc;
    if (d == 0) {
      part[q] = M;
      part[G + q] = lt;
    }
  }
}

// Combine pass: one block of D threads per (query head, KV head, stream);
// thread d owns output column d. The live partials (positive sum) of a chunk
// of D splits are listed in LDS with their weights 2^(m_s - M); the output
// column then sums over the list with independent, coalesced row loads.
template <int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(DecodeParams p, RopeDev rope) {
  constexpr int NW = D / 64;  // waves per block
  constexpr int CH = D / 8;   // 8-element chunks of a head vector
  __shared__ int lidx[D];
  __shared__ float lwt[D], lsm[D];
  __shared__ float red[NW];
  __shared__ int cnt[NW];
  __shared__ float sown;

  const int q = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int G = p.G;
  const size_t head = (size_t)b * p.Hkv + kvh;
  const int hq = kvh * G + q;
  const size_t pstride = decode_split_floats(G, D);
  const float *parts = p.ws + head * p.nsplit * pstride;

  // own-token score: the rotated, scaled, bf16 query (as the split pass
  // sees it) against the rotated bf16 key the append will store
  const RopeReg rg = rope_reg(rope);
  if (wave == 0) {
    float part = 0.f;
    if (lane < CH) {
      const long long L = p.seq_len[b];
      int co[3];
      rope_coords(rg, L, co);
      const u32x4 qx =
          *reinterpret_cast<const u32x4 *>(p.q + ((size_t)b * p.Hq + hq) * D + 8 * lane);
      const u32x4 kx = *reinterpret_cast<const u32x4 *>(p.k_new + head * D + 8 * lane);
      const u32x4 qy = rotate8_round(rg, co, 4 * lane, qx, p.qmul);
      const u32x4 ky = rotate8_round(rg, co, 4 * lane, kx, 1.0);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        part += bf16_bits_to_f32(qy[w] & 0xFFFFu) * bf16_bits_to_f32(ky[w] & 0xFFFFu);
        part += bf16_bits_to_f32(qy[w] >> 16) * bf16_bits_to_f32(ky[w] >> 16);
      }
    }
#pragma unroll
    for (int off = CH / 2; off >= 1; off >>= 1) part += __shfl_xor(part, off);
    if (lane == 0) sown = part;
  }

  // common max over the own score and every live partial
  float mx = kNegInf;
  for (int s = t; s < p.nsplit; s += D) {
    const float *pp = parts + s * pstride;
    if (pp[G + q] > 0.f) mx = fmaxf(mx, pp[q]);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  float M = sown;
#pragma unroll
  for (int w = 0; w < NW; ++w) M = fmaxf(M, red[w]);

  const float fo = __builtin_amdgcn_exp2f(sown - M);
  float lt = fo;
  float acc = fo * bf16_bits_to_f32(p.v_new[head * D + t]);
  const float *orow = parts + 2 * G + (size_t)q * D + t;
  for (int base = 0; base < p.nsplit; base += D) {
    const int s = base + t;
    float ls = 0.f, ms = 0.f;
    if (s < p.nsplit) {
      ls = parts[s * pstride + G + q];
      ms = parts[s * pstride + q];
    }
    const bool live = ls > 0.f;
    const uint64_t bal = __ballot(live);
    const int pos = __builtin_popcountll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) cnt[wave] = __builtin_popcountll(bal);
    __syncthreads();
    int off = 0, n = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      off += w < wave ? cnt[w] : 0;
      n += cnt[w];
    }
    if (live) {
      const float f = __builtin_amdgcn_exp2f(ms - M);
      lidx[off + pos] = s;
      lwt[off + pos] = f;
      lsm[off + pos] = ls * f;
    }
    __syncthreads();
    int i = 0;
    for (; i + 4 <= n; i += 4) {
      const float o0 = orow[lidx[i] * pstride], o1 = orow[lidx[i + 1] * pstride];
      const float o2 = orow[lidx[i + 2] * pstride], o3 = orow[lidx[i + 3] * pstride];
      acc += o0 * lwt[i] + o1 * lwt[i + 1] + o2 * lwt[i + 2] + o3 * lwt[i + 3];
      lt += lsm[i] + lsm[i + 1] + lsm[i + 2] + lsm[i + 3];
    }
    for (; i < n; ++i) {
      acc += orow[lidx[i] * pstride] * lwt[i];
      lt += lsm[i];
    }
    __syncthreads();
  }
  p.out[((size_t)b * p.Hq + hq) * D + t] = (uint16_t)f32_to_bf16_rne(acc / lt);
  if (t == 0 && p.lse != nullptr)
    p.lse[(size_t)b * p.Hq + hq] = (M + __builtin_amdgcn_logf(lt)) * 0.6931471805599453f;
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
  dim3 grid(p.G, p.Hkv, p.B);
  if (p.D == 128)
    hipLaunchKernelGGL(decode_combine_kernel<128>, grid, dim3(128), 0, s, p, r);
  else
    hipLaunchKernelGGL(decode_combine_kernel<64>, grid, dim3(64), 0, s, p, r);
  return hipGetLastError();
}

}  // namespace frt
