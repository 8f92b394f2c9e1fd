// One-token decode over the ring: split-KV partials, then a combine pass.
//
// Split pass: every wave owns one split of 256 ring slots of one (stream,
// KV head) and streams it as 8 tiles of 32 keys straight from HBM into MFMA
// operand registers (no LDS), software-pipelined two tiles deep: the loads of
// tile t+2 are issued as soon as tile t has been consumed, so each wave keeps
// its K/V stream in flight for the whole split. All G = Hq/Hkv query heads of
// the KV head are the columns of one 16x16x32 bf16 MFMA, so K and V are read
// once for the whole group. S^T = K Q^T puts one query per lane column; the K
// rows are loaded in the order that makes a lane's 8 scores 8 consecutive
// slots, so the V^T operand of O^T = V^T P^T is one 16-byte load. The wave
// writes its own partial (max, sum, unnormalised output); one more wave per
// (stream, KV head) writes the partial of the step's own token. Combine pass:
// one block per (query head, KV head, stream) rescales the live partials to
// the common max.
#include "frt_launch.hpp"

namespace frt {

namespace {

constexpr int kDecWaves = 4;                          // splits per block
constexpr int kDecTile = 32;                          // keys per tile
constexpr int kDecTiles = kDecodeSplit / kDecTile;    // tiles per split
constexpr float kNegInf = -__builtin_inff();
constexpr uint32_t kOob = 0x80000000u;  // >= every descriptor size (< 2^31)

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void decode_split_kernel(DecodeParams p,
                                                                                     RopeDev rope) {
  constexpr int NDB = D / 16;  // 16-row d blocks of O^T
  constexpr int NKS = D / 32;  // k-steps of S^T
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sp = blockIdx.x * kDecWaves + wave;  // this wave's split
  const int kvh = blockIdx.y, b = blockIdx.z;
  const int c16 = lane & 15, g4 = lane >> 4;
  const int G = p.G, C = p.C;
  if (sp > p.nsplit) return;
  const long long L = p.seq_len[b];
  const size_t head = (size_t)b * p.Hkv + kvh;

  if (sp == p.nsplit) {
    // Partial nsplit is the step's own token alone: score so = q . k with both
    // rotated and rounded as everywhere else (the key as the append will
    // store it), sum 1, output v_new. Query c16 = lane & 15, d chunk of lane
    // group g4 as in the split loop below.
    const RopeReg rg = rope_reg(rope);
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(p.q + ((size_t)b * p.Hq + kvh * G) * D, (uint32_t)(G * D * 2));
    const __amdgpu_buffer_rsrc_t rkn = make_rsrc(p.k_new + head * D, (uint32_t)(D * 2));
    int co[3];
    rope_coords(rg, L, co);
    float so = 0.f;
#pragma unroll
    for (int k = 0; k < NKS; ++k) {
      const int d0 = 32 * k + 8 * g4;
      const Rope4 rot = rope_fetch4(rg, co, d0 / 2);
      const u32x4 kr = rotate8_apply(rot, buf_load16(rkn, (uint32_t)(d0 * 2)), 1.0);
      const u32x4 qw = rotate8_apply(rot, buf_load16(rq, (uint32_t)((c16 * D + d0) * 2)), p.qmul);
#pragma unroll
      for (int w = 0; w < 4; ++w)
        so = __builtin_amdgcn_fdot2_f32_bf16(u32_as_bf16x2(qw[w]), u32_as_bf16x2(kr[w]), so, false);
    }
    so += __shfl_xor(so, 16);
    so += __shfl_xor(so, 32);
    float *part = p.ws + ((head * (p.nsplit + 1)) + sp) * decode_split_floats(G, D);
    if (c16 < G) {
      // lanes (c16, g4) write output elements d = 32*k + 8*g4 .. +8 of query c16
#pragma unroll
      for (int k = 0; k < NKS; ++k) {
        const int d0 = 32 * k + 8 * g4;
        const u32x4 v = *reinterpret_cast<const u32x4 *>(p.v_new + head * D + d0);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          part[2 * G + c16 * D + d0 + 2 * w] = bf16_bits_to_f32(v[w] & 0xFFFFu);
          part[2 * G + c16 * D + d0 + 2 * w + 1] = bf16_bits_to_f32(v[w] >> 16);
        }
      }
      if (g4 == 0) {
        part[c16] = so;
        part[G + c16] = 1.f;
      }
    }
    return;
  }

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

  const int s0 = sp * kDecodeSplit;
  float *part = p.ws + ((head * (p.nsplit + 1)) + sp) * decode_split_floats(G, D);
  if (!any_visible(s0, s0 + kDecodeSplit)) {
    // empty split: only the header, which the combine pass reads first
    if (lane < G) {
      part[lane] = kNegInf;
      part[G + lane] = 0.f;
    }
    return;
  }

  // Query fragment (B operand): query c16 (< G), d chunk 32*ks + 8*g4, so that
  // the four lane groups of one K load cover 64 contiguous bytes of a row.
  // Its raw values and rotary table entries are loaded first: vector loads
  // retire in order, so anything issued after the K/V stream would wait for it.
  // Columns c16 >= G read past the group's descriptor and get zeros.
  const RopeReg rg = rope_reg(rope);
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
  // Tile t of the split: slots s0 + 32t .. +32. A tile with no visible slot
  // (uniform) gets offsets past the descriptor: its loads return zeros
  // without touching memory and its compute is skipped.
  u32x4 kraw[2][2][NKS];
  u32x4 vraw[2][NDB];
  bool live[2];
  auto issue = [&](int t, int buf) __attribute__((always_inline)) {
    const int sb = s0 + t * kDecTile;
    const bool any = any_visible(sb, sb + kDecTile);
    live[buf] = any;
    // K rows: block kb, A-row rho = c16 -> slot sb + 8*(rho/4) + 4*kb + rho%4
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int slot = sb + 8 * (c16 >> 2) + 4 * kb + (c16 & 3);
#pragma unroll
      for (int k = 0; k < NKS; ++k) {
        const uint32_t off = (uint32_t)(((size_t)slot * D + 32 * k + 8 * g4) * 2);
        kraw[buf][kb][k] = buf_load16(rk, any ? off : kOob);
      }
    }
    // V^T rows: d = 16*db + c16, slots sb + 8*g4 .. +8
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const uint32_t off = (uint32_t)(((size_t)(16 * db + c16) * C + sb + 8 * g4) * 2);
      vraw[buf][db] = buf_load16(rv, any ? off : kOob);
    }
  };
  issue(0, 0);
  issue(1, 1);

  bf16x8 qf[NKS];
#pragma unroll
  for (int k = 0; k < NKS; ++k)
    qf[k] = __builtin_bit_cast(bf16x8, rotate8_apply(qrot[k], qraw[k], p.qmul));

  f32x4 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = kNegInf, lsum = 0.f;

#pragma unroll
  for (int t = 0; t < kDecTiles; ++t) {
    const int buf = t & 1;
    if (live[buf]) {
      const int sb = s0 + t * kDecTile;
      f32x4 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        sacc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < NKS; ++k)
          sacc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, kraw[buf][kb][k]), qf[k], sacc[kb], 0, 0, 0);
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
        o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, vraw[buf][db]), pf, o[db], 0, 0, 0);
      }
    }
    if (t + 2 < kDecTiles) issue(t + 2, buf);
  }

  // Split 0 also takes the step's own token: its key rotated and rounded as
  // the append will store it, its value as given.
  // partial: lane column c16 = query, O^T row (d) = 16*db + 4*g4 + r
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if (c16 < G) {
    float *orow = part + 2 * G + c16 * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r) orow[16 * db + 4 * g4 + r] = o[db][r];
    if (g4 == 0) {
      part[c16] = m;
      part[G + c16] = lsum;
    }
  }
}

// Combine pass: one block of D threads per (query head, KV head, stream);
// thread d owns output column d. The live partials (positive sum; the own
// token's always is) of a chunk of D splits are
// listed in LDS with their weights 2^(m_s - M); the output column then sums
// over the list with independent, coalesced row loads.
template <int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(DecodeParams p) {
  constexpr int NW = D / 64;  // waves per block
  __shared__ int lidx[D];
  __shared__ float lwt[D], lsm[D];
  __shared__ float red[NW];
  __shared__ int cnt[NW];

  const int q = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int G = p.G;
  const size_t head = (size_t)b * p.Hkv + kvh;
  const int hq = kvh * G + q;
  const size_t pstride = decode_split_floats(G, D);
  const int np = p.nsplit + 1;  // ring splits, then the own token
  const float *parts = p.ws + head * np * pstride;

  // common max over every live partial
  float mx = kNegInf;
  for (int s = t; s < np; s += D) {
    const float *pp = parts + s * pstride;
    if (pp[G + q] > 0.f) mx = fmaxf(mx, pp[q]);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  float M = kNegInf;
#pragma unroll
  for (int w = 0; w < NW; ++w) M = fmaxf(M, red[w]);

  float lt = 0.f, acc = 0.f;
  const float *orow = parts + 2 * G + (size_t)q * D + t;
  for (int base = 0; base < np; base += D) {
    const int s = base + t;
    float ls = 0.f, ms = 0.f;
    if (s < np) {
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
  dim3 grid((p.nsplit + 1 + kDecWaves - 1) / kDecWaves, p.Hkv, p.B);  // + the own-token wave
  if (p.D == 128)
    hipLaunchKernelGGL(decode_split_kernel<128>, grid, dim3(256), 0, s, p, r);
  else
    hipLaunchKernelGGL(decode_split_kernel<64>, grid, dim3(256), 0, s, p, r);
  return hipGetLastError();
}

hipError_t launch_decode_combine(const DecodeParams &p, hipStream_t s) {
  dim3 grid(p.G, p.Hkv, p.B);
  if (p.D == 128)
    hipLaunchKernelGGL(decode_combine_kernel<128>, grid, dim3(128), 0, s, p);
  else
    hipLaunchKernelGGL(decode_combine_kernel<64>, grid, dim3(64), 0, s, p);
  return hipGetLastError();
}

}  // namespace frt
