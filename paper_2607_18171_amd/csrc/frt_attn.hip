// Chunk-streamed attention: one block per (stream, KV head, tile of 32*NW
// query rows), rows ordered (token, query head of the group). Each wave owns
// 32 query rows and computes S^T = K Q^T with bf16 32x32x16 MFMAs, so every
// lane holds the scores of one query row: the online-softmax max/sum stays in
// the lane except for one exchange with the lane 32 away. O^T = V^T P^T reuses
// the score registers directly as the B operand.
//
// Keys come from up to three runs: at most two physical runs of ring slots
// (the visible token range wraps at most once) and the chunk's own keys.
// Tiles of 64 keys are staged in LDS (double buffered: the next tile's global
// loads are issued before the current tile's MFMAs). Tiles wholly visible to
// every row of the block skip masking.
//
// Operand layout. For the 32x32x16 MFMA the accumulator register r of lane l
// holds row 8*(r/4) + 4*(l/32) + r%4 and column l%32. The K tile row loaded
// as A-row rho is key 32*kb + perm(rho), perm swapping bits 2 and 3, which
// makes register r of key block kb hold key 32*kb + 16*(r/8) + 8*(l/32) + r%8:
// the 8 scores a lane feeds to one PV MFMA are 8 consecutive keys, so the V^T
// operand is one contiguous 16-byte LDS read.
#include "frt_launch.hpp"

namespace frt {

namespace {

__device__ __forceinline__ int perm23(int x) {
  return (x & ~0xC) | ((x & 4) << 1) | ((x & 8) >> 1);
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void chunk_attn_kernel(AttnParams p) {
  constexpr int BN = kChunkBN;
  constexpr int BM = 32 * NW;
  constexpr int NT = NW * 64;
  constexpr int KST = D + 8;   // K tile row stride (elements)
  constexpr int VST = BN + 8;  // V^T tile row stride (elements)
  constexpr int KCH = BN * D / 8;
  constexpr int VCH = D * BN / 8;
  constexpr int KPT = KCH / NT;
  constexpr int VPT = VCH / NT;
  static_assert(KPT >= 1 && VPT >= 1, "tile too small for the block");
  __shared__ __attribute__((aligned(16))) uint16_t ks[2][BN * KST];
  __shared__ __attribute__((aligned(16))) uint16_t vs[2][D * VST];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  const int rt = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const long long L = p.seq_len[b];
  const int G = p.G, n = p.n, C = p.C;
  const int rows = n * G;
  const int row0 = rt * BM;
  const int myrow = row0 + wave * 32 + l32;
  const int myi = min(myrow, rows - 1) / G;
  const int i_lo = row0 / G;
  const int i_hi = (min(row0 + BM, rows) - 1) / G;

  // visibility, relative to L
  long long lo, hi;
  visible_range(p.mask_kind, p.mask_block, p.mask_window, L + myi, lo, hi);
  const int vlo = clamp_i32(lo - L), vhi = clamp_i32(hi - L);
  visible_range(p.mask_kind, p.mask_block, p.mask_window, L + i_lo, lo, hi);
  const int ulo = clamp_i32(lo - L), ihi = clamp_i32(hi - L);
  visible_range(p.mask_kind, p.mask_block, p.mask_window, L + i_hi, lo, hi);
  const int ilo = clamp_i32(lo - L), uhi = clamp_i32(hi - L);

  const int lc = (int)(L < C ? L : (long long)C);     // ring tokens held
  const int hh = (int)(L % C);                         // slot of token L
  // relative token of ring slot s: s-hh (s < hh) or s-hh-C (s >= hh)

  // runs of keys: ring run 0 [ra0, re0), ring run 1 [ra1, re1), own run [oa, oe)
  int ra0 = 0, re0 = 0, ra1 = 0, re1 = 0, oa = 0, oe = 0;
  {
    const int rlo = max(ulo, -lc), rhi = min(uhi, -1);
    if (rlo <= rhi) {
      const int cnt = rhi - rlo + 1;
      if (cnt == C) {
        re0 = C;
      } else {
        const int s0 = (int)((L + rlo) % C);
        ra0 = s0;
        if (s0 + cnt <= C) {
          re0 = s0 + cnt;
        } else {
          re0 = C;
          re1 = s0 + cnt - C;
        }
      }
    }
    const int olo = max(ulo, 0), ohi = min(uhi, n - 1);
    if (olo <= ohi) {
      oa = olo;
      oe = ohi + 1;
    }
  }
  const int rf0 = ra0 & ~(BN - 1), rf1 = ra1 & ~(BN - 1), of = oa & ~(BN - 1);
  const int c0 = re0 > ra0 ? (re0 - rf0 + BN - 1) / BN : 0;
  const int c1 = re1 > ra1 ? (re1 - rf1 + BN - 1) / BN : 0;
  const int c2 = oe > oa ? (oe - of + BN - 1) / BN : 0;

  const size_t head = (size_t)b * p.Hkv + kvh;
  const __amdgpu_buffer_rsrc_t rk_ring =
      make_rsrc(p.k_ring + head * (size_t)C * D, (uint32_t)((size_t)C * D * 2));
  const __amdgpu_buffer_rsrc_t rv_ring =
      make_rsrc(p.v_ring + head * (size_t)D * C, (uint32_t)((size_t)D * C * 2));
  const __amdgpu_buffer_rsrc_t rk_own =
      make_rsrc(p.kr + head * (size_t)p.n_pad * D, (uint32_t)((size_t)p.n_pad * D * 2));
  const __amdgpu_buffer_rsrc_t rv_own =
      make_rsrc(p.vt + head * (size_t)D * p.n_pad, (uint32_t)((size_t)D * p.n_pad * 2));

  // Q fragments: B operand of S^T = K Q^T (row myrow, d chunk 16*ks + 8*h)
  bf16x8 qf[D / 16];
  {
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(p.qr + head * (size_t)rows * D, (uint32_t)((size_t)rows * D * 2));
#pragma unroll
    for (int k = 0; k < D / 16; ++k) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (myrow < rows) v = buf_load16(rq, (uint32_t)(((size_t)myrow * D + 16 * k + 8 * h) * 2));
      qf[k] = __builtin_bit_cast(bf16x8, v);
    }
  }

  f32x16 o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m = -__builtin_inff();
  float lsum = 0.f;

  u32x4 kreg[KPT], vreg[VPT];

  // tile t -> run (0, 1: ring; 2: own) and first key (slot or own index)
  auto tile_of = [&](int t, int &run, int &base) {
    if (t < c0) {
      run = 0;
      base = rf0 + t * BN;
    } else if (t < c0 + c1) {
      run = 1;
      base = rf1 + (t - c0) * BN;
    } else {
      run = 2;
      base = of + (t - c0 - c1) * BN;
    }
  };

  auto load_tile = [&](int t) {
    int run, base;
    tile_of(t, run, base);
    if (run != 2) {
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        const int idx = tid + NT * u;
        const int kr = idx / (D / 8), kc = idx % (D / 8);
        kreg[u] = buf_load16(rk_ring, (uint32_t)(((size_t)(base + kr) * D + kc * 8) * 2));
      }
#pragma unroll
      for (int u = 0; u < VPT; ++u) {
        const int idx = tid + NT * u;
        const int dd = idx / (BN / 8), vc = idx % (BN / 8);
        vreg[u] = buf_load16(rv_ring, (uint32_t)(((size_t)dd * C + base + vc * 8) * 2));
      }
    } else {
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        const int idx = tid + NT * u;
        const int kr = idx / (D / 8), kc = idx % (D / 8);
        kreg[u] = buf_load16(rk_own, (uint32_t)(((size_t)(base + kr) * D + kc * 8) * 2));
      }
#pragma unroll
      for (int u = 0; u < VPT; ++u) {
        const int idx = tid + NT * u;
        const int dd = idx / (BN / 8), vc = idx % (BN / 8);
        vreg[u] = buf_load16(rv_own, (uint32_t)(((size_t)dd * p.n_pad + base + vc * 8) * 2));
      }
    }
  };

  auto store_tile = [&](int buf) {
#pragma unroll
    for (int u = 0; u < KPT; ++u) {
      const int idx = tid + NT * u;
      const int kr = idx / (D / 8), kc = idx % (D / 8);
      *reinterpret_cast<u32x4 *>(&ks[buf][kr * KST + kc * 8]) = kreg[u];
    }
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int idx = tid + NT * u;
      const int dd = idx / (BN / 8), vc = idx % (BN / 8);
      *reinterpret_cast<u32x4 *>(&vs[buf][dd * VST + vc * 8]) = vreg[u];
    }
  };

  const int T = c0 + c1 + c2;
  if (T > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();

  const int prow = perm23(l32);
  for (int t = 0; t < T; ++t) {
    const int buf = t & 1;
    if (t + 1 < T) load_tile(t + 1);

    int run, base;
    tile_of(t, run, base);
    const int ra = run == 0 ? ra0 : (run == 1 ? ra1 : oa);
    const int re = run == 0 ? re0 : (run == 1 ? re1 : oe);
    const bool own = run == 2;
    bool fast;
    if (own) {
      fast = base >= ra && base + BN <= re && base >= ilo && base + BN - 1 <= ihi;
    } else {
      const int end = base + BN;
      int kmin, kmax;
      if (base < hh && hh < end) {
        kmin = -C;
        kmax = -1;
      } else {
        kmin = base < hh ? base - hh : base - hh - C;
        kmax = (end - 1) < hh ? end - 1 - hh : end - 1 - hh - C;
      }
      fast = base >= ra && end <= re && end <= C && kmin >= max(ilo, -lc) && kmax <= ihi;
    }

    // S^T = K Q^T for two blocks of 32 keys
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
      const uint16_t *krow = &ks[buf][(32 * kb + prow) * KST + 8 * h];
#pragma unroll
      for (int k = 0; k < D / 16; ++k) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(krow + 16 * k);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[k], sacc[kb], 0, 0, 0);
      }
    }

    if (!fast) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int off = 32 * kb + 16 * (r >> 3) + 8 * h + (r & 7);
          const int s = base + off;
          bool ok;
          if (own) {
            ok = s >= ra && s < re && s >= vlo && s <= vhi;
          } else {
            const int krel = s < hh ? s - hh : s - hh - C;
            ok = s >= ra && s < re && s < C && krel >= -lc && krel >= vlo && krel <= vhi;
          }
          if (!ok) sacc[kb][r] = -__builtin_inff();
        }
      }
    }

    float mt = sacc[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, sacc[kb][r]);
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float mnew = fmaxf(m, mt);
    const float msafe = mnew == -__builtin_inff() ? 0.f : mnew;
    const float alpha = __builtin_amdgcn_exp2f(m - msafe);
    m = mnew;

    float ts = 0.f;
    bf16x8 pf[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = __builtin_amdgcn_exp2f(sacc[kb][r] - msafe);
        ts += e;
        pf[kb][r >> 3][r & 7] = (__bf16)e;
      }
    lsum = lsum * alpha + ts;
    if (__ballot(alpha != 1.f)) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    }

    // O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const uint16_t *vrow = &vs[buf][(32 * db + l32) * VST + 8 * h];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const bf16x8 vf = *reinterpret_cast<const bf16x8 *>(vrow + 32 * kb + 16 * j);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kb][j], o[db], 0, 0, 0);
        }
    }

    if (t + 1 < T) store_tile(buf ^ 1);
    __syncthreads();
  }

  const float ltot = lsum + __shfl_xor(lsum, 32);
  if (myrow < rows) {
    const float inv = 1.f / ltot;
    const int i = myrow / G, g = myrow % G;
    uint16_t *orow = p.out + (((size_t)b * n + i) * p.Hq + kvh * G + g) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d0 = 32 * db + 8 * q4 + 4 * h;
        u32x2 w;
        w[0] = f32_to_bf16_rne(o[db][4 * q4 + 0] * inv) |
               (f32_to_bf16_rne(o[db][4 * q4 + 1] * inv) << 16);
        w[1] = f32_to_bf16_rne(o[db][4 * q4 + 2] * inv) |
               (f32_to_bf16_rne(o[db][4 * q4 + 3] * inv) << 16);
        *reinterpret_cast<u32x2 *>(orow + d0) = w;
      }
    if (p.lse != nullptr && h == 0)
      p.lse[((size_t)b * p.Hq + kvh * G + g) * n + i] =
          (m + __builtin_amdgcn_logf(ltot)) * 0.6931471805599453f;
  }
}

}  // namespace

hipError_t launch_chunk_attn(const AttnParams &p, int D, hipStream_t s) {
  dim3 grid(p.row_tiles, p.Hkv, p.B);
  if (D == 128)
    hipLaunchKernelGGL((chunk_attn_kernel<128, kChunkWaves>), grid, dim3(kChunkWaves * 64), 0, s,
                       p);
  else
    hipLaunchKernelGGL((chunk_attn_kernel<64, kChunkWaves>), grid, dim3(kChunkWaves * 64), 0, s,
                       p);
  return hipGetLastError();
}

}  // namespace frt
