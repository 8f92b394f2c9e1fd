// Chunk-streamed attention: one block per (stream, KV head, tile of 32*NW
// query rows), rows ordered (token, query head of the group). Each wave owns
// 32 query rows and computes S^T = K Q^T with bf16 32x32x16 MFMAs, so every
// lane holds the scores of one query row: the online-softmax max and sum stay
// in the lane except for one exchange with the lane 32 away
// (v_permlane32_swap). O^T = V^T P^T reuses the score registers directly as
// the B operand.
//
// Keys come from up to three runs: at most two physical runs of ring slots
// (the visible token range wraps at most once) and the chunk's own keys,
// processed in tiles of 64 keys staged in LDS. Tiles wholly visible to every
// row of the block skip masking.
//
// Software pipeline. Iteration t issues the QK MFMAs of tile t+1 next to the
// softmax VALU work of tile t, then the PV MFMAs of tile t next to the row
// max of tile t+1, so each wave keeps the matrix pipe fed while it does its
// vector work. K therefore runs one tile ahead of V in LDS: iteration t reads
// K(t+1) and V(t) while the global loads of K(t+2) and V(t+1) are in flight
// (both double buffered). Masking of edge tiles and the rare rescale of the
// running max happen between iterations, outside that instruction stream.
//
// Operand layout. For the 32x32x16 MFMA the accumulator register r of lane l
// holds row 8*(r/4) + 4*(l/32) + r%4 and column l%32. The K tile row loaded
// as A-row rho is key 32*kb + perm(rho), perm swapping bits 2 and 3, which
// makes register r of key block kb hold key 32*kb + 16*(r/8) + 8*(l/32) + r%8:
// the 8 scores a lane feeds to one PV MFMA are 8 consecutive keys, so the V^T
// operand is one contiguous 16-byte LDS read.
//
// Online softmax in base-2 units (queries arrive pre-scaled by
// scale*log2(e)) with a lazily raised reference max m per row: m moves only
// when a tile's max exceeds it by more than kTau, or at the row's first
// visible key, so weights stay below 2^kTau and the O rescale is rare. The
// QK MFMA chain starts from -m in its accumulator, so the scores come out
// already relative to m and each weight costs one exp2 and no subtraction;
// a raise of m subtracts its step from the tile it was found in.
#include "frt_launch.hpp"

namespace frt {

namespace {


__device__ __forceinline__ int perm23(int x) {
  return (x & ~0xC) | ((x & 4) << 1) | ((x & 8) >> 1);
}

// max of x over lanes l and l^32
__device__ __forceinline__ float max_pair32(float x) {
  const u32x2 r = __builtin_bit_cast(
      u32x2, __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                              false));
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// sum of x over lanes l and l^32
__device__ __forceinline__ float sum_pair32(float x) {
  const u32x2 r = __builtin_bit_cast(
      u32x2, __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                              false));
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

typedef __attribute__((address_space(3))) void lds_void;

// 16-byte HBM -> LDS load; lane i of the wave writes lds_base + 16*i
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off,
                                      const void *lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)lds_base, 16, (int)byte_off, 0, 0, 0);
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void chunk_attn_kernel(AttnParams p) {
  constexpr int BN = kChunkBN;
  constexpr int BM = 32 * NW;
  constexpr int CPR = D / 8;                  // 16-byte chunks per K row
  constexpr int KDW = BN * CPR / 64 / NW;     // 1 KB LDS loads per wave per K tile
  constexpr int VDW = D * (BN / 8) / 64 / NW;  // ... per V^T tile
  constexpr float kTau = 8.f;
  constexpr float kNegInf = -__builtin_inff();
  static_assert(BN == 64 && KDW >= 1 && VDW >= 1, "tile split");
  __shared__ __attribute__((aligned(16))) uint16_t ks0[BN * D];
  __shared__ __attribute__((aligned(16))) uint16_t ks1[BN * D];
  __shared__ __attribute__((aligned(16))) uint16_t vs0[D * BN];
  __shared__ __attribute__((aligned(16))) uint16_t vs1[D * BN];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // scalar: LDS load bases in M0
  const int l32 = lane & 31, h = lane >> 5;

  // Blocks are dealt to the 8 XCDs round robin; give each XCD a contiguous
  // range of logical tiles (row tiles of one head are adjacent) so the
  // blocks sharing a head's K/V tiles share one L2.
  const int nlog = p.row_tiles * p.Hkv * p.B;
  const int jlog = (int)(blockIdx.x % 8) * (int)(gridDim.x / 8) + (int)(blockIdx.x / 8);
  if (jlog >= nlog) return;
  const int rt = jlog % p.row_tiles;
  const int kvh = (jlog / p.row_tiles) % p.Hkv;
  const int b = jlog / (p.row_tiles * p.Hkv);

  const long long L = p.seq_len[b];
  const int G = p.G, n = p.n, C = p.C;
  const int rows = n * G;
  const int row0 = rt * BM;
  const int myrow = row0 + wave * 32 + l32;
  const int i_lo = row0 / G;
  const int i_hi = (min(row0 + BM, rows) - 1) / G;

  // visibility, relative to L: this lane's row [vlo, vhi]; the block's union
  // [ulo, uhi] and intersection [ilo, ihi]
  long long lo, hi;
  visible_range(p.mask_kind, p.mask_block, p.mask_window, L + min(myrow, rows - 1) / G, lo, hi);
  const int vlo = clamp_i32(lo - L), vhi = clamp_i32(hi - L);
  visible_range(p.mask_kind, p.mask_block, p.mask_window, L + i_lo, lo, hi);
  const int ulo = clamp_i32(lo - L), ihi = clamp_i32(hi - L);
  visible_range(p.mask_kind, p.mask_block, p.mask_window, L + i_hi, lo, hi);
  const int ilo = clamp_i32(lo - L), uhi = clamp_i32(hi - L);

  const int lc = (int)(L < C ? L : (long long)C);  // ring tokens held
  const int hh = (int)(L % C);                      // slot of token L
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
  const int T = c0 + c1 + c2;

  const int c01 = c0 + c1;

  // Tiles wholly visible to every row of the block, as absolute tile index
  // ranges [fa_r, fb_r) per run; every other tile is masked. Keys of a run
  // map to relative tokens key = slot - off (one physical run never wraps).
  // A run holding slot hh strictly inside is the whole ring: it is fast only
  // if every row sees every ring token.
  const int klo = max(ilo, -lc), khi = min(ihi, -1);
  auto fast_range = [&](int ra, int re, int rf, int off, int kl, int kh, int t0, int nt, int &fa,
                        int &fb) __attribute__((always_inline)) {
    const int lo_s = max(ra, kl + off), hi_s = min(re - 1, kh + off);
    const int jmin = lo_s >= rf ? (lo_s - rf + BN - 1) / BN : 0;
    const int num = hi_s + 1 - rf;
    const int jend = num > 0 ? num / BN : 0;
    const int a = min(jmin, nt), e = max(a, min(jend, nt));
    fa = t0 + a;
    fb = t0 + e;
  };
  int fa0 = 0, fb0 = 0, fa1 = 0, fb1 = 0, fa2 = 0, fb2 = 0;
  if (c0 > 0) {
    if (ra0 < hh && hh < re0) {
      if (klo <= -C && khi >= -1) {
        fa0 = 0;
        fb0 = min(c0, (re0 - rf0) / BN);
      }
    } else {
      fast_range(ra0, re0, rf0, ra0 < hh ? hh : hh + C, klo, khi, 0, c0, fa0, fb0);
    }
  }
  if (c1 > 0) fast_range(ra1, re1, rf1, ra1 < hh ? hh : hh + C, klo, khi, c0, c1, fa1, fb1);
  if (c2 > 0) fast_range(oa, oe, of, 0, ilo, ihi, c01, c2, fa2, fb2);

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
  float m = 0.f, lsum = 0.f;
  bool mset = false;
  f32x16 negm = {};  // -m in every element: the accumulator the QK chain starts from

  // ---- tile bookkeeping (block-uniform, scalar, branch free) ----
  // tile t: first key (slot, or own index for t >= c01) and fast flag
  const int dl0 = rf0, dl1 = rf1 - c0 * BN, dl2 = of - c01 * BN;
  auto tile_base = [&](int t) __attribute__((always_inline)) {
    return t * BN + pick(t < c0, dl0, pick(t < c01, dl1, dl2));
  };
  auto tile_fast = [&](int t) __attribute__((always_inline)) {
    return (t >= fa0 && t < fb0) || (t >= fa1 && t < fb1) || (t >= fa2 && t < fb2);
  };

  // ---- tile loads: HBM -> LDS directly (no staging registers) ----
  // One wave instruction writes 1 KB of consecutive LDS; the HBM chunk each
  // lane fetches makes the LDS hold the tile XOR-swizzled, so that the MFMA
  // fragment reads below are free of bank conflicts:
  //   K tile:   LDS chunk (row, pc) holds key row `row`, d-chunk pc ^ (row % CPR)
  //   V^T tile: LDS chunk (d, pc) holds row d, key chunk pc ^ ((d >> 1) & 7)
  // Per-lane HBM offsets are fixed; the tile's first key is added per load, so
  // the buffer descriptors bound every access.
  // V (ring and own chunk alike) is stored in blocks of kVBlock keys, row d
  // of a block contiguous; a tile starts on a block boundary, so a lane's
  // chunk (d, c) sits at a fixed offset from the tile's first block. Only a
  // partial last ring block (C not a multiple of the block) breaks that.
  static_assert(BN % kVBlock == 0, "tiles start on V block boundaries");
  uint32_t kdo[KDW], vdo[VDW];
#pragma unroll
  for (int u = 0; u < KDW; ++u) {
    const int pos = 64 * (wave * KDW + u) + lane;
    const int row = pos / CPR, c = (pos % CPR) ^ (row % CPR);
    kdo[u] = (uint32_t)((row * D + 8 * c) * 2);
  }
  auto vchunk = [&](int u, int &d, int &c) __attribute__((always_inline)) {
    const int pos = 64 * (wave * VDW + u) + lane;
    d = pos / 8;
    c = (pos % 8) ^ ((d >> 1) & 7);
  };
#pragma unroll
  for (int u = 0; u < VDW; ++u) {
    int d, c;
    vchunk(u, d, c);
    vdo[u] = (uint32_t)((kVBlock * D * (8 * c / kVBlock) + kVBlock * d + 8 * c % kVBlock) * 2);
  }
  // first ring slot of a partial last block (no such block: never reached)
  const int vpart = C % kVBlock ? C - C % kVBlock : 0x7fffffff;
  auto dma_k = [&](int t, uint16_t *kb) __attribute__((always_inline)) {
    t = __builtin_amdgcn_readfirstlane(t);  // uniform: the descriptor stays scalar
    const bool own = t >= c01;
    const __amdgpu_buffer_rsrc_t rk = pick(own, rk_own, rk_ring);
    const uint32_t sb = (uint32_t)tile_base(t) * (uint32_t)(D * 2);
#pragma unroll
    for (int u = 0; u < KDW; ++u) dma16(rk, kdo[u] + sb, kb + 512 * (wave * KDW + u));
  };
  auto dma_v = [&](int t, uint16_t *vb) __attribute__((always_inline)) {
    t = __builtin_amdgcn_readfirstlane(t);
    const bool own = t >= c01;
    const __amdgpu_buffer_rsrc_t rv = pick(own, rv_own, rv_ring);
    const int base = tile_base(t);
    if (!own && base + BN > vpart) {
      // the ring tile reaching the partial last block: per-lane offsets; keys
      // past C land on later rows (masked) or past the descriptor (read 0)
#pragma unroll
      for (int u = 0; u < VDW; ++u) {
        int d, c;
        vchunk(u, d, c);
        dma16(rv, vring_elem(base + 8 * c, d, C, D) * 2u, vb + 512 * (wave * VDW + u));
      }
    } else {
      const uint32_t sb = (uint32_t)base * (uint32_t)(D * 2);
#pragma unroll
      for (int u = 0; u < VDW; ++u) dma16(rv, vdo[u] + sb, vb + 512 * (wave * VDW + u));
    }
  };
  // all of this thread's tile loads have landed in LDS
  auto wait_dma = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  };

  // ---- per-wave compute pieces ----
  const int prow = perm23(l32);
  // per-lane element offsets of the MFMA fragments inside a (swizzled) tile
  int kfo[D / 16];
#pragma unroll
  for (int k = 0; k < D / 16; ++k) kfo[k] = (prow * CPR + ((2 * k + h) ^ (prow % CPR))) * 8;
  int vfo[2][2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int j = 0; j < 2; ++j) vfo[kb][j] = (l32 * 8 + ((4 * kb + 2 * j + h) ^ ((l32 >> 1) & 7))) * 8;
  // S^T - m for the 64 keys of a K buffer. The two key blocks' chains are
  // issued alternately, each query fragment serving both in a row (1% faster
  // than one chain after the other; every chain sums in the same order).
  auto qk = [&](const uint16_t *kt, f32x16 (&s)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
      s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          *reinterpret_cast<const bf16x8 *>(kt + kb * 32 * D + kfo[0]), qf[0], negm, 0, 0, 0);
#pragma unroll
    for (int k = 1; k < D / 16; ++k)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            *reinterpret_cast<const bf16x8 *>(kt + kb * 32 * D + kfo[k]), qf[k], s[kb], 0, 0, 0);
  };
  // row max over the tile: one chain of three-input maxima (v_max3), then
  // the lane 32 away
  auto row_max = [&](const f32x16 (&s)[2]) __attribute__((always_inline)) {
    float mt = fmaxf(fmaxf(s[0][0], s[0][1]), s[0][2]);
#pragma unroll
    for (int i = 3; i < 31; i += 2)
      mt = fmaxf(fmaxf(mt, s[i >> 4][i & 15]), s[(i + 1) >> 4][(i + 1) & 15]);
    mt = fmaxf(mt, s[1][15]);
    return max_pair32(mt);
  };
  // Mask of an edge tile, branch free. Key (slot or own index) sl is visible to
  // this lane's row iff it lies in the tile's run and its token, relative to
  // L, lies in [vlo, vhi]; ring slots at or after hh hold tokens one ring
  // length further back.
  auto mask_tile = [&](int t, f32x16 (&s)[2]) __attribute__((always_inline)) {
    const int base = tile_base(t);
    const bool own = t >= c01, r0 = t < c0;
    const int ra = pick(r0, ra0, pick(own, oa, ra1));
    const int re = pick(r0, re0, pick(own, oe, re1));
    const int kbase = own ? 0 : hh;
    const int hsplit = own ? 0x7fffffff : hh;
    const uint32_t rspan = (uint32_t)(re - ra);
    const uint32_t vspan = (uint32_t)(vhi - vlo);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int sl = base + 32 * kb + 16 * (r >> 3) + 8 * h + (r & 7);
        const int krel = sl - kbase - (sl >= hsplit ? C : 0);
        const bool ok = ((uint32_t)(sl - ra) < rspan) & ((uint32_t)(krel - vlo) <= vspan);
        s[kb][r] = ok ? s[kb][r] : kNegInf;
      }
  };
  // raise the reference max when the tile's max exceeds it (rare, uniform
  // branch); mt is the max of the tile's scores sx, which are relative to m
  auto rescale = [&](float mt, f32x16 (&sx)[2]) __attribute__((always_inline)) {
    const float rel = mt;
    const bool need = rel > kTau || (!mset && mt != kNegInf);
    if (__ballot(need)) {
      const float delta = need ? rel : 0.f;
      // a row's first visible tile finds O and the sum still zero: alpha = 1
      // there, since exp2(-delta) overflows for a tile max below -128
      const float alpha = mset ? __builtin_amdgcn_exp2f(-delta) : 1.f;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      lsum *= alpha;
      m += delta;
      mset = mset || need;
#pragma unroll
      for (int r = 0; r < 16; ++r) negm[r] = -m;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sx[kb][r] -= delta;
    }
  };
  const bf16x2 ones = {(__bf16)1.f, (__bf16)1.f};
  auto softmax = [&](const f32x16 (&s)[2], bf16x8 (&pf)[2][2]) __attribute__((always_inline)) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        pf[kb][r >> 3][r & 7] = (__bf16)__builtin_amdgcn_exp2f(s[kb][r]);
    // row sum of the rounded weights the PV product uses
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const bf16x2 pr = {pf[kb][jj][2 * w], pf[kb][jj][2 * w + 1]};
          lsum = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, lsum, false);
        }
  };
  // O^T += V^T P^T for the 64 keys of a V^T buffer: each weight fragment
  // serves the D/32 output blocks in a row (each block sums in key order)
  auto pv = [&](const uint16_t *vt, const bf16x8 (&pf)[2][2]) __attribute__((always_inline)) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              *reinterpret_cast<const bf16x8 *>(vt + db * 32 * BN + vfo[kb][j]), pf[kb][j],
              o[db], 0, 0, 0);
  };

  // One pipelined iteration for a tile t that has a successor (par = t & 1):
  // QK(t+1) with softmax(t), PV(t) with max(t+1); K(t+2) and V(t+1) land in
  // the buffers tile t and tile t-1 left free.
  auto step = [&](int t, const int par, f32x16 (&scur)[2], f32x16 (&snext)[2])
                  __attribute__((always_inline)) {
    dma_k(min(t + 2, T - 1), par ? ks1 : ks0);
    dma_v(t + 1, par ? vs0 : vs1);
    bf16x8 pf[2][2];
    qk(par ? ks0 : ks1, snext);
    softmax(scur, pf);
    // QK(t+1) and softmax(t) are independent: interleave them
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // VALU
    }
    pv(par ? vs1 : vs0, pf);
    float mt = row_max(snext);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);  // VALU
    }
    if (!tile_fast(t + 1)) {
      mask_tile(t + 1, snext);
      mt = row_max(snext);
    }
    rescale(mt, snext);
    wait_dma();
    __syncthreads();
  };

  f32x16 sa[2], sb[2];
  if (T > 0) {
    dma_k(0, ks0);
    dma_v(0, vs0);
    dma_k(min(1, T - 1), ks1);
    wait_dma();
    __syncthreads();
    qk(ks0, sa);
    if (!tile_fast(0)) mask_tile(0, sa);
    rescale(row_max(sa), sa);
    __syncthreads();  // K buffer 0 is refilled by the first step

    int t = 0;
    for (; t + 2 < T; t += 2) {
      step(t, 0, sa, sb);
      step(t + 1, 1, sb, sa);
    }
    bf16x8 pf[2][2];
    if (t + 1 < T) {  // two tiles left (t is even)
      step(t, 0, sa, sb);
      softmax(sb, pf);
      pv(vs1, pf);
    } else {  // one tile left
      softmax(sa, pf);
      pv(vs0, pf);
    }
  }

  const float ltot = sum_pair32(lsum);
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
  const int nlog = p.row_tiles * p.Hkv * p.B;
  dim3 grid((nlog + 7) / 8 * 8);
  dim3 block(kChunkWaves * 64);
  if (D == 128)
    dispatch((chunk_attn_kernel<128, kChunkWaves>), grid, block, s, p);
  else
    dispatch((chunk_attn_kernel<64, kChunkWaves>), grid, block, s, p);
  return hipGetLastError();
}

}  // namespace frt
