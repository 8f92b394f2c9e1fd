// FP8 (OCP e4m3fn) chunk attention: the FP8 KV-cache / FP8 QK^T-PV variant
// of chunk_attn_kernel, with the same blocks (8 waves x 32 query rows), the
// same runs of keys and edge-tile masks, the same software pipeline and the
// same lazily raised reference max, here kept an integer (and raised when a
// tile's max passes it by more than 1) so that the coded weights do not
// depend on it: they are code(2^(s - m + 7)), the largest near 2^7.
//
// Raising m does not rescale O: O and the normaliser stay relative to the
// reference max m0 of the row's first visible tile, and the PV products of
// later tiles are scaled up by 2^(m - m0), the E8M0 scale of the MFMA's B
// operand (one per column, i.e. per query row). Scaling by a power of two is
// exact, so this gives the same O / sum as rescaling O at every raise, and
// the output bits are the same; LSE takes m0. A row whose m climbs more than
// kFrameMax above m0 re-bases (one real rescale), which keeps O far inside
// the fp32 range.
//
// MFMA: v_mfma_f32_32x32x64_f8f6f4 with both operands e4m3. A lane holds 32
// bytes of each operand: lane l is row / column l % 32, and its half
// h = l / 32 owns 32 of the 64 k-slots. The two operands pair their slots the
// same way, so any consistent assignment of the contracted index to (h, byte)
// computes the product; the output layout is that of the 32x32 bf16 MFMA.
//
// S^T = K Q^T per 32-key block and 64-wide d step: A is K (LDS row rho holds
// the key perm(rho) of the block, 32 consecutive bytes of d per lane), B is
// the query codes (registers). perm moves bit 2 of the A row to bit 4, so the
// accumulator register r of a lane in half h holds key 16h + r: a lane's 32
// weights of a 64-key tile are keys 32kb + 16h + r, and they are the lane's B
// bytes of O^T = V^T P^T in register order. V^T comes from the ring's 32-key
// blocks, 16 bytes per (d row, 16 keys), two reads per MFMA. A fifth PV MFMA
// whose A operand is all ones gives sum_k p_k in fp32, the normaliser of the
// same coded weights.
//
// Scores: the MFMA gives q8 . k8; the score in base-2 units is that times
// 2^e_row * s_k (exact scaling by a power of two, then the key scale), folded
// into the fma that subtracts the reference max before exp2.
#include "frt_fp8.hpp"
#include "frt_launch.hpp"

namespace frt {
typedef int i32x4 __attribute__((ext_vector_type(4)));

namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));

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
__global__ __launch_bounds__(NW * 64) void chunk_attn_fp8_kernel(AttnFp8Params p) {
  constexpr int BN = kChunkBN;
  constexpr int BM = 32 * NW;
  constexpr int CPR = D / 16;                  // 16-byte chunks per K row
  constexpr int KDW = BN * CPR / 64 / NW;      // 1 KB LDS loads per wave per K tile
  constexpr int VDW = D * BN / 16 / 64 / NW;   // ... per V tile
  constexpr int NS = D / 64;                   // 64-wide d steps of S^T
  constexpr int SWZ = 16 / CPR;                // K rows sharing one swizzle value
  // Weights are coded at 2^kShift times their ratio to 2^m (m the integer
  // reference max): the largest lies in [2^(kShift-1), 2^kShift] when m is the
  // row's ceiling, and below 2^(kShift+kTau) while m lags by at most kTau, so
  // it never reaches 448; the first subnormal code sits 2^-13 under it.
  constexpr float kTau = 1.f;
  constexpr float kShift = 7.f;
  constexpr float kNegInf = -__builtin_inff();
  static_assert(BN == 64 && KDW >= 1 && VDW >= 1 && NS >= 1, "tile split");
  __shared__ __attribute__((aligned(16))) uint8_t ks0[BN * D];
  __shared__ __attribute__((aligned(16))) uint8_t ks1[BN * D];
  __shared__ __attribute__((aligned(16))) uint8_t vs0[D * BN];
  __shared__ __attribute__((aligned(16))) uint8_t vs1[D * BN];

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
      make_rsrc(p.k_ring + head * (size_t)C * D, (uint32_t)((size_t)C * D));
  const __amdgpu_buffer_rsrc_t rv_ring =
      make_rsrc(p.v_ring + head * (size_t)D * C, (uint32_t)((size_t)D * C));
  const __amdgpu_buffer_rsrc_t rk_own =
      make_rsrc(p.kr + head * (size_t)p.n_pad * D, (uint32_t)((size_t)p.n_pad * D));
  const __amdgpu_buffer_rsrc_t rv_own =
      make_rsrc(p.vt + head * (size_t)D * p.n_pad, (uint32_t)((size_t)D * p.n_pad));
  const float sk = p.sc.k[head], sv = p.sc.v[head];

  // query codes: B operand of S^T = K Q^T (row myrow, d bytes 64*s + 32*h ..)
  i32x8 qf[NS];
  float cq = 1.f;  // score scale of this row: 2^e * s_k (padding rows: any positive)
  {
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(p.qr + head * (size_t)rows * D, (uint32_t)((size_t)rows * D));
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      u32x4 lo = {0u, 0u, 0u, 0u}, hi = {0u, 0u, 0u, 0u};
      if (myrow < rows) {
        const uint32_t off = (uint32_t)((size_t)myrow * D + 64 * s + 32 * h);
        lo = buf_load16(rq, off);
        hi = buf_load16(rq, off + 16);
      }
      qf[s] = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                    (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
    }
    if (myrow < rows) cq = p.qs[head * (size_t)rows + myrow] * sk;
  }

  f32x16 o[D / 32], osum;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) osum[r] = 0.f;
  float m = 0.f;   // reference max, an integer
  bool mset = false;
  float m0 = 0.f;  // the reference max O and the normaliser are relative to
  int bsc = 127;   // E8M0 code of 2^(m - m0): the B scale of the PV MFMAs
  constexpr float kFrameMax = 64.f;
  const i32x8 ones8 = {0x38383838, 0x38383838, 0x38383838, 0x38383838,
                       0x38383838, 0x38383838, 0x38383838, 0x38383838};  // e4m3 1.0

  // ---- tile bookkeeping (block-uniform, scalar, branch free) ----
  // tile t: first key (slot, or own index for t >= c01) and fast flag
  const int dl0 = rf0, dl1 = rf1 - c0 * BN, dl2 = of - c01 * BN;
  auto tile_base = [&](int t) __attribute__((always_inline)) {
    return t * BN + pick(t < c0, dl0, pick(t < c01, dl1, dl2));
  };
  auto tile_fast = [&](int t) __attribute__((always_inline)) {
    return (t >= fa0 && t < fb0) || (t >= fa1 && t < fb1) || (t >= fa2 && t < fb2);
  };

  // ---- tile loads: HBM -> LDS directly, one wave instruction = 1 KB ----
  // K tile: LDS row rt (0..63) holds key 32*(rt/32) + perm(rt%32) of the tile,
  // its 16-byte chunk c at position c ^ ((rt / SWZ) % CPR): the 16 lanes of a
  // read pass then cover all 64 banks.
  // V tile: two 32-key blocks [d][32 bytes]; the half (16 keys) hh of row d
  // sits at position hh ^ ((d >> 3) & 1), again one pass over 64 banks.
  // Per-lane HBM offsets are fixed; the tile's first key is added per load.
  static_assert(BN % kVBlock == 0, "tiles start on V block boundaries");
  auto perm = [](int rho) { return (((rho >> 2) & 1) << 4) | (((rho >> 3) & 3) << 2) | (rho & 3); };
  uint32_t kdo[KDW], vdo[VDW];
#pragma unroll
  for (int u = 0; u < KDW; ++u) {
    const int pos = 64 * (wave * KDW + u) + lane;
    const int rt = pos / CPR, c = (pos % CPR) ^ ((rt / SWZ) % CPR);
    const int key = 32 * (rt / 32) + perm(rt % 32);
    kdo[u] = (uint32_t)(key * D + 16 * c);
  }
  auto vchunk = [&](int u, int &kb, int &d, int &hh) __attribute__((always_inline)) {
    const int pos = 64 * (wave * VDW + u) + lane;  // 16-byte position in the V tile
    kb = pos / (2 * D);
    d = (pos % (2 * D)) / 2;
    hh = (pos % 2) ^ ((d >> 3) & 1);
  };
#pragma unroll
  for (int u = 0; u < VDW; ++u) {
    int kb, d, hh;
    vchunk(u, kb, d, hh);
    vdo[u] = (uint32_t)(kVBlock * D * kb + kVBlock * d + 16 * hh);
  }
  const int vpart = C % kVBlock ? C - C % kVBlock : 0x7fffffff;
  auto dma_k = [&](int t, uint8_t *kbuf) __attribute__((always_inline)) {
    t = __builtin_amdgcn_readfirstlane(t);
    const bool own = t >= c01;
    const __amdgpu_buffer_rsrc_t rk = pick(own, rk_own, rk_ring);
    const uint32_t sb = (uint32_t)tile_base(t) * (uint32_t)D;
#pragma unroll
    for (int u = 0; u < KDW; ++u) dma16(rk, kdo[u] + sb, kbuf + 1024 * (wave * KDW + u));
  };
  auto dma_v = [&](int t, uint8_t *vbuf) __attribute__((always_inline)) {
    t = __builtin_amdgcn_readfirstlane(t);
    const bool own = t >= c01;
    const __amdgpu_buffer_rsrc_t rv = pick(own, rv_own, rv_ring);
    const int base = tile_base(t);
    if (!own && base + BN > vpart) {
      // the ring tile reaching the partial last block: per-lane offsets
#pragma unroll
      for (int u = 0; u < VDW; ++u) {
        int kb, d, hh;
        vchunk(u, kb, d, hh);
        dma16(rv, vring_elem(base + 32 * kb + 16 * hh, d, C, D), vbuf + 1024 * (wave * VDW + u));
      }
    } else {
      const uint32_t sb = (uint32_t)base * (uint32_t)D;
#pragma unroll
      for (int u = 0; u < VDW; ++u) dma16(rv, vdo[u] + sb, vbuf + 1024 * (wave * VDW + u));
    }
  };
  auto wait_dma = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  };

  // ---- per-wave compute pieces ----
  // K fragment: LDS row rt = 32*kb + l32, chunks 4s + 2h + {0, 1}, swizzled
  int kfo[NS][2];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      kfo[s][j] = l32 * D + 16 * ((4 * s + 2 * h + j) ^ ((l32 / SWZ) % CPR));
  // V fragment of d row 32*db + l32: 16 keys 16h.. of block kb (kb*32*D bytes on)
  const int vfo = l32 * 32 + 16 * (h ^ ((l32 >> 3) & 1));
  auto frag32 = [](const uint8_t *p0, const uint8_t *p1) __attribute__((always_inline)) {
    const i32x4 a = *reinterpret_cast<const i32x4 *>(p0);
    const i32x4 c = *reinterpret_cast<const i32x4 *>(p1);
    return (i32x8)__builtin_shufflevector(a, c, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  // raw S^T (q8 . k8) for the 64 keys of a K buffer
  auto qk = [&](const uint8_t *kt, f32x16 (&s)[2]) __attribute__((always_inline)) {
    const f32x16 zero = {};
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const uint8_t *kblk = kt + kb * 32 * D;
      s[kb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
          frag32(kblk + kfo[0][0], kblk + kfo[0][1]), qf[0], zero, 0, 0, 0, 0, 0, 0);
#pragma unroll
      for (int st = 1; st < NS; ++st)
        s[kb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            frag32(kblk + kfo[st][0], kblk + kfo[st][1]), qf[st], s[kb], 0, 0, 0, 0, 0, 0);
    }
  };
  // row max of the raw scores over the tile (one chain of three-input
  // maxima), then the lane 32 away
  auto row_max = [&](const f32x16 (&s)[2]) __attribute__((always_inline)) {
    float mt = fmaxf(fmaxf(s[0][0], s[0][1]), s[0][2]);
#pragma unroll
    for (int i = 3; i < 31; i += 2)
      mt = fmaxf(fmaxf(mt, s[i >> 4][i & 15]), s[(i + 1) >> 4][(i + 1) & 15]);
    mt = fmaxf(mt, s[1][15]);
    return max_pair32(mt);
  };
  // Edge-tile mask, branch free: register r of block kb is key 32kb + 16h + r.
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
        const int sl = base + 32 * kb + 16 * h + r;
        const int krel = sl - kbase - (sl >= hsplit ? C : 0);
        const bool ok = ((uint32_t)(sl - ra) < rspan) & ((uint32_t)(krel - vlo) <= vspan);
        s[kb][r] = ok ? s[kb][r] : kNegInf;
      }
  };
  // raise the reference max (an integer) when the tile's max exceeds it by
  // more than kTau, or at the row's first visible key; the products of later
  // weights carry 2^(m - m0) (see the head of the file)
  auto rescale = [&](float mraw) __attribute__((always_inline)) {
    const float mt = mraw * cq;
    const float rel = mt - m;
    const bool need = rel > kTau || (!mset && mt != kNegInf);
    if (__ballot(need)) {
      const float delta = need ? ceilf(rel) : 0.f;
      const float mn = m + delta;
      float m0n = mset ? m0 : mn;  // a row's first visible tile sets its frame
      const bool rebase = mn - m0n > kFrameMax;
      if (__ballot(rebase)) {
        const float alpha = rebase ? __builtin_amdgcn_exp2f(m0n - mn) : 1.f;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
#pragma unroll
        for (int r = 0; r < 16; ++r) osum[r] *= alpha;
        m0n = rebase ? mn : m0n;
      }
      m = mn;
      m0 = m0n;
      bsc = 127 + (int)(m - m0);
      mset = mset || need;
    }
  };
  // coded weights q8(2^(raw * cq - m + kShift)) of the tile, in B-operand order
  auto softmax = [&](const f32x16 (&s)[2], i32x8 &pf) __attribute__((always_inline)) {
    const float nm = kShift - m;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int r = 4 * w;
        pf[4 * kb + w] = (int)e4m3x4_inrange(__builtin_amdgcn_exp2f(fmaf(s[kb][r], cq, nm)),
                                     __builtin_amdgcn_exp2f(fmaf(s[kb][r + 1], cq, nm)),
                                     __builtin_amdgcn_exp2f(fmaf(s[kb][r + 2], cq, nm)),
                                     __builtin_amdgcn_exp2f(fmaf(s[kb][r + 3], cq, nm)));
      }
  };
  // O^T += V^T P^T and the normaliser for the 64 keys of a V buffer
  auto pv = [&](const uint8_t *vt, const i32x8 &pf) __attribute__((always_inline)) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const uint8_t *vrow = vt + db * 32 * 32 + vfo;
      o[db] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
          frag32(vrow, vrow + 32 * D), pf, o[db], 0, 0, 0, 127, 0, bsc);
    }
    osum = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ones8, pf, osum, 0, 0, 0, 127, 0, bsc);
  };

  auto step = [&](int t, const int par, f32x16 (&scur)[2], f32x16 (&snext)[2])
                  __attribute__((always_inline)) {
    dma_k(min(t + 2, T - 1), par ? ks1 : ks0);
    dma_v(t + 1, par ? vs0 : vs1);
    i32x8 pf;
    qk(par ? ks0 : ks1, snext);
    softmax(scur, pf);
#pragma unroll
    for (int i = 0; i < 2 * NS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // LDS read
      __builtin_amdgcn_sched_group_barrier(0x002, 16, 0);  // VALU
    }
    pv(par ? vs1 : vs0, pf);
    float mt = row_max(snext);
#pragma unroll
    for (int i = 0; i < D / 32 + 1; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // LDS read
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);  // VALU
    }
    if (!tile_fast(t + 1)) {
      mask_tile(t + 1, snext);
      mt = row_max(snext);
    }
    rescale(mt);
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
    rescale(row_max(sa));
    __syncthreads();  // K buffer 0 is refilled by the first step

    int t = 0;
    for (; t + 2 < T; t += 2) {
      step(t, 0, sa, sb);
      step(t + 1, 1, sb, sa);
    }
    i32x8 pf;
    if (t + 1 < T) {  // two tiles left (t is even)
      step(t, 0, sa, sb);
      softmax(sb, pf);
      pv(vs1, pf);
    } else {  // one tile left
      softmax(sa, pf);
      pv(vs0, pf);
    }
  }

  // out = s_v * O / l (both relative to m0); lse = (m0 - kShift + log2 l) * ln 2
  const float ltot = osum[0];
  if (myrow < rows) {
    const float f = sv / ltot;
    const int i = myrow / G, g = myrow % G;
    uint16_t *orow = p.out + (((size_t)b * n + i) * p.Hq + kvh * G + g) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d0 = 32 * db + 8 * q4 + 4 * h;
        u32x2 w;
        w[0] = f32_to_bf16_rne(o[db][4 * q4 + 0] * f) |
               (f32_to_bf16_rne(o[db][4 * q4 + 1] * f) << 16);
        w[1] = f32_to_bf16_rne(o[db][4 * q4 + 2] * f) |
               (f32_to_bf16_rne(o[db][4 * q4 + 3] * f) << 16);
        *reinterpret_cast<u32x2 *>(orow + d0) = w;
      }
    if (p.lse != nullptr && h == 0)
      p.lse[((size_t)b * p.Hq + kvh * G + g) * n + i] =
          (m0 - kShift + __builtin_amdgcn_logf(ltot)) * 0.6931471805599453f;
  }
}

}  // namespace

hipError_t launch_chunk_attn_fp8(const AttnFp8Params &p, int D, hipStream_t s) {
  const int nlog = p.row_tiles * p.Hkv * p.B;
  dim3 grid((nlog + 7) / 8 * 8);
  dim3 block(kChunkWaves * 64);
  if (D != 128) return hipErrorInvalidValue;  // the host API admits head_dim 128 only
  dispatch((chunk_attn_fp8_kernel<128, kChunkWaves>), grid, block, s, p);
  return hipGetLastError();
}

}  // namespace frt
