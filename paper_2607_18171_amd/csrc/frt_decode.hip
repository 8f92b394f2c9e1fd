// One-token decode over the ring: stream-K split pass, then a combine pass.
//
// Work. For stream b the query is token L = seq_len[b]; its visible ring
// tokens [lo, L-1] are covered by n_b tiles of 32 tokens aligned to
// multiples of 32 (token t lives in slot t mod C). Every (stream, KV head) is
// cut into pc pieces of at most `per` tiles, `per` chosen from the total so
// that the pieces spread evenly over the waves resident on the GPU at once;
// piece j takes every pc-th tile from tile j, so that the waves of one head
// read neighbouring memory at any moment. Wave k of the split pass streams
// piece k and writes its partial to slot k. One more wave per (stream, KV head) writes the partial of the
// step's own token.
//
// Split pass tiles stream straight from HBM into MFMA operand registers (no
// LDS), software-pipelined kDecBufs tiles deep. All G = Hq/Hkv query heads of the
// KV head are the columns of one 16x16x32 bf16 MFMA, so K and V are read once
// for the whole group. S^T = K Q^T puts one query per lane column; the K rows
// are loaded in the order that makes a lane's 8 scores 8 consecutive tokens,
// so the V^T operand of O^T = V^T P^T is one 16-byte load (8 consecutive
// tokens start at a slot that is a multiple of 8, and C is too, so they never
// wrap or leave their V block). With C a multiple of 32 a tile is exactly one
// V block: 64*D contiguous bytes. Combine pass: one block per (stream, KV
// head) loads the head's partials in groups, rescales them to their common
// max and normalises.
#include "frt_decode_pieces.hpp"

namespace frt {

namespace {

// Own-token partial slot (32-bit words): max[G], sum[G] (= 1), then, where a
// piece's outputs start, the head's piece range {K, np}, the query token L as
// two words, and the key as the ring stores it (D/2 words of bf16 pairs). Its
// output row is v_new, which the combine pass reads from the input.
constexpr int kOwnHdr = 4;

constexpr bf16x2 kOnes2 = {(__bf16)1.f, (__bf16)1.f};

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kDecWavesPerSimd))) void decode_split_kernel(
    DecodeParams p, RopeDev rope) {
  constexpr int NDB = D / 16;  // 16-row d blocks of O^T
  constexpr int NKS = D / 32;  // k-steps of S^T
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c16 = lane & 15, g4 = lane >> 4;
  const int G = p.G, C = p.C, H = p.B * p.Hkv;
  const size_t pfl = decode_split_floats(G, D);
  const RopeReg rg = rope_reg(rope);

  // query fragment of (stream b, KV head kvh) at token L: B operand, query
  // c16 (< G), d chunk 32*ks + 8*g4 (the four lane groups of one K load cover
  // 64 contiguous bytes of a row); columns c16 >= G read past the
  // descriptor and get zeros
  auto query_frag = [&](int b, int kvh, long long L, bf16x8 (&qf)[NKS])
                        __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(p.q + ((size_t)b * p.Hq + kvh * G) * D, (uint32_t)(G * D * 2));
    int co[3];
    rope_coords(rg, L, co);
#pragma unroll
    for (int k = 0; k < NKS; ++k) {
      const int d0 = 32 * k + 8 * g4;
      const Rope4 rot = rope_fetch4(rg, co, d0 / 2);
      const u32x4 x = buf_load16(rq, (uint32_t)((c16 * D + d0) * 2));
      qf[k] = __builtin_bit_cast(bf16x8, rotate8_apply(rot, x, p.qmul));
    }
  };

  const int own_first = p.nwaves / kDecWaves;  // blocks from here write own-token partials
  if ((int)blockIdx.x >= own_first) {
    // Partial of the step's own token alone: score = q . k with both rotated
    // and rounded as everywhere else (the key as the append will store it),
    // sum 1, output v_new; plus what the combine pass needs of this head.
    const int h = ((int)blockIdx.x - own_first) * kDecWaves + wave;
    if (h >= H) return;
    const int b = h / p.Hkv, kvh = h % p.Hkv;
    const long long L = p.seq_len[b];
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(p.q + ((size_t)b * p.Hq + kvh * G) * D, (uint32_t)(G * D * 2));
    const __amdgpu_buffer_rsrc_t rkn = make_rsrc(p.k_new + (size_t)h * D, (uint32_t)(D * 2));
    int co[3];
    rope_coords(rg, L, co);
    float so = 0.f;
    u32x4 krot[NKS];
#pragma unroll
    for (int k = 0; k < NKS; ++k) {
      const int d0 = 32 * k + 8 * g4;
      const Rope4 rot = rope_fetch4(rg, co, d0 / 2);
      const u32x4 kr = rotate8_apply(rot, buf_load16(rkn, (uint32_t)(d0 * 2)), 1.0);
      krot[k] = kr;
      const u32x4 qw = rotate8_apply(rot, buf_load16(rq, (uint32_t)((c16 * D + d0) * 2)), p.qmul);
#pragma unroll
      for (int w = 0; w < 4; ++w)
        so = __builtin_amdgcn_fdot2_f32_bf16(u32_as_bf16x2(qw[w]), u32_as_bf16x2(kr[w]), so, false);
    }
    so += __shfl_xor(so, 16);
    so += __shfl_xor(so, 32);
    int K, np;
    head_pieces(p, lane, b, kvh, K, np);
    float *part = p.ws + (size_t)(p.nwaves + h) * pfl;
    uint32_t *hdr = reinterpret_cast<uint32_t *>(part + decode_out_off(G));
    if (c16 < G && g4 == 0) {
      part[c16] = so;
      part[G + c16] = 1.f;
    }
    if (lane == 0) {
      hdr[0] = (uint32_t)K;
      hdr[1] = (uint32_t)np;
      hdr[2] = (uint32_t)(unsigned long long)L;
      hdr[3] = (uint32_t)((unsigned long long)L >> 32);
    }
    if (c16 == 0) {
      // the rotated key (every c16 holds it): d chunk 32*k + 8*g4
#pragma unroll
      for (int k = 0; k < NKS; ++k) {
        const int d0 = 32 * k + 8 * g4;
#pragma unroll
        for (int w = 0; w < 4; ++w) hdr[kOwnHdr + d0 / 2 + w] = krot[k][w];
      }
    }
    return;
  }

  // ---- piece wave: pieces are consecutive runs of at most `per` tiles of one
  // (stream, KV head); wave wv takes piece wv ----
  const int wv = (int)blockIdx.x * kDecWaves + wave;
  const int n0 = lane < p.B ? stream_tiles(p, lane).n : 0;  // streams 0..63, kept
  const long long T = total_tiles(p, lane, n0);
  if (T == 0) return;
  const int per = piece_tiles(p, T);
  // the stream holding piece wv: Kb = index of its first piece
  int b = 0;
  long long Kb = 0;
  bool found = false;
  for (int b0 = 0; b0 < p.B; b0 += 64) {
    const int bl = b0 + lane;
    const int nl = b0 == 0 ? n0 : (bl < p.B ? stream_tiles(p, bl).n : 0);
    const long long np = (long long)((nl + per - 1) / per) * p.Hkv;
    long long incl = np;  // inclusive scan over the wave
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const long long y = __shfl_up(incl, off);
      if (lane >= off) incl += y;
    }
    const uint64_t hit = __ballot(np > 0 && Kb + incl > wv);
    if (hit) {
      const int l = __builtin_ctzll(hit);
      b = b0 + l;
      Kb += __shfl(incl - np, l);
      found = true;
      break;
    }
    Kb += __shfl(incl, 63);
  }
  if (!found) return;  // more waves than pieces

  {
    const StreamTiles st = stream_tiles(p, b);
    const int pc = (st.n + per - 1) / per;  // pieces per KV head of this stream
    // The piece is the same in every lane (it comes from a ballot, shuffles
    // and per-stream values); stating it keeps its descriptors scalar and its
    // tile branches uniform: a descriptor the compiler takes for divergent
    // costs a readfirstlane loop per load.
    // piece j of the head takes tiles j, j + pc, j + 2 pc, ... (at most per
    // of them): the head's pieces stream neighbouring tiles at the same time
    const int kvh = uniform_i32((int)((wv - Kb) / pc));
    const int j0 = uniform_i32((int)((wv - Kb) % pc));
    const int cnt = uniform_i32((st.n - j0 + pc - 1) / pc);
    u32x4 kraw[kDecBufs][2][NKS];
    u32x4 vraw[kDecBufs][NDB];
    bf16x8 qf[NKS];
    const size_t head = (size_t)b * p.Hkv + kvh;
    const __amdgpu_buffer_rsrc_t rk = make_rsrc(p.k_ring + head * (size_t)C * D,
                                                (uint32_t)((size_t)C * D * 2));
    const __amdgpu_buffer_rsrc_t rv = make_rsrc(p.v_ring + head * (size_t)D * C,
                                                (uint32_t)((size_t)D * C * 2));
    const int tstride = kDecTile * pc;                       // tokens from one tile to the next
    const long long tk0 = st.T0 + (long long)kDecTile * j0;  // token of the first tile
    const int sb0 = (int)(tk0 % C);                           // its slot
    // visible tokens relative to tk0
    const long long rlo64 = st.lo - tk0, rhi64 = st.hi - tk0;
    const int rlo = (int)(rlo64 < -0x40000000LL ? -0x40000000LL : rlo64);
    const int rhi = (int)(rhi64 > 0x40000000LL ? 0x40000000LL : rhi64);


    // tile i of the piece: K rows (block kb, A-row rho = c16 -> token
    // 8*(rho/4) + 4*kb + rho%4 of the tile) and V rows (d = 16*db + c16,
    // tokens 8*g4 .. +8, one 16-byte piece of the slot's V block). The head's
    // tiles span at most C + 62 tokens, so sb0 + tstride i < 2C + 32: at most
    // two wraps.
    auto issue = [&](int i, int buf) __attribute__((always_inline)) {
      int sb = sb0 + tstride * i;
      sb = sb >= C ? sb - C : sb;
      sb = sb >= C ? sb - C : sb;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        int slot = sb + 8 * (c16 >> 2) + 4 * kb + (c16 & 3);
        slot = slot >= C ? slot - C : slot;
#pragma unroll
        for (int k = 0; k < NKS; ++k)
          kraw[buf][kb][k] = buf_load16(rk, (uint32_t)(((size_t)slot * D + 32 * k + 8 * g4) * 2));
      }
      int vslot = sb + 8 * g4;
      vslot = vslot >= C ? vslot - C : vslot;
      const uint32_t v0 = vring_elem(vslot, c16, C, D), vw = vring_width(vslot, C);
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        vraw[buf][db] = buf_load16(rv, (v0 + 16 * db * vw) * 2);
    };

    f32x4 o[NDB];
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m = kNegInf, lsum = 0.f;

    // the piece's tiles, unrolled so that the register buffers stay
    // statically indexed; tiles past cnt are skipped (uniform branches)
#pragma unroll
    for (int j = 0; j < kDecBufs; ++j)
      if (j < cnt) issue(j, j);
    // The query is loaded and rotated while the first tiles are in flight:
    // waiting for its loads waits for theirs too (loads retire in order),
    // but the wave's streaming starts a round trip and the rotation earlier.
    query_frag(b, kvh, st.L, qf);
#pragma unroll
    for (int i = 0; i < kDecChunk; ++i) {
      const int buf = i % kDecBufs;
      if (i < cnt) {
        f32x4 sacc[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          sacc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int k = 0; k < NKS; ++k)
            sacc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, kraw[buf][kb][k]), qf[k], sacc[kb], 0, 0, 0);
        }
        // score (kb, r) of lane group g4 is token 8*g4 + 4*kb + r of tile i
        float mt = kNegInf;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int rel = tstride * i + 8 * g4 + 4 * kb + r;
            if (rel < rlo || rel > rhi) sacc[kb][r] = kNegInf;
            mt = fmaxf(mt, sacc[kb][r]);
          }
        mt = fmaxf(mt, __shfl_xor(mt, 16));
        mt = fmaxf(mt, __shfl_xor(mt, 32));
        const float mnew = fmaxf(m, mt);
        const float msafe = mnew == kNegInf ? 0.f : mnew;
        const float alpha = __builtin_amdgcn_exp2f(m - msafe);
        m = mnew;
        bf16x8 pf;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            pf[4 * kb + r] = (__bf16)__builtin_amdgcn_exp2f(sacc[kb][r] - msafe);
        // the sum takes the rounded weights the PV product uses, so that the
        // output is a convex combination of the V rows
        float ts = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const bf16x2 pr = {pf[2 * w], pf[2 * w + 1]};
          ts = __builtin_amdgcn_fdot2_f32_bf16(pr, kOnes2, ts, false);
        }
        lsum = lsum * alpha + ts;
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          o[db] *= alpha;
          o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, vraw[buf][db]), pf, o[db], 0, 0, 0);
        }
      }
      if (i + kDecBufs < cnt) issue(i + kDecBufs, buf);
    }

    // partial of this piece in slot (wave + head): lane column c16 = query,
    // O^T row (d) = 16*db + 4*g4 + r
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    float *part = p.ws + (size_t)wv * pfl;
    if (c16 < G) {
      float *orow = part + decode_out_off(G) + c16 * D;
#pragma unroll
      for (int db = 0; db < NDB; ++db) *reinterpret_cast<f32x4 *>(orow + 16 * db + 4 * g4) = o[db];
      if (g4 == 0) {
        part[c16] = m;
        part[G + c16] = lsum;
      }
    }

  }
}

// Combine pass: one block of kCombineThreads threads per (stream, KV head).
// Thread t owns the 4-float groups t, t + kCombineThreads, ... of the head's
// G x D outputs (query g = group / (D/4)). The head's partials are its
// own-token partial, which starts the merge, and its pieces (their slot range
// is recorded in the own-token slot by the split pass), merged online in
// groups of kCombineGroup whose (max, sum, outputs) loads are independent, so
// the pass waits on memory once for the own-token slot and once per group.
constexpr int kCombineThreads = 256;
constexpr int kCombineGroup = 16;

template <int D, int F>
__global__ __launch_bounds__(kCombineThreads) void decode_combine_kernel(DecodeParams p) {
  constexpr int Q4 = D / 4;  // 4-float groups per output row
  const int kvh = blockIdx.x, b = blockIdx.y;
  const int t = threadIdx.x;
  const int G = p.G;
  const int head = b * p.Hkv + kvh;
  const size_t pstride = decode_split_floats(G, D);
  const int oo = decode_out_off(G);

  // the head's pieces (slots K .. K+np-1) and query token, as the split pass
  // recorded them in the own-token slot; seq_len is not read here, so that an
  // appending combine may advance it
  const float *own = p.ws + (size_t)(p.nwaves + head) * pstride;
  const uint32_t *hdr = reinterpret_cast<const uint32_t *>(own + oo);
  const int K = (int)hdr[0], np = (int)hdr[1];
  const long long L = (long long)((unsigned long long)hdr[2] | ((unsigned long long)hdr[3] << 32));

  int gq[F], e4[F];  // query and first element of each of this thread's groups
  bool live[F];
#pragma unroll
  for (int f = 0; f < F; ++f) {
    const int idx = t + kCombineThreads * f;
    live[f] = idx < G * Q4;
    gq[f] = live[f] ? idx / Q4 : 0;
    e4[f] = live[f] ? 4 * (idx % Q4) : 0;
  }
  // the merge starts from the own token's partial: its max and sum (1) from
  // the own-token slot, its output row v_new itself
  float M[F], lt[F];
  f32x4 acc[F];
#pragma unroll
  for (int f = 0; f < F; ++f) {
    M[f] = own[gq[f]];
    lt[f] = own[G + gq[f]];
    const u32x2 w = *reinterpret_cast<const u32x2 *>(p.v_new + (size_t)head * D + e4[f]);
    acc[f] = f32x4{bf16_bits_to_f32(w[0] & 0xffffu), bf16_bits_to_f32(w[0] >> 16),
                   bf16_bits_to_f32(w[1] & 0xffffu), bf16_bits_to_f32(w[1] >> 16)};
  }
  // then the pieces, kCombineGroup at a time. A group's loads carry no
  // branch, so that they are all in flight together: entries past the last
  // piece read the last piece again (finite: every piece holds a visible
  // key) and count with weight zero.
  for (int c0 = 0; c0 < np; c0 += kCombineGroup) {
    float mv[kCombineGroup][F], lv[kCombineGroup][F];
    f32x4 ov[kCombineGroup][F];
#pragma unroll
    for (int j = 0; j < kCombineGroup; ++j) {
      const int c = min(c0 + j, np - 1);
      const float *pp = p.ws + (size_t)(K + c) * pstride;
#pragma unroll
      for (int f = 0; f < F; ++f) {
        mv[j][f] = pp[gq[f]];
        lv[j][f] = pp[G + gq[f]];
        ov[j][f] = *reinterpret_cast<const f32x4 *>(pp + oo + gq[f] * D + e4[f]);
      }
    }
#pragma unroll
    for (int f = 0; f < F; ++f) {
      // every piece has a positive sum; the running state already has one
      float Mg = M[f];
#pragma unroll
      for (int j = 0; j < kCombineGroup; ++j)
        if (c0 + j < np) Mg = fmaxf(Mg, mv[j][f]);
      const float a = __builtin_amdgcn_exp2f(M[f] - Mg);
      acc[f] *= a;
      lt[f] *= a;
#pragma unroll
      for (int j = 0; j < kCombineGroup; ++j) {
        const float w = c0 + j < np ? __builtin_amdgcn_exp2f(mv[j][f] - Mg) : 0.f;
        acc[f] += ov[j][f] * w;
        lt[f] += lv[j][f] * w;
      }
      M[f] = Mg;
    }
  }
#pragma unroll
  for (int f = 0; f < F; ++f) {
    if (!live[f]) continue;
    const float inv = 1.f / lt[f];
    const int hq = kvh * G + gq[f];
    u32x2 w;
    w[0] = f32_to_bf16_rne(acc[f][0] * inv) | (f32_to_bf16_rne(acc[f][1] * inv) << 16);
    w[1] = f32_to_bf16_rne(acc[f][2] * inv) | (f32_to_bf16_rne(acc[f][3] * inv) << 16);
    *reinterpret_cast<u32x2 *>(p.out + ((size_t)b * p.Hq + hq) * D + e4[f]) = w;
    if (e4[f] == 0 && p.lse != nullptr)
      p.lse[(size_t)b * p.Hq + hq] = (M[f] + __builtin_amdgcn_logf(lt[f])) * 0.6931471805599453f;
  }

  // the append: the split pass has finished every read of the ring and of
  // seq_len, and no combine block reads either
  if (p.append) {
    const int slot = (int)(L % p.C);
    if (t < D / 2)
      reinterpret_cast<uint32_t *>(p.k_ring + ((size_t)head * p.C + slot) * D)[t] =
          hdr[kOwnHdr + t];
    if (t < D)
      p.v_ring[(size_t)head * D * p.C + vring_elem(slot, t, p.C, D)] =
          p.v_new[(size_t)head * D + t];
    if (kvh == 0 && t == 0) p.seq_len[b] = L + 1;
  }
}

}  // namespace

hipError_t launch_decode_split(const DecodeParams &p, const RopeDev &r, hipStream_t s) {
  const int H = p.B * p.Hkv;
  dim3 grid(p.nwaves / kDecWaves + (H + kDecWaves - 1) / kDecWaves);  // + own-token waves
  if (p.D == 128)
    dispatch(decode_split_kernel<128>, grid, dim3(256), s, p, r);
  else
    dispatch(decode_split_kernel<64>, grid, dim3(256), s, p, r);
  return hipGetLastError();
}

hipError_t launch_decode_combine(const DecodeParams &p, hipStream_t s) {
  dim3 grid(p.Hkv, p.B);
  const bool two = p.G * p.D / 4 > kCombineThreads;  // at most 2 groups of 4 per thread
  if (p.D == 128 && two)
    dispatch(decode_combine_kernel<128, 2>, grid, dim3(kCombineThreads), s, p);
  else if (p.D == 128)
    dispatch(decode_combine_kernel<128, 1>, grid, dim3(kCombineThreads), s, p);
  else
    dispatch(decode_combine_kernel<64, 1>, grid, dim3(kCombineThreads), s, p);
  return hipGetLastError();
}

}  // namespace frt
