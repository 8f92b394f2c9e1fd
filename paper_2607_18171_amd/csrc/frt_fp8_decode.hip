// One-token decode over an FP8 (OCP e4m3fn) ring: the split pass and the
// combine pass of the bf16 decode, with the same pieces and the same merge of
// (max, sum, output) partials.
//
// MFMA v_mfma_f32_16x16x128_f8f6f4, both operands e4m3: lane l holds row (A)
// or column (B) l%16 and the 32 k-slots of group l/16 (A and B pair their
// slots the same way); the output D[row][col] sits in lane col + 16*(row/4),
// register row%4.
//  * Scores S^T = K Q^T, one MFMA per 16 keys (all of d = 128): A row rho of
//    key block kb is key 8*(rho/4) + 4*kb + rho%4 of the 32-key tile, so a
//    lane's 8 scores are keys 8*(l/16) .. +8 of its query l%16. The query
//    codes (B) follow the FP8 step: the query rotated and scaled to base-2
//    score units in double, rounded to fp32, coded with a power-of-two scale
//    per query.
//  * Weights p = code(2^(s - m + 7)) against an integer reference max m per
//    query, raised when a tile's max passes it by more than 1, as in the FP8
//    step. They are the B operand of O^T = V^T P^T in bytes 0..7 of the lane's
//    k-slots (zeros elsewhere); A is the matching 8 value codes of d-row
//    16*db + l%16, one 8-byte load from the ring's 32-slot block. A ninth MFMA
//    with ones in A gives sum(p).
//  * A partial is (m, sum p, s_v * sum p v); the merge of partials with
//    integer references m only rescales by powers of two.
// The own token's partial holds the token alone, its key and value coded as
// the append stores them; its slot also carries the head's piece range, the
// query position and the token's codes for the combine pass.
#include "frt_decode_pieces.hpp"
#include "frt_fp8.hpp"

namespace frt {

namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int kOwnHdr8 = 4;   // header words before the own token's codes
#ifndef FRT_DEC8_BUFS
#define FRT_DEC8_BUFS 2
#endif
constexpr int kDec8Bufs = FRT_DEC8_BUFS;  // tiles in flight per piece wave (8 KB each)
constexpr uint32_t kNullOffset = 0x80000000u;  // beyond every ring descriptor
constexpr float kTau8 = 1.f;  // the reference max lags the row max by at most this
constexpr float kShift8 = 7.f;

__device__ __forceinline__ f32x4 mfma16(i32x8 a, i32x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// max over the four lanes sharing l % 16 (one query)
__device__ __forceinline__ float max_query(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}

__device__ __forceinline__ u32x2 buf_load8(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, (int)byte_off, 0, 0);
}

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kDecWavesPerSimd))) void
decode_split_fp8_kernel(DecodeFp8Params p, RopeDev rope) {
  static_assert(D == 128, "one MFMA covers the head dimension");
  constexpr int NDB = D / 16;  // 16-row d blocks of O^T
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c16 = lane & 15, g4 = lane >> 4;
  const int G = p.G, C = p.C, H = p.B * p.Hkv;
  const size_t pfl = decode_fp8_split_floats(G, D);
  const RopeReg rg = rope_reg(rope);
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};

  // query codes of (stream b, KV head kvh) at token L: B operand, column c16
  // (< G; columns past G read beyond the descriptor and get zeros), d bytes
  // 32*g4 .. +32; cq = 2^e * s_k turns a code product into base-2 units
  auto query_codes = [&](int b, int kvh, long long L, float sk, i32x8 &qf, float &cq)
                         __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(p.q + ((size_t)b * p.Hq + kvh * G) * D, (uint32_t)(G * D * 2));
    int co[3];
    rope_coords(rg, L, co);
    float a[32];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int d0 = 32 * g4 + 8 * w;
      rotate8_f32(rope_fetch4(rg, co, d0 / 2), buf_load16(rq, (uint32_t)((c16 * D + d0) * 2)),
                  p.qmul, a + 8 * w);
    }
    float mx = 0.f;
#pragma unroll
    for (int j = 0; j < 32; ++j) mx = fmaxf(mx, fabsf(a[j]));
    const int e = fp8_row_exponent(max_query(mx));
#pragma unroll
    for (int w = 0; w < 8; ++w)  // |a| / 2^e <= 448 by the choice of e
      qf[w] = (int)e4m3x4_inrange(ldexpf(a[4 * w], -e), ldexpf(a[4 * w + 1], -e),
                                  ldexpf(a[4 * w + 2], -e), ldexpf(a[4 * w + 3], -e));
    cq = ldexpf(1.f, e) * sk;
  };

  const int own_first = p.nwaves / kDecWaves;  // blocks from here write own-token partials
  if ((int)blockIdx.x >= own_first) {
    const int h = ((int)blockIdx.x - own_first) * kDecWaves + wave;
    if (h >= H) return;
    const int b = h / p.Hkv, kvh = h % p.Hkv;
    const long long L = p.seq_len[b];
    const float sk = p.sc.k[h], sv = p.sc.v[h];
    i32x8 qf;
    float cq;
    query_codes(b, kvh, L, sk, qf, cq);
    // the token's key and value codes, d bytes 32*g4 .. +32 (as the append stores them)
    const __amdgpu_buffer_rsrc_t rkn = make_rsrc(p.k_new + (size_t)h * D, (uint32_t)(D * 2));
    const __amdgpu_buffer_rsrc_t rvn = make_rsrc(p.v_new + (size_t)h * D, (uint32_t)(D * 2));
    int co[3];
    rope_coords(rg, L, co);
    i32x8 kc, vc;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int d0 = 32 * g4 + 8 * w;
      float y[8];
      rotate8_f32(rope_fetch4(rg, co, d0 / 2), buf_load16(rkn, (uint32_t)(d0 * 2)), 1.0, y);
      const u32x2 kw = code8(y, sk);
      float v[8];
      bf16x8_to_f32(buf_load16(rvn, (uint32_t)(d0 * 2)), v);
      const u32x2 vw = code8(v, sv);
      kc[2 * w] = (int)kw[0];
      kc[2 * w + 1] = (int)kw[1];
      vc[2 * w] = (int)vw[0];
      vc[2 * w + 1] = (int)vw[1];
    }
    // every A row is the token's key: each output row is the score
    const float s = mfma16(kc, qf, zero4)[0] * cq;
    const float m = ceilf(s);
    const uint32_t pc = e4m3x4_inrange(__builtin_amdgcn_exp2f(s - m + kShift8), 0.f, 0.f, 0.f);
    const float pw = __builtin_amdgcn_cvt_f32_fp8((int)pc, 0);
    int K, np;
    head_pieces(p, lane, b, kvh, K, np);
    float *part = p.ws + (size_t)(p.nwaves + h) * pfl;
    uint32_t *hdr = reinterpret_cast<uint32_t *>(part + (size_t)G * (2 + D));
    if (c16 < G) {
      if (g4 == 0) {
        part[c16] = m;
        part[G + c16] = pw;
      }
      float *orow = part + 2 * G + c16 * D + 32 * g4;
      const float f = pw * sv;
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        orow[4 * w] = f * __builtin_amdgcn_cvt_f32_fp8(vc[w], 0);
        orow[4 * w + 1] = f * __builtin_amdgcn_cvt_f32_fp8(vc[w], 1);
        orow[4 * w + 2] = f * __builtin_amdgcn_cvt_f32_fp8(vc[w], 2);
        orow[4 * w + 3] = f * __builtin_amdgcn_cvt_f32_fp8(vc[w], 3);
      }
    }
    if (lane == 0) {
      hdr[0] = (uint32_t)K;
      hdr[1] = (uint32_t)np;
      hdr[2] = (uint32_t)(unsigned long long)L;
      hdr[3] = (uint32_t)((unsigned long long)L >> 32);
    }
    if (c16 == 0) {
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        hdr[kOwnHdr8 + 8 * g4 + w] = (uint32_t)kc[w];
        hdr[kOwnHdr8 + D / 4 + 8 * g4 + w] = (uint32_t)vc[w];
      }
    }
    return;
  }

  // ---- piece wave: wave wv takes piece wv (the bf16 decode's mapping) ----
  const int wv = (int)blockIdx.x * kDecWaves + wave;
  const int n0 = lane < p.B ? stream_tiles(p, lane).n : 0;  // streams 0..63, kept
  const long long T = total_tiles(p, lane, n0);
  if (T == 0) return;
  const int per = piece_tiles(p, T);
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

  const StreamTiles st = stream_tiles(p, b);
  const int pc = (st.n + per - 1) / per;  // pieces per KV head of this stream
  // one piece for the whole wave: keep its descriptors scalar
  const int kvh = uniform_i32((int)((wv - Kb) / pc));
  const int j0 = uniform_i32((int)((wv - Kb) % pc) * per);
  const int cnt = uniform_i32(min(st.n - j0, per));
  const size_t head = (size_t)b * p.Hkv + kvh;
  const float sk = p.sc.k[head], sv = p.sc.v[head];
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(p.k_ring + head * (size_t)C * D, (uint32_t)((size_t)C * D));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(p.v_ring + head * (size_t)D * C, (uint32_t)((size_t)D * C));
  const long long tk0 = st.T0 + (long long)kDecTile * j0;  // token of the first tile
  const int sb0 = (int)(tk0 % C);
  const long long rlo64 = st.lo - tk0, rhi64 = st.hi - tk0;
  const int rlo = (int)(rlo64 < -0x40000000LL ? -0x40000000LL : rlo64);
  const int rhi = (int)(rhi64 > 0x40000000LL ? 0x40000000LL : rhi64);

  i32x8 qf;
  float cq;
  query_codes(b, kvh, st.L, sk, qf, cq);

  // tile i: K rows (block kb, A-row rho = c16 -> key 8*(rho/4) + 4*kb + rho%4,
  // d bytes 32*g4 .. +32) and V (d-row 16*db + c16, keys 8*g4 .. +8: 8 bytes
  // of the slot's V block; 8 keys starting at a multiple of 8 never leave it).
  // Tiles past the piece are issued too, with offsets outside the descriptors
  // (no memory traffic, zeros), so that every path leaves the same loads
  // outstanding and the waits for a tile count exactly.
  u32x4 kraw[kDec8Bufs][2][2];
  u32x2 vraw[kDec8Bufs][NDB];
  auto issue = [&](int i, int buf) __attribute__((always_inline)) {
    const bool live = i < cnt;
    int sb = sb0 + kDecTile * (live ? i : 0);
    sb = sb >= C ? sb - C : sb;
    sb = sb >= C ? sb - C : sb;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      int slot = sb + 8 * (c16 >> 2) + 4 * kb + (c16 & 3);
      slot = slot >= C ? slot - C : slot;
      const uint32_t off = live ? (uint32_t)slot * D + 32 * g4 : kNullOffset;
      kraw[buf][kb][0] = buf_load16(rk, off);
      kraw[buf][kb][1] = buf_load16(rk, off + 16);
    }
    int vslot = sb + 8 * g4;
    vslot = vslot >= C ? vslot - C : vslot;
    const uint32_t v0 = live ? vring_elem(vslot, c16, C, D) : kNullOffset;
    const uint32_t vw = live ? vring_width(vslot, C) : 0u;
#pragma unroll
    for (int db = 0; db < NDB; ++db) vraw[buf][db] = buf_load8(rv, v0 + 16 * db * vw);
  };

  f32x4 o[NDB], lacc = zero4;
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = zero4;
  float m = kNegInf;  // reference max of this lane's query, an integer
  const i32x8 ones = {0x38383838, 0x38383838, 0, 0, 0, 0, 0, 0};  // e4m3 1.0 in bytes 0..7

  // one tile from buffer buf: scores, the reference max, coded weights, O^T
  // and sum(p)
  auto tile = [&](int i, int buf) __attribute__((always_inline)) {
    f32x4 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const u32x4 lo = kraw[buf][kb][0], hi = kraw[buf][kb][1];
      const i32x8 a = {(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                       (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
      sacc[kb] = mfma16(a, qf, zero4);
    }
    // register r of block kb: key 8*g4 + 4*kb + r of tile i
    float mt = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rel = kDecTile * i + 8 * g4 + 4 * kb + r;
        if (rel < rlo || rel > rhi) sacc[kb][r] = kNegInf;
        mt = fmaxf(mt, sacc[kb][r] * cq);
      }
    mt = max_query(mt);
    const bool raise = mt > m + kTau8 || (m == kNegInf && mt != kNegInf);
    if (__ballot(raise)) {
      const float mn = raise ? ceilf(mt) : m;
      const float alpha = raise ? (m == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m - mn)) : 1.f;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] *= alpha;
      lacc *= alpha;
      m = mn;
    }
    const float nm = kShift8 - (m == kNegInf ? 0.f : m);
    uint32_t pw[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)  // at most 2^(kTau + 7) < 448
      pw[kb] = e4m3x4_inrange(__builtin_amdgcn_exp2f(fmaf(sacc[kb][0], cq, nm)),
                              __builtin_amdgcn_exp2f(fmaf(sacc[kb][1], cq, nm)),
                              __builtin_amdgcn_exp2f(fmaf(sacc[kb][2], cq, nm)),
                              __builtin_amdgcn_exp2f(fmaf(sacc[kb][3], cq, nm)));
    const i32x8 pb = {(int)pw[0], (int)pw[1], 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const i32x8 a = {(int)vraw[buf][db][0], (int)vraw[buf][db][1], 0, 0, 0, 0, 0, 0};
      o[db] = mfma16(a, pb, o[db]);
    }
    lacc = mfma16(ones, pb, lacc);
  };

#pragma unroll
  for (int j = 0; j < kDec8Bufs; ++j) issue(j, j);
  for (int i0 = 0; i0 < cnt; i0 += kDec8Bufs) {
#pragma unroll
    for (int u = 0; u < kDec8Bufs; ++u) {
      if (i0 + u < cnt) tile(i0 + u, u);
      issue(i0 + u + kDec8Bufs, u);
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the loads past the piece

  // partial of this piece in slot wv: lane column c16 = query, O^T row (d)
  // = 16*db + 4*g4 + r
  float *part = p.ws + (size_t)wv * pfl;
  if (c16 < G) {
    float *orow = part + 2 * G + c16 * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r) orow[16 * db + 4 * g4 + r] = o[db][r] * sv;
    if (g4 == 0) {
      part[c16] = m;
      part[G + c16] = lacc[0];
    }
  }
}

// Combine pass: one block of D threads per (query head, KV head, stream),
// thread d owns output column d; the head's partials are its pieces and its
// own token's, merged online in groups (as in the bf16 decode).
constexpr int kCombineGroup8 = 16;

template <int D>
__global__ __launch_bounds__(D) void decode_combine_fp8_kernel(DecodeFp8Params p) {
  const int q = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int t = threadIdx.x;
  const int G = p.G;
  const int head = b * p.Hkv + kvh;
  const int hq = kvh * G + q;
  const size_t pstride = decode_fp8_split_floats(G, D);
  // the head's pieces (slots K .. K+np-1), query token and codes, as the
  // split pass recorded them; seq_len is not read here, so that an
  // appending combine may advance it
  const float *own = p.ws + (size_t)(p.nwaves + head) * pstride;
  const uint32_t *hdr = reinterpret_cast<const uint32_t *>(own + (size_t)G * (2 + D));
  const int K = (int)hdr[0], np = (int)hdr[1];
  const long long L = (long long)((unsigned long long)hdr[2] | ((unsigned long long)hdr[3] << 32));
  const int ncand = np + 1;  // pieces, then the own token

  float M = kNegInf, acc = 0.f, lt = 0.f;
  for (int c0 = 0; c0 < ncand; c0 += kCombineGroup8) {
    float mv[kCombineGroup8], lv[kCombineGroup8], ov[kCombineGroup8];
#pragma unroll
    for (int j = 0; j < kCombineGroup8; ++j) {
      const int c = c0 + j;
      mv[j] = kNegInf;
      lv[j] = 0.f;
      ov[j] = 0.f;
      if (c <= np) {
        const float *pp = c < np ? p.ws + (size_t)(K + c) * pstride : own;
        mv[j] = pp[q];
        lv[j] = pp[G + q];
        ov[j] = pp[2 * G + q * D + t];
      }
    }
    float Mg = M;  // live partials have a positive sum (the own token's always has)
#pragma unroll
    for (int j = 0; j < kCombineGroup8; ++j) Mg = lv[j] > 0.f ? fmaxf(Mg, mv[j]) : Mg;
    if (Mg != kNegInf) {
      const float a = __builtin_amdgcn_exp2f(M - Mg);  // M = -inf gives 0
      acc *= a;
      lt *= a;
#pragma unroll
      for (int j = 0; j < kCombineGroup8; ++j) {
        const float w = lv[j] > 0.f ? __builtin_amdgcn_exp2f(mv[j] - Mg) : 0.f;
        acc += ov[j] * w;
        lt += lv[j] * w;
      }
      M = Mg;
    }
  }
  p.out[((size_t)b * p.Hq + hq) * D + t] = (uint16_t)f32_to_bf16_rne(acc / lt);
  if (t == 0 && p.lse != nullptr)
    p.lse[(size_t)b * p.Hq + hq] =
        (M - kShift8 + __builtin_amdgcn_logf(lt)) * 0.6931471805599453f;

  // the append: the split pass has finished every read of the ring and of
  // seq_len, and no combine block reads either
  if (p.append && q == 0) {
    const int slot = (int)(L % p.C);
    if (t < D / 4)
      reinterpret_cast<uint32_t *>(p.k_ring + ((size_t)head * p.C + slot) * D)[t] =
          hdr[kOwnHdr8 + t];
    const uint8_t *vcodes = reinterpret_cast<const uint8_t *>(hdr + kOwnHdr8 + D / 4);
    p.v_ring[(size_t)head * D * p.C + vring_elem(slot, t, p.C, D)] = vcodes[t];
    if (kvh == 0 && t == 0) p.seq_len[b] = L + 1;
  }
}

}  // namespace

hipError_t launch_decode_split_fp8(const DecodeFp8Params &p, const RopeDev &r, hipStream_t s) {
  const int H = p.B * p.Hkv;
  dim3 grid(p.nwaves / kDecWaves + (H + kDecWaves - 1) / kDecWaves);  // + own-token waves
  if (p.D != 128) return hipErrorInvalidValue;  // the host API admits head_dim 128 only
  dispatch(decode_split_fp8_kernel<128>, grid, dim3(256), s, p, r);
  return hipGetLastError();
}

hipError_t launch_decode_combine_fp8(const DecodeFp8Params &p, hipStream_t s) {
  dim3 grid(p.G, p.Hkv, p.B);
  if (p.D != 128) return hipErrorInvalidValue;
  dispatch(decode_combine_fp8_kernel<128>, grid, dim3(128), s, p);
  return hipGetLastError();
}

}  // namespace frt
