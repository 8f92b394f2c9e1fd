// Piece sizing of the decode split passes (bf16 and FP8 rings): the visible
// ring tokens of each (stream, KV head) as 32-token tiles, cut into pieces of
// at most `per` tiles, one wave each (which tiles a piece takes is the
// pass's choice). Templates over the pass's parameter block (seq_len, mask,
// C, B, Hkv are all they read).
#pragma once
#include "frt_launch.hpp"

namespace frt {

constexpr int kDecWaves = 4;   // waves per block
constexpr int kDecTile = 32;   // tokens per tile
constexpr int kMinTilesPerWave = 4;
constexpr float kNegInf = -__builtin_inff();

// Visible ring tokens of stream b's decode query, as 32-token tiles.
struct StreamTiles {
  long long L, lo, hi, T0;  // query token, visible [lo, hi], first tile token
  int n;                    // tiles
};

template <class P>
__device__ __forceinline__ StreamTiles stream_tiles(const P &p, int b) {
  StreamTiles s;
  s.L = p.seq_len[b];
  long long vlo, vhi;
  visible_range(p.mask_kind, p.mask_block, p.mask_window, s.L, vlo, vhi);
  const long long held = s.L < p.C ? s.L : (long long)p.C;
  s.lo = vlo > s.L - held ? vlo : s.L - held;
  s.hi = s.L - 1;
  s.T0 = s.lo & ~(long long)(kDecTile - 1);
  s.n = s.lo <= s.hi ? (int)((s.hi - s.T0) / kDecTile + 1) : 0;
  return s;
}

// Tiles of every (stream, KV head): the tiles of streams lane, lane+64, ...
// summed over the wave, times Hkv. n0 is this lane's count for stream lane.
template <class P>
__device__ __forceinline__ long long total_tiles(const P &p, int lane, int n0) {
  long long tot = 0;
  for (int b0 = 0; b0 < p.B; b0 += 64) {
    const int b = b0 + lane;
    long long n = b0 == 0 ? n0 : (b < p.B ? stream_tiles(p, b).n : 0);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) n += __shfl_xor(n, off);
    tot += n;
  }
  return tot * p.Hkv;
}

// Tiles per piece: every (stream, KV head) is cut into pieces of at most
// `per` tiles, one wave each. per ~ T / (resident waves - heads) spreads the
// tiles evenly over the waves that run at once; it is kept in
// [kMinTilesPerWave, kDecChunk], and the grid is large enough for the number
// of pieces that gives (at most T / per + heads).
template <class P>
__device__ __forceinline__ int piece_tiles(const P &p, long long T) {
  const long long heads = (long long)p.B * p.Hkv;
  const long long slots = kDecResident - heads > kDecResident / 2 ? kDecResident - heads
                                                                   : kDecResident / 2;
  long long per = (T + slots - 1) / slots;
  per = per < kMinTilesPerWave ? kMinTilesPerWave : per;
  return (int)(per > kDecChunk ? kDecChunk : per);
}

// First partial slot and number of pieces of (stream b, KV head kvh), in the
// order the piece waves take them: streams in order, each stream's KV heads
// in order, each head's pieces in token order. A wave-wide computation.
template <class P>
__device__ __forceinline__ void head_pieces(const P &p, int lane, int b, int kvh, int &K,
                                            int &np) {
  const int n0 = lane < p.B ? stream_tiles(p, lane).n : 0;  // streams 0..63
  const long long T = total_tiles(p, lane, n0);
  int n = __shfl(n0, b & 63);
  if (b >= 64) n = stream_tiles(p, b).n;
  K = 0;
  np = 0;
  if (n > 0) {
    const int per = piece_tiles(p, T);
    long long before = 0;  // pieces per KV head of streams before b
    for (int b0 = 0; b0 < b; b0 += 64) {
      const int bl = b0 + lane;
      const int nl = b0 == 0 ? n0 : (bl < p.B ? stream_tiles(p, bl).n : 0);
      long long c = bl < b ? (nl + per - 1) / per : 0;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off);
      before += c;
    }
    np = (n + per - 1) / per;
    K = (int)(before * p.Hkv) + kvh * np;
  }
}

}  // namespace frt
