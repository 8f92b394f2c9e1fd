// C ABI of libfrt: argument validation, launch planning, rotary tables and
// built-in kernel timing. See include/frt.h for the contract of each call.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "frt.h"
#include "frt_launch.hpp"

using namespace frt;

namespace {

thread_local std::string g_err;

frt_status fail(frt_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------- timing --
}  // namespace

namespace frt {
DispatchEvents &pending_dispatch_events() {
  thread_local DispatchEvents ev;
  return ev;
}
}  // namespace frt

namespace {

struct TimingRec {
  const char *name;
  hipEvent_t start, stop;
};

std::mutex g_tmu;
bool g_timing = false;
std::vector<TimingRec> g_recs;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <class F>
frt_status launch(const char *name, hipStream_t s, F &&f) {
  hipEvent_t a = nullptr, b = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_tmu);
    if (g_timing) {
      a = take_event();
      b = take_event();
    }
  }
  if (a && b) pending_dispatch_events() = DispatchEvents{a, b};
  hipError_t e = f();
  // the dispatch takes the events; a launcher that failed before it did not
  const bool taken = pending_dispatch_events().start == nullptr;
  pending_dispatch_events() = DispatchEvents{};
  if (a && b) {
    std::lock_guard<std::mutex> lk(g_tmu);
    if (taken && e == hipSuccess) {
      g_recs.push_back({name, a, b});
    } else {
      g_pool.push_back(a);
      g_pool.push_back(b);
    }
  } else {
    std::lock_guard<std::mutex> lk(g_tmu);
    if (a) g_pool.push_back(a);
    if (b) g_pool.push_back(b);
  }
  if (e != hipSuccess) return fail(FRT_ERR_HIP, "%s launch failed: %s", name, hipGetErrorString(e));
  return FRT_OK;
}

// ------------------------------------------------------------ validation --
frt_status check_ring(const frt_ring *r) {
  if (!r) return fail(FRT_ERR_NULL, "ring is NULL");
  if (!r->k_ring || !r->v_ring || !r->seq_len) return fail(FRT_ERR_NULL, "ring buffer pointer is NULL");
  if (r->num_streams < 1 || r->num_kv_heads < 1)
    return fail(FRT_ERR_SHAPE, "num_streams=%d num_kv_heads=%d must be >= 1", r->num_streams,
                r->num_kv_heads);
  if (r->head_dim != 64 && r->head_dim != 128)
    return fail(r->head_dim > 0 ? FRT_ERR_UNSUPPORTED : FRT_ERR_SHAPE,
                "head_dim=%d (supported: 64, 128)", r->head_dim);
  if (r->capacity < 8) return fail(FRT_ERR_SHAPE, "capacity=%d must be >= 8", r->capacity);
  if (r->capacity % 8) return fail(FRT_ERR_ALIGN, "capacity=%d is not a multiple of 8", r->capacity);
  if ((size_t)r->capacity * r->head_dim * 2 >= (size_t)1 << 31)
    return fail(FRT_ERR_SHAPE, "capacity*head_dim*2 must be below 2^31");
  if (!aligned(r->k_ring, 16) || !aligned(r->v_ring, 16) || !aligned(r->seq_len, 8))
    return fail(FRT_ERR_ALIGN, "ring buffers must be 16-byte aligned (seq_len 8-byte)");
  return FRT_OK;
}

frt_status check_rope(const frt_rope *r, int d) {
  if (!r) return fail(FRT_ERR_NULL, "rope is NULL");
  if (r->mode == FRT_ROPE_NONE) return FRT_OK;
  if (r->mode != FRT_ROPE_1D && r->mode != FRT_ROPE_3D)
    return fail(FRT_ERR_SHAPE, "rope mode %d unknown", r->mode);
  if (!(r->base > 0.0)) return fail(FRT_ERR_SHAPE, "rope base must be > 0");
  const int naxes = r->mode == FRT_ROPE_1D ? 1 : 3;
  int sum = 0;
  for (int a = 0; a < naxes; ++a) {
    if (r->axis_dims[a] < 0 || r->axis_dims[a] % 2)
      return fail(FRT_ERR_SHAPE, "rope axis_dims[%d]=%d must be even and >= 0", a, r->axis_dims[a]);
    if (r->axis_dims[a] > 0 && r->max_pos[a] < 1)
      return fail(FRT_ERR_SHAPE, "rope max_pos[%d]=%d must be >= 1", a, r->max_pos[a]);
    sum += r->axis_dims[a];
  }
  if (sum < 2 || sum > d) return fail(FRT_ERR_SHAPE, "rope dims sum %d must be in [2, head_dim]", sum);
  if (r->mode == FRT_ROPE_3D && (r->frame_hw[0] < 1 || r->frame_hw[1] < 1))
    return fail(FRT_ERR_SHAPE, "rope frame_hw must be >= 1");
  if (frt_rope_table_bytes(r) >= (size_t)1 << 31)
    return fail(FRT_ERR_SHAPE, "rope table must be below 2^31 bytes");
  if (!r->table) return fail(FRT_ERR_NULL, "rope table is NULL");
  if (!aligned(r->table, 8)) return fail(FRT_ERR_ALIGN, "rope table must be 8-byte aligned");
  return FRT_OK;
}

frt_status check_mask(const frt_mask *m, int C) {
  if (!m) return fail(FRT_ERR_NULL, "mask is NULL");
  if (m->window < 0) return fail(FRT_ERR_SHAPE, "mask window must be >= 0");
  if (m->kind == FRT_MASK_BLOCK_CAUSAL) {
    if (m->block < 1) return fail(FRT_ERR_SHAPE, "block-causal block must be >= 1");
    if ((long long)m->window * m->block > C)
      return fail(FRT_ERR_CAPACITY, "capacity %d < window %d x block %d", C, m->window, m->block);
  } else if (m->kind == FRT_MASK_CAUSAL) {
    if (m->window > 0 && m->window - 1 > C)
      return fail(FRT_ERR_CAPACITY, "capacity %d < causal window %d - 1", C, m->window);
  } else {
    return fail(FRT_ERR_SHAPE, "mask kind %d unknown", m->kind);
  }
  return FRT_OK;
}

frt_status check_io(const void *p, const char *what) {
  if (!p) return fail(FRT_ERR_NULL, "%s is NULL", what);
  if (!aligned(p, 16)) return fail(FRT_ERR_ALIGN, "%s must be 16-byte aligned", what);
  return FRT_OK;
}

RopeDev rope_dev(const frt_rope *r) {
  RopeDev d;
  std::memset(&d, 0, sizeof(d));
  d.mode = r->mode;
  d.frame_h = d.frame_w = 1;
  if (r->mode == FRT_ROPE_NONE) return d;
  const int naxes = r->mode == FRT_ROPE_1D ? 1 : 3;
  size_t off = 0;  // in (cos, sin) entries
  for (int a = 0; a < naxes; ++a) {
    d.npairs[a] = r->axis_dims[a] / 2;
    d.maxpos[a] = d.npairs[a] ? r->max_pos[a] : 1;
    d.tab_off[a] = (int)off;
    off += (size_t)(d.npairs[a] ? r->max_pos[a] : 0) * d.npairs[a];
  }
  if (r->mode == FRT_ROPE_3D) {
    d.frame_h = r->frame_hw[0];
    d.frame_w = r->frame_hw[1];
  }
  d.tab_bytes = (uint32_t)frt_rope_table_bytes(r);
  d.table = reinterpret_cast<const float2 *>(r->table);
  return d;
}

double q_multiplier(float softmax_scale, int d) {
  const double scale = softmax_scale > 0.f ? (double)softmax_scale : 1.0 / std::sqrt((double)d);
  return scale * 1.4426950408889634;  // log2(e): scores are kept in base-2 units
}

struct StepLayout {
  size_t q_off, k_off, v_off, l_off, bytes;
  int n_pad;
};

StepLayout step_layout(const frt_ring *r, int n, int hq) {
  StepLayout L;
  const size_t d = (size_t)r->head_dim;
  L.n_pad = (int)round_up((size_t)n, kChunkBN);
  L.q_off = 0;
  L.k_off = round_up((size_t)r->num_streams * n * hq * d * 2, 256);
  L.v_off = L.k_off + round_up((size_t)r->num_streams * r->num_kv_heads * L.n_pad * d * 2, 256);
  L.l_off = L.v_off + round_up((size_t)r->num_streams * r->num_kv_heads * L.n_pad * d * 2, 256);
  L.bytes = L.l_off + round_up((size_t)r->num_streams * 8, 256);
  return L;
}

}  // namespace

extern "C" {

const char *frt_status_str(frt_status s) {
  switch (s) {
    case FRT_OK: return "ok";
    case FRT_ERR_NULL: return "null pointer";
    case FRT_ERR_SHAPE: return "invalid shape";
    case FRT_ERR_UNSUPPORTED: return "unsupported";
    case FRT_ERR_CAPACITY: return "ring capacity too small";
    case FRT_ERR_ALIGN: return "misaligned";
    case FRT_ERR_WORKSPACE: return "workspace too small";
    case FRT_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char *frt_last_error(void) { return g_err.c_str(); }

size_t frt_rope_table_bytes(const frt_rope *r) {
  if (!r || r->mode == FRT_ROPE_NONE) return 0;
  const int naxes = r->mode == FRT_ROPE_1D ? 1 : (r->mode == FRT_ROPE_3D ? 3 : 0);
  size_t floats = 0;
  for (int a = 0; a < naxes; ++a) {
    if (r->axis_dims[a] <= 0 || r->max_pos[a] <= 0) continue;
    floats += (size_t)r->max_pos[a] * (r->axis_dims[a] / 2) * 2;
  }
  return floats * sizeof(float);
}

frt_status frt_rope_table_fill(const frt_rope *r, float *out, size_t bytes) {
  if (!r) return fail(FRT_ERR_NULL, "rope is NULL");
  if (r->mode == FRT_ROPE_NONE) return FRT_OK;
  if (r->mode != FRT_ROPE_1D && r->mode != FRT_ROPE_3D)
    return fail(FRT_ERR_SHAPE, "rope mode %d unknown", r->mode);
  if (!out) return fail(FRT_ERR_NULL, "table output is NULL");
  const size_t need = frt_rope_table_bytes(r);
  if (bytes < need) return fail(FRT_ERR_SHAPE, "table buffer %zu < %zu bytes", bytes, need);
  const int naxes = r->mode == FRT_ROPE_1D ? 1 : 3;
  size_t off = 0;
  for (int a = 0; a < naxes; ++a) {
    const int D = r->axis_dims[a];
    if (D <= 0 || r->max_pos[a] <= 0) continue;
    const int np = D / 2;
    std::vector<double> theta(np);
    for (int i = 0; i < np; ++i) theta[i] = std::pow(r->base, -(2.0 * i) / D);
    for (int pos = 0; pos < r->max_pos[a]; ++pos)
      for (int i = 0; i < np; ++i) {
        const double ang = (double)pos * theta[i];
        out[off++] = (float)std::cos(ang);
        out[off++] = (float)std::sin(ang);
      }
  }
  return FRT_OK;
}

frt_status frt_kv_append(const frt_ring *ring, const frt_rope *rope, const void *k_new,
                         const void *v_new, int32_t n_new, void *stream) {
  frt_status s;
  if ((s = check_ring(ring)) != FRT_OK) return s;
  if ((s = check_rope(rope, ring->head_dim)) != FRT_OK) return s;
  if (n_new < 0) return fail(FRT_ERR_SHAPE, "n_new=%d < 0", n_new);
  if (n_new > ring->capacity)
    return fail(FRT_ERR_CAPACITY, "n_new=%d > capacity=%d", n_new, ring->capacity);
  if (n_new == 0) return FRT_OK;
  if ((s = check_io(k_new, "k_new")) != FRT_OK) return s;
  if ((s = check_io(v_new, "v_new")) != FRT_OK) return s;
  AppendParams p;
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  p.k_ring = static_cast<uint16_t *>(ring->k_ring);
  p.v_ring = static_cast<uint16_t *>(ring->v_ring);
  p.seq_len = ring->seq_len;
  p.B = ring->num_streams;
  p.Hkv = ring->num_kv_heads;
  p.D = ring->head_dim;
  p.C = ring->capacity;
  p.n = n_new;
  const RopeDev rd = rope_dev(rope);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (n_new <= kAppendSmall)  // one block per stream, seq_len advanced in the same launch
    return launch("rope_append", st, [&] { return launch_rope_append_small(p, rd, st); });
  if ((s = launch("rope_append", st, [&] { return launch_rope_append(p, rd, st); })) != FRT_OK)
    return s;
  return launch("seq_advance", st, [&] { return launch_seq_advance(ring->seq_len, p.B, n_new, st); });
}

size_t frt_stream_attn_workspace_bytes(const frt_ring *ring, int32_t n_new, int32_t num_q_heads) {
  if (!ring || n_new <= 0 || num_q_heads <= 0 || ring->head_dim <= 0) return 0;
  return step_layout(ring, n_new, num_q_heads).bytes;
}

namespace {

frt_status stream_impl(const frt_ring *ring, const frt_rope *rope, const frt_mask *mask,
                       const void *q, const void *k_new, const void *v_new, int32_t n_new,
                       int32_t num_q_heads, float softmax_scale, void *workspace,
                       size_t workspace_bytes, void *out, float *lse, void *stream, bool append) {
  frt_status s;
  if ((s = check_ring(ring)) != FRT_OK) return s;
  if ((s = check_rope(rope, ring->head_dim)) != FRT_OK) return s;
  if ((s = check_mask(mask, ring->capacity)) != FRT_OK) return s;
  if (num_q_heads < 1 || num_q_heads % ring->num_kv_heads)
    return fail(FRT_ERR_SHAPE, "num_q_heads=%d is not a multiple of num_kv_heads=%d", num_q_heads,
                ring->num_kv_heads);
  if (n_new < 0) return fail(FRT_ERR_SHAPE, "n_new=%d < 0", n_new);
  if (n_new > ring->capacity)
    return fail(FRT_ERR_CAPACITY, "n_new=%d > capacity=%d", n_new, ring->capacity);
  if (n_new == 0) return FRT_OK;
  const int G = num_q_heads / ring->num_kv_heads;
  if ((size_t)n_new * G * ring->head_dim * 2 >= (size_t)1 << 31)
    return fail(FRT_ERR_SHAPE, "n_new*G*head_dim*2 must be below 2^31");
  if ((s = check_io(q, "q")) != FRT_OK) return s;
  if ((s = check_io(k_new, "k_new")) != FRT_OK) return s;
  if ((s = check_io(v_new, "v_new")) != FRT_OK) return s;
  if ((s = check_io(out, "out")) != FRT_OK) return s;
  if (lse && !aligned(lse, 4)) return fail(FRT_ERR_ALIGN, "lse must be 4-byte aligned");
  const StepLayout lay = step_layout(ring, n_new, num_q_heads);
  if (!workspace) return fail(FRT_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", lay.bytes);
  if (workspace_bytes < lay.bytes)
    return fail(FRT_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, lay.bytes);
  if (!aligned(workspace, 256)) return fail(FRT_ERR_ALIGN, "workspace must be 256-byte aligned");

  char *ws = static_cast<char *>(workspace);
  PrepParams pp;
  pp.q = static_cast<const uint16_t *>(q);
  pp.k_new = static_cast<const uint16_t *>(k_new);
  pp.v_new = static_cast<const uint16_t *>(v_new);
  pp.seq_len = ring->seq_len;
  pp.qr = reinterpret_cast<uint16_t *>(ws + lay.q_off);
  pp.kr = reinterpret_cast<uint16_t *>(ws + lay.k_off);
  pp.vt = reinterpret_cast<uint16_t *>(ws + lay.v_off);
  pp.lrec = reinterpret_cast<int64_t *>(ws + lay.l_off);
  pp.B = ring->num_streams;
  pp.Hq = num_q_heads;
  pp.Hkv = ring->num_kv_heads;
  pp.G = G;
  pp.D = ring->head_dim;
  pp.n = n_new;
  pp.n_pad = lay.n_pad;
  pp.qmul = q_multiplier(softmax_scale, ring->head_dim);

  AttnParams ap;
  ap.qr = pp.qr;
  ap.kr = pp.kr;
  ap.vt = pp.vt;
  ap.k_ring = static_cast<const uint16_t *>(ring->k_ring);
  ap.v_ring = static_cast<const uint16_t *>(ring->v_ring);
  ap.seq_len = ring->seq_len;
  ap.out = static_cast<uint16_t *>(out);
  ap.lse = lse;
  ap.B = pp.B;
  ap.Hq = num_q_heads;
  ap.Hkv = pp.Hkv;
  ap.G = G;
  ap.n = n_new;
  ap.n_pad = lay.n_pad;
  ap.C = ring->capacity;
  ap.mask_kind = mask->kind;
  ap.mask_block = mask->block;
  ap.mask_window = mask->window;
  ap.row_tiles = (n_new * G + kChunkRows - 1) / kChunkRows;

  const RopeDev rd = rope_dev(rope);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((s = launch("chunk_prep", st, [&] { return launch_chunk_prep(pp, rd, st); })) != FRT_OK)
    return s;
  if ((s = launch("chunk_attn", st, [&] { return launch_chunk_attn(ap, ring->head_dim, st); })) !=
          FRT_OK ||
      !append)
    return s;
  ChunkAppendParams cp;
  cp.kr = pp.kr;
  cp.v_new = pp.v_new;
  cp.lrec = pp.lrec;
  cp.k_ring = static_cast<uint16_t *>(ring->k_ring);
  cp.v_ring = static_cast<uint16_t *>(ring->v_ring);
  cp.seq_len = ring->seq_len;
  cp.B = pp.B;
  cp.Hkv = pp.Hkv;
  cp.D = pp.D;
  cp.C = ring->capacity;
  cp.n = n_new;
  cp.n_pad = lay.n_pad;
  return launch("chunk_append", st, [&] { return launch_chunk_append(cp, st); });
}

}  // namespace

frt_status frt_stream_attn_step(const frt_ring *ring, const frt_rope *rope, const frt_mask *mask,
                                const void *q, const void *k_new, const void *v_new, int32_t n_new,
                                int32_t num_q_heads, float softmax_scale, void *workspace,
                                size_t workspace_bytes, void *out, float *lse, void *stream) {
  return stream_impl(ring, rope, mask, q, k_new, v_new, n_new, num_q_heads, softmax_scale,
                     workspace, workspace_bytes, out, lse, stream, false);
}

frt_status frt_stream_step(const frt_ring *ring, const frt_rope *rope, const frt_mask *mask,
                           const void *q, const void *k_new, const void *v_new, int32_t n_new,
                           int32_t num_q_heads, float softmax_scale, void *workspace,
                           size_t workspace_bytes, void *out, float *lse, void *stream) {
  if (ring && n_new > ring->capacity)
    return fail(FRT_ERR_CAPACITY, "n_new=%d > capacity=%d", n_new, ring->capacity);
  return stream_impl(ring, rope, mask, q, k_new, v_new, n_new, num_q_heads, softmax_scale,
                     workspace, workspace_bytes, out, lse, stream, true);
}

// ---------------------------------------------------------------- FP8 --
namespace {

struct Fp8Layout {
  size_t q_off, s_off, k_off, v_off, l_off, bytes;
  int n_pad;
};

Fp8Layout fp8_layout(const frt_ring *r, int n, int hq) {
  Fp8Layout L;
  const size_t d = (size_t)r->head_dim;
  const size_t rows = (size_t)r->num_streams * n * hq;  // query rows of all heads
  L.n_pad = (int)round_up((size_t)n, kChunkBN);
  L.q_off = 0;
  L.s_off = round_up(rows * d, 256);
  L.k_off = L.s_off + round_up(rows * 4, 256);
  L.v_off = L.k_off + round_up((size_t)r->num_streams * r->num_kv_heads * L.n_pad * d, 256);
  L.l_off = L.v_off + round_up((size_t)r->num_streams * r->num_kv_heads * L.n_pad * d, 256);
  L.bytes = L.l_off + round_up((size_t)r->num_streams * 8, 256);
  return L;
}

frt_status check_scales(const frt_fp8_scales *sc) {
  if (!sc || !sc->k_scale || !sc->v_scale) return fail(FRT_ERR_NULL, "FP8 scales are NULL");
  if (!aligned(sc->k_scale, 4) || !aligned(sc->v_scale, 4))
    return fail(FRT_ERR_ALIGN, "FP8 scales must be 4-byte aligned");
  return FRT_OK;
}

}  // namespace

frt_status frt_kv_append_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                             const frt_rope *rope, const void *k_new, const void *v_new,
                             int32_t n_new, void *stream) {
  frt_status s;
  if ((s = check_ring(ring)) != FRT_OK) return s;
  if ((s = check_scales(scales)) != FRT_OK) return s;
  if ((s = check_rope(rope, ring->head_dim)) != FRT_OK) return s;
  if (n_new < 0) return fail(FRT_ERR_SHAPE, "n_new=%d < 0", n_new);
  if (n_new > ring->capacity)
    return fail(FRT_ERR_CAPACITY, "n_new=%d > capacity=%d", n_new, ring->capacity);
  if (n_new == 0) return FRT_OK;
  if ((s = check_io(k_new, "k_new")) != FRT_OK) return s;
  if ((s = check_io(v_new, "v_new")) != FRT_OK) return s;
  AppendFp8Params p;
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  p.k_ring = static_cast<uint8_t *>(ring->k_ring);
  p.v_ring = static_cast<uint8_t *>(ring->v_ring);
  p.seq_len = ring->seq_len;
  p.sc.k = scales->k_scale;
  p.sc.v = scales->v_scale;
  p.B = ring->num_streams;
  p.Hkv = ring->num_kv_heads;
  p.D = ring->head_dim;
  p.C = ring->capacity;
  p.n = n_new;
  const RopeDev rd = rope_dev(rope);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((s = launch("rope_append", st, [&] { return launch_rope_append_fp8(p, rd, st); })) != FRT_OK)
    return s;
  return launch("seq_advance", st, [&] { return launch_seq_advance(ring->seq_len, p.B, n_new, st); });
}

size_t frt_stream_attn_fp8_workspace_bytes(const frt_ring *ring, int32_t n_new,
                                           int32_t num_q_heads) {
  if (!ring || n_new <= 0 || num_q_heads <= 0 || ring->head_dim <= 0) return 0;
  return fp8_layout(ring, n_new, num_q_heads).bytes;
}

}  // extern "C"

namespace {

// The FP8 step: preparation and attention, then (append) the chunk's codes
// into the ring and seq_len advanced, in one launch.
frt_status stream_fp8_impl(const frt_ring *ring, const frt_fp8_scales *scales,
                           const frt_rope *rope, const frt_mask *mask, const void *q,
                           const void *k_new, const void *v_new, int32_t n_new,
                           int32_t num_q_heads, float softmax_scale, void *workspace,
                           size_t workspace_bytes, void *out, float *lse, void *stream,
                           bool append) {
  frt_status s;
  if ((s = check_ring(ring)) != FRT_OK) return s;
  if ((s = check_scales(scales)) != FRT_OK) return s;
  if (ring->head_dim != 128)
    return fail(FRT_ERR_UNSUPPORTED, "FP8 attention supports head_dim 128 (got %d)",
                ring->head_dim);
  if ((s = check_rope(rope, ring->head_dim)) != FRT_OK) return s;
  if ((s = check_mask(mask, ring->capacity)) != FRT_OK) return s;
  if (num_q_heads < 1 || num_q_heads % ring->num_kv_heads)
    return fail(FRT_ERR_SHAPE, "num_q_heads=%d is not a multiple of num_kv_heads=%d", num_q_heads,
                ring->num_kv_heads);
  if (n_new < 0) return fail(FRT_ERR_SHAPE, "n_new=%d < 0", n_new);
  if (n_new > ring->capacity)
    return fail(FRT_ERR_CAPACITY, "n_new=%d > capacity=%d", n_new, ring->capacity);
  if (n_new == 0) return FRT_OK;
  const int G = num_q_heads / ring->num_kv_heads;
  if ((size_t)n_new * G * ring->head_dim >= (size_t)1 << 31)
    return fail(FRT_ERR_SHAPE, "n_new*G*head_dim must be below 2^31");
  if ((s = check_io(q, "q")) != FRT_OK) return s;
  if ((s = check_io(k_new, "k_new")) != FRT_OK) return s;
  if ((s = check_io(v_new, "v_new")) != FRT_OK) return s;
  if ((s = check_io(out, "out")) != FRT_OK) return s;
  if (lse && !aligned(lse, 4)) return fail(FRT_ERR_ALIGN, "lse must be 4-byte aligned");
  const Fp8Layout lay = fp8_layout(ring, n_new, num_q_heads);
  if (!workspace) return fail(FRT_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", lay.bytes);
  if (workspace_bytes < lay.bytes)
    return fail(FRT_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, lay.bytes);
  if (!aligned(workspace, 256)) return fail(FRT_ERR_ALIGN, "workspace must be 256-byte aligned");

  char *ws = static_cast<char *>(workspace);
  PrepFp8Params pp;
  pp.q = static_cast<const uint16_t *>(q);
  pp.k_new = static_cast<const uint16_t *>(k_new);
  pp.v_new = static_cast<const uint16_t *>(v_new);
  pp.seq_len = ring->seq_len;
  pp.qr = reinterpret_cast<uint8_t *>(ws + lay.q_off);
  pp.qs = reinterpret_cast<float *>(ws + lay.s_off);
  pp.kr = reinterpret_cast<uint8_t *>(ws + lay.k_off);
  pp.vt = reinterpret_cast<uint8_t *>(ws + lay.v_off);
  pp.lrec = reinterpret_cast<int64_t *>(ws + lay.l_off);
  pp.sc.k = scales->k_scale;
  pp.sc.v = scales->v_scale;
  pp.B = ring->num_streams;
  pp.Hq = num_q_heads;
  pp.Hkv = ring->num_kv_heads;
  pp.G = G;
  pp.D = ring->head_dim;
  pp.n = n_new;
  pp.n_pad = lay.n_pad;
  pp.qmul = q_multiplier(softmax_scale, ring->head_dim);

  AttnFp8Params ap;
  ap.qr = pp.qr;
  ap.qs = pp.qs;
  ap.kr = pp.kr;
  ap.vt = pp.vt;
  ap.k_ring = static_cast<const uint8_t *>(ring->k_ring);
  ap.v_ring = static_cast<const uint8_t *>(ring->v_ring);
  ap.seq_len = ring->seq_len;
  ap.sc = pp.sc;
  ap.out = static_cast<uint16_t *>(out);
  ap.lse = lse;
  ap.B = pp.B;
  ap.Hq = num_q_heads;
  ap.Hkv = pp.Hkv;
  ap.G = G;
  ap.n = n_new;
  ap.n_pad = lay.n_pad;
  ap.C = ring->capacity;
  ap.mask_kind = mask->kind;
  ap.mask_block = mask->block;
  ap.mask_window = mask->window;
  ap.row_tiles = (n_new * G + kChunkRows - 1) / kChunkRows;

  const RopeDev rd = rope_dev(rope);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((s = launch("chunk_prep", st, [&] { return launch_chunk_prep_fp8(pp, rd, st); })) != FRT_OK)
    return s;
  if ((s = launch("chunk_attn", st, [&] { return launch_chunk_attn_fp8(ap, ring->head_dim, st); })) !=
      FRT_OK)
    return s;
  if (!append) return FRT_OK;
  ChunkAppendFp8Params cp;
  cp.kr = pp.kr;
  cp.vt = pp.vt;
  cp.lrec = pp.lrec;
  cp.k_ring = static_cast<uint8_t *>(ring->k_ring);
  cp.v_ring = static_cast<uint8_t *>(ring->v_ring);
  cp.seq_len = ring->seq_len;
  cp.B = pp.B;
  cp.Hkv = pp.Hkv;
  cp.D = ring->head_dim;
  cp.C = ring->capacity;
  cp.n = n_new;
  cp.n_pad = lay.n_pad;
  return launch("chunk_append", st, [&] { return launch_chunk_append_fp8(cp, st); });
}

}  // namespace

extern "C" {

frt_status frt_stream_attn_step_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                                    const frt_rope *rope, const frt_mask *mask, const void *q,
                                    const void *k_new, const void *v_new, int32_t n_new,
                                    int32_t num_q_heads, float softmax_scale, void *workspace,
                                    size_t workspace_bytes, void *out, float *lse, void *stream) {
  return stream_fp8_impl(ring, scales, rope, mask, q, k_new, v_new, n_new, num_q_heads,
                         softmax_scale, workspace, workspace_bytes, out, lse, stream, false);
}

size_t frt_decode_fp8_workspace_bytes(const frt_ring *ring, int32_t num_q_heads) {
  if (!ring || ring->num_kv_heads <= 0 || num_q_heads <= 0 || ring->head_dim <= 0) return 0;
  const int G = num_q_heads / ring->num_kv_heads;
  // a partial per piece wave, and one per (stream, KV head) for its own token
  const size_t heads = (size_t)ring->num_streams * ring->num_kv_heads;
  return ((size_t)frt_decode_max_splits(ring) + heads) *
         decode_fp8_split_floats(G, ring->head_dim) * sizeof(float);
}

}  // extern "C"

namespace {

frt_status decode_fp8_impl(const frt_ring *ring, const frt_fp8_scales *scales,
                           const frt_rope *rope, const frt_mask *mask, const void *q,
                           const void *k_new, const void *v_new, int32_t num_q_heads,
                           float softmax_scale, void *workspace, size_t workspace_bytes,
                           void *out, float *lse, void *stream, bool append) {
  frt_status s;
  if ((s = check_ring(ring)) != FRT_OK) return s;
  if ((s = check_scales(scales)) != FRT_OK) return s;
  if (ring->head_dim != 128)
    return fail(FRT_ERR_UNSUPPORTED, "FP8 decode supports head_dim 128 (got %d)",
                ring->head_dim);
  if ((s = check_rope(rope, ring->head_dim)) != FRT_OK) return s;
  if ((s = check_mask(mask, ring->capacity)) != FRT_OK) return s;
  if (num_q_heads < 1 || num_q_heads % ring->num_kv_heads)
    return fail(FRT_ERR_SHAPE, "num_q_heads=%d is not a multiple of num_kv_heads=%d", num_q_heads,
                ring->num_kv_heads);
  const int G = num_q_heads / ring->num_kv_heads;
  if (G > 16) return fail(FRT_ERR_UNSUPPORTED, "decode supports up to 16 query heads per KV head");
  if ((s = check_io(q, "q")) != FRT_OK) return s;
  if ((s = check_io(k_new, "k_new")) != FRT_OK) return s;
  if ((s = check_io(v_new, "v_new")) != FRT_OK) return s;
  if ((s = check_io(out, "out")) != FRT_OK) return s;
  if (lse && !aligned(lse, 4)) return fail(FRT_ERR_ALIGN, "lse must be 4-byte aligned");
  const size_t need = frt_decode_fp8_workspace_bytes(ring, num_q_heads);
  if (!workspace) return fail(FRT_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (workspace_bytes < need)
    return fail(FRT_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, need);
  if (!aligned(workspace, 16)) return fail(FRT_ERR_ALIGN, "workspace must be 16-byte aligned");

  DecodeFp8Params p;
  p.q = static_cast<const uint16_t *>(q);
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  p.k_ring = static_cast<uint8_t *>(ring->k_ring);
  p.v_ring = static_cast<uint8_t *>(ring->v_ring);
  p.seq_len = ring->seq_len;
  p.sc.k = scales->k_scale;
  p.sc.v = scales->v_scale;
  p.ws = static_cast<float *>(workspace);
  p.out = static_cast<uint16_t *>(out);
  p.lse = lse;
  p.B = ring->num_streams;
  p.Hq = num_q_heads;
  p.Hkv = ring->num_kv_heads;
  p.G = G;
  p.D = ring->head_dim;
  p.C = ring->capacity;
  p.nwaves = frt_decode_max_splits(ring);
  p.mask_kind = mask->kind;
  p.mask_block = mask->block;
  p.mask_window = mask->window;
  p.append = append ? 1 : 0;
  p.qmul = q_multiplier(softmax_scale, ring->head_dim);
  const RopeDev rd = rope_dev(rope);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((s = launch("decode_split", st, [&] { return launch_decode_split_fp8(p, rd, st); })) !=
      FRT_OK)
    return s;
  return launch("decode_combine", st, [&] { return launch_decode_combine_fp8(p, st); });
}

}  // namespace

extern "C" {

frt_status frt_decode_attn_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                               const frt_rope *rope, const frt_mask *mask, const void *q,
                               const void *k_new, const void *v_new, int32_t num_q_heads,
                               float softmax_scale, void *workspace, size_t workspace_bytes,
                               void *out, float *lse, void *stream) {
  return decode_fp8_impl(ring, scales, rope, mask, q, k_new, v_new, num_q_heads, softmax_scale,
                         workspace, workspace_bytes, out, lse, stream, false);
}

frt_status frt_decode_step_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                               const frt_rope *rope, const frt_mask *mask, const void *q,
                               const void *k_new, const void *v_new, int32_t num_q_heads,
                               float softmax_scale, void *workspace, size_t workspace_bytes,
                               void *out, float *lse, void *stream) {
  return decode_fp8_impl(ring, scales, rope, mask, q, k_new, v_new, num_q_heads, softmax_scale,
                         workspace, workspace_bytes, out, lse, stream, true);
}

frt_status frt_stream_step_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                               const frt_rope *rope, const frt_mask *mask, const void *q,
                               const void *k_new, const void *v_new, int32_t n_new,
                               int32_t num_q_heads, float softmax_scale, void *workspace,
                               size_t workspace_bytes, void *out, float *lse, void *stream) {
  return stream_fp8_impl(ring, scales, rope, mask, q, k_new, v_new, n_new, num_q_heads,
                         softmax_scale, workspace, workspace_bytes, out, lse, stream, true);
}

int32_t frt_decode_max_splits(const frt_ring *ring) {
  if (!ring || ring->capacity <= 0 || ring->num_streams <= 0 || ring->num_kv_heads <= 0) return 0;
  return decode_piece_waves(ring->num_streams, ring->num_kv_heads, ring->capacity);
}

size_t frt_decode_workspace_bytes(const frt_ring *ring, int32_t num_q_heads) {
  if (!ring || ring->num_kv_heads <= 0 || num_q_heads <= 0 || ring->head_dim <= 0) return 0;
  const int G = num_q_heads / ring->num_kv_heads;
  // a partial per piece wave, and one per (stream, KV head) for its own token
  const size_t heads = (size_t)ring->num_streams * ring->num_kv_heads;
  return ((size_t)frt_decode_max_splits(ring) + heads) * decode_split_floats(G, ring->head_dim) *
         sizeof(float);
}

namespace {

frt_status decode_impl(const frt_ring *ring, const frt_rope *rope, const frt_mask *mask,
                       const void *q, const void *k_new, const void *v_new, int32_t num_q_heads,
                       float softmax_scale, void *workspace, size_t workspace_bytes, void *out,
                       float *lse, void *stream, bool append) {
  frt_status s;
  if ((s = check_ring(ring)) != FRT_OK) return s;
  if ((s = check_rope(rope, ring->head_dim)) != FRT_OK) return s;
  if ((s = check_mask(mask, ring->capacity)) != FRT_OK) return s;
  if (num_q_heads < 1 || num_q_heads % ring->num_kv_heads)
    return fail(FRT_ERR_SHAPE, "num_q_heads=%d is not a multiple of num_kv_heads=%d", num_q_heads,
                ring->num_kv_heads);
  const int G = num_q_heads / ring->num_kv_heads;
  if (G > 16) return fail(FRT_ERR_UNSUPPORTED, "decode supports up to 16 query heads per KV head");
  if ((s = check_io(q, "q")) != FRT_OK) return s;
  if ((s = check_io(k_new, "k_new")) != FRT_OK) return s;
  if ((s = check_io(v_new, "v_new")) != FRT_OK) return s;
  if ((s = check_io(out, "out")) != FRT_OK) return s;
  if (lse && !aligned(lse, 4)) return fail(FRT_ERR_ALIGN, "lse must be 4-byte aligned");
  const size_t need = frt_decode_workspace_bytes(ring, num_q_heads);
  if (!workspace) return fail(FRT_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (workspace_bytes < need)
    return fail(FRT_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, need);
  if (!aligned(workspace, 16)) return fail(FRT_ERR_ALIGN, "workspace must be 16-byte aligned");

  DecodeParams p;
  p.q = static_cast<const uint16_t *>(q);
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  p.k_ring = static_cast<uint16_t *>(ring->k_ring);
  p.v_ring = static_cast<uint16_t *>(ring->v_ring);
  p.seq_len = ring->seq_len;
  p.ws = static_cast<float *>(workspace);
  p.append = append ? 1 : 0;
  p.out = static_cast<uint16_t *>(out);
  p.lse = lse;
  p.B = ring->num_streams;
  p.Hq = num_q_heads;
  p.Hkv = ring->num_kv_heads;
  p.G = G;
  p.D = ring->head_dim;
  p.C = ring->capacity;
  p.nwaves = frt_decode_max_splits(ring);
  p.mask_kind = mask->kind;
  p.mask_block = mask->block;
  p.mask_window = mask->window;
  p.qmul = q_multiplier(softmax_scale, ring->head_dim);
  const RopeDev rd = rope_dev(rope);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((s = launch("decode_split", st, [&] { return launch_decode_split(p, rd, st); })) != FRT_OK)
    return s;
  return launch("decode_combine", st, [&] { return launch_decode_combine(p, st); });
}

}  // namespace

frt_status frt_decode_attn(const frt_ring *ring, const frt_rope *rope, const frt_mask *mask,
                           const void *q, const void *k_new, const void *v_new,
                           int32_t num_q_heads, float softmax_scale, void *workspace,
                           size_t workspace_bytes, void *out, float *lse, void *stream) {
  return decode_impl(ring, rope, mask, q, k_new, v_new, num_q_heads, softmax_scale, workspace,
                     workspace_bytes, out, lse, stream, false);
}

frt_status frt_decode_step(const frt_ring *ring, const frt_rope *rope, const frt_mask *mask,
                           const void *q, const void *k_new, const void *v_new,
                           int32_t num_q_heads, float softmax_scale, void *workspace,
                           size_t workspace_bytes, void *out, float *lse, void *stream) {
  return decode_impl(ring, rope, mask, q, k_new, v_new, num_q_heads, softmax_scale, workspace,
                     workspace_bytes, out, lse, stream, true);
}

}  // extern "C"

// ------------------------------------------- no-allocation decode step --
// Device scratch of frt_decode_step_noalloc: file scope, one copy on every
// GPU the library runs on, held until the process ends. Host code never
// passes the array's name to a kernel (on the host it is a stand-in, not a
// device address); it uses the address hipGetSymbolAddress returns for the
// current device, looked up once per device.
static __device__ __align__(256) unsigned char scratch[FRT_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices] = {};

// This device's address of `scratch`, for a launch on `stream`.
frt_status scratch_address(void *stream, void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0)
    return fail(FRT_ERR_HIP, "hipGetDevice failed");
  if (dev >= kMaxDevices) return fail(FRT_ERR_UNSUPPORTED, "device %d: at most %d devices", dev,
                                      kMaxDevices);
  if (stream != nullptr) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev) != hipSuccess)
      return fail(FRT_ERR_HIP, "hipStreamGetDevice failed");
    if (sdev != dev)
      return fail(FRT_ERR_UNSUPPORTED, "the stream belongs to device %d but device %d is current",
                  (int)sdev, dev);
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || ptr == nullptr)
      return fail(FRT_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d failed: %s", dev,
                  hipGetErrorString(e));
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return FRT_OK;
}

}  // namespace

extern "C" {

frt_status frt_decode_step_noalloc(const frt_ring *ring, const frt_rope *rope,
                                   const frt_mask *mask, const void *q, const void *k_new,
                                   const void *v_new, int32_t num_q_heads, float softmax_scale,
                                   void *out, float *lse, void *stream) {
  const size_t need = frt_decode_workspace_bytes(ring, num_q_heads);
  if (need > (size_t)FRT_NOALLOC_SCRATCH_BYTES)
    return fail(FRT_ERR_WORKSPACE,
                "decode needs %zu bytes of scratch; frt_decode_step_noalloc holds %zu",
                need, (size_t)FRT_NOALLOC_SCRATCH_BYTES);
  void *ws = nullptr;
  frt_status s = scratch_address(stream, &ws);
  if (s != FRT_OK) return s;
  return decode_impl(ring, rope, mask, q, k_new, v_new, num_q_heads, softmax_scale, ws,
                     (size_t)FRT_NOALLOC_SCRATCH_BYTES, out, lse, stream, true);
}

frt_status frt_timing_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = on != 0;
  return FRT_OK;
}

frt_status frt_timing_query(const char *kernel, int32_t *count, double *total_ms) {
  if (!kernel || !count || !total_ms) return fail(FRT_ERR_NULL, "timing query argument is NULL");
  std::lock_guard<std::mutex> lk(g_tmu);
  int c = 0;
  double tot = 0.0;
  for (const TimingRec &r : g_recs) {
    if (std::strcmp(r.name, kernel) != 0) continue;
    if (hipEventSynchronize(r.stop) != hipSuccess)
      return fail(FRT_ERR_HIP, "hipEventSynchronize failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
      return fail(FRT_ERR_HIP, "hipEventElapsedTime failed");
    tot += ms;
    ++c;
  }
  *count = c;
  *total_ms = tot;
  return FRT_OK;
}

frt_status frt_timing_samples(const char *kernel, float *ms_out, int32_t capacity,
                              int32_t *count) {
  if (!kernel || !count || (capacity > 0 && !ms_out))
    return fail(FRT_ERR_NULL, "timing samples argument is NULL");
  std::lock_guard<std::mutex> lk(g_tmu);
  int c = 0;
  for (const TimingRec &r : g_recs) {
    if (std::strcmp(r.name, kernel) != 0) continue;
    if (c < capacity) {
      if (hipEventSynchronize(r.stop) != hipSuccess)
        return fail(FRT_ERR_HIP, "hipEventSynchronize failed");
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
        return fail(FRT_ERR_HIP, "hipEventElapsedTime failed");
      ms_out[c] = ms;
    }
    ++c;
  }
  *count = c;
  return FRT_OK;
}

void frt_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_tmu);
  for (const TimingRec &r : g_recs) {
    (void)hipEventSynchronize(r.stop);
    g_pool.push_back(r.start);
    g_pool.push_back(r.stop);
  }
  g_recs.clear();
}

}  // extern "C"
