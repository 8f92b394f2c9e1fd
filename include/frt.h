/*
 * frt.h - chunk-streamed attention over per-stream ring-buffer KV caches,
 * C ABI of libfrt.so (HIP, gfx950 / MI355X).
 *
 * What a streaming step is. The FlashRT paper models a real-time pipeline as
 * a task graph processed batch by batch; a node of batch j may depend on the
 * persistent state its own instance left behind in batch j-1 (Problem
 * Formulation: cross-batch lambda=1 edges, whose example is an attention
 * key/value cache carried from one batch to the next; Chain-of-Program, IR
 * design: node-level persistent-state read/write annotations; appendix
 * "Formal Analysis of Pipeline Graphs"). In the
 * autoregressive video DiTs and multimodal LLMs the paper deploys, that state
 * is the attention KV cache, and each step's new query chunk attends to the
 * cached keys plus its own. This library implements that step:
 *
 *   frt_stream_attn_step  READS the ring: out = attention(q, ring keys + own keys)
 *   frt_stream_step       frt_stream_attn_step then frt_kv_append, fused
 *   frt_decode_attn       the same for one token per stream (split-KV + combine)
 *   frt_decode_step       frt_decode_attn then frt_kv_append, fused (decode loop)
 *   frt_kv_append         WRITES the ring: stores the chunk's RoPE'd K and its V
 *
 * A step is frt_stream_attn_step (or frt_decode_attn) followed by
 * frt_kv_append on the same HIP stream, or one frt_stream_step / frt_decode_step. Attention never sees the chunk through
 * the ring: it reads k_new / v_new directly, so a ring whose capacity equals
 * the visible window works even though the append then overwrites the oldest
 * visible chunk.
 *
 * Arithmetic (the paper gives none; standard definitions):
 *   score(p, k) = (rot(q_p, p) . K_k) * scale, scale = 1/sqrt(d) by default;
 *   out_p = sum_k softmax_k(score) V_k over the keys visible to p;
 *   rot: rotary embedding (RoFormer) on interleaved pairs (x[2i], x[2i+1]) by
 *   angle pos * theta_i, theta_i = base^(-2i/D); 3D variant: the head
 *   dimension is split into t/h/w slices, each rotated by that coordinate of
 *   the token in a latent frame of H x W tokens (raster order).
 * Stored keys are bit-exact: K = bf16(fp32(rot_fp64(k))) with fp32 cos/sin
 * from frt_rope_table_fill and round-to-nearest-even at both roundings.
 *
 * Memory. Every buffer is owned by the caller; the library keeps no device
 * allocations. Device pointers must be 16-byte aligned. bf16 is stored as
 * 16-bit IEEE bfloat16 bit patterns. Calls are asynchronous on the given
 * hipStream_t (NULL = the null stream) and never synchronise the host,
 * except frt_timing_query.
 *
 * Errors. Every entry point validates its arguments on the host before
 * launching anything; on failure it returns a non-zero frt_status, launches
 * nothing and sets a thread-local message (frt_last_error). A failed launch
 * returns FRT_ERR_HIP. Conditions the host cannot see (values of the device
 * array seq_len) are caller contracts, stated per call.
 */
#ifndef FRT_H_
#define FRT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FRT_OK = 0,
  FRT_ERR_NULL = 1,         /* a required pointer is NULL */
  FRT_ERR_SHAPE = 2,        /* a size is out of range or inconsistent */
  FRT_ERR_UNSUPPORTED = 3,  /* valid but not implemented (e.g. head_dim 96) */
  FRT_ERR_CAPACITY = 4,     /* ring capacity too small for n_new or the window */
  FRT_ERR_ALIGN = 5,        /* capacity not a multiple of 8, or misaligned pointer */
  FRT_ERR_WORKSPACE = 6,    /* workspace missing or smaller than required */
  FRT_ERR_HIP = 7           /* a HIP launch/runtime call failed */
} frt_status;

enum { FRT_ROPE_NONE = 0, FRT_ROPE_1D = 1, FRT_ROPE_3D = 2 };
enum { FRT_MASK_BLOCK_CAUSAL = 1, FRT_MASK_CAUSAL = 2 };

/*
 * Persistent per-stream state (the paper's cross-batch KV-cache state).
 * Token t of stream b lives in slot t mod capacity. seq_len[b] counts the
 * tokens ever appended to stream b; the tokens still held are
 * [max(0, seq_len-capacity), seq_len).
 *   k_ring : bf16 [num_streams][num_kv_heads][capacity][head_dim]   (row per slot)
 *   v_ring : bf16 [num_streams][num_kv_heads][capacity*head_dim] in blocks of
 *            32 slots: block k (slots 32k ..) starts at element 32*head_dim*k of
 *            the head and holds its slots row by row of the head dimension, so
 *            (slot s, dim d) is element 32*head_dim*(s/32) + w*d + s%32, where
 *            w = 32 for a full block and w = capacity%32 for a partial last one.
 *            The 32 keys of one block are one contiguous 64*head_dim-byte run.
 *   seq_len: int64 [num_streams], device memory.
 * head_dim is 64 or 128; capacity is a positive multiple of 8. A new ring
 * must be zero-filled with seq_len = 0 (slot contents must stay finite:
 * never-written and masked slots are multiplied by a zero weight).
 * The per-head size capacity*head_dim*2 bytes must be below 2^31.
 */
typedef struct {
  int32_t num_streams;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t capacity;
  void *k_ring;
  void *v_ring;
  int64_t *seq_len;
} frt_ring;

/*
 * Rotary embedding description.
 *   mode FRT_ROPE_NONE: no rotation (table unused, may be NULL).
 *   mode FRT_ROPE_1D  : axis_dims = {D, 0, 0}, D even, D <= head_dim; pairs
 *                       beyond D/2 are not rotated. max_pos[0] = positions held.
 *   mode FRT_ROPE_3D  : axis_dims = {Dt, Dh, Dw}, each even, sum <= head_dim;
 *                       frame_hw = {H, W}; token p has coordinates
 *                       (p div HW, (p mod HW) div W, p mod W);
 *                       max_pos = {frames, H, W} held in the table.
 *   base: theta base (10000 in the paper's models).
 *   table: device copy of the buffer written by frt_rope_table_fill; its size
 *          frt_rope_table_bytes(rope) must be below 2^31 (FRT_ERR_SHAPE).
 * Contract: every token position rotated by a call lies inside max_pos
 * (positions beyond it are clamped to the last table row, which is wrong but
 * never reads out of bounds).
 */
typedef struct {
  int32_t mode;
  int32_t axis_dims[3];
  int32_t frame_hw[2];
  int32_t max_pos[3];
  double base;
  const float *table;
} frt_rope;

/*
 * Visibility of key token k to query token p.
 *   FRT_MASK_BLOCK_CAUSAL: block = tokens per block (>= 1), window = blocks
 *       (0 = unlimited): visible iff k div block <= p div block and
 *       (window = 0 or p div block - k div block <= window).
 *   FRT_MASK_CAUSAL: window = keys including self (0 = unlimited):
 *       visible iff k <= p and (window = 0 or p - k < window).
 */
typedef struct {
  int32_t kind;
  int32_t block;
  int32_t window;
} frt_mask;

/* Bytes of the rotary table for `rope` (0 for FRT_ROPE_NONE or bad input). */
size_t frt_rope_table_bytes(const frt_rope *rope);

/*
 * Fill host memory `host_out` (frt_rope_table_bytes(rope) bytes) with the
 * rotary table: for each axis a in order, for pos < max_pos[a] and pair
 * i < axis_dims[a]/2, the float pair (cos(pos*theta), sin(pos*theta)) with
 * theta = base^(-2i/axis_dims[a]); cos/sin are evaluated in double by the C
 * library and rounded to float. The caller copies it to device memory and
 * sets rope->table. Host-only; launches nothing.
 */
frt_status frt_rope_table_fill(const frt_rope *rope, float *host_out, size_t bytes);

/*
 * Append n_new tokens to every stream (a write of the persistent state).
 *   k_new, v_new: bf16 [num_streams][n_new][num_kv_heads][head_dim], device.
 * For stream b with L = seq_len[b] and i < n_new: slot (L+i) mod capacity
 * receives K = bf16(fp32(rot_fp64(k_new, L+i))) and V = v_new (bytes
 * copied); then seq_len[b] = L + n_new. Other slots keep their bytes.
 * Requires 1 <= n_new <= capacity (n_new = 0 is a no-op returning FRT_OK).
 */
frt_status frt_kv_append(const frt_ring *ring, const frt_rope *rope,
                         const void *k_new, const void *v_new, int32_t n_new,
                         void *hip_stream);

/*
 * Workspace bytes frt_stream_attn_step and frt_stream_step need: the chunk's
 * rotated, scaled queries and own keys and its own values in the ring's block
 * layout (bf16), and each stream's seq_len at the step's start, rounded up.
 */
size_t frt_stream_attn_workspace_bytes(const frt_ring *ring, int32_t n_new,
                                       int32_t num_q_heads);

/*
 * One streaming step's attention (a read of the persistent state).
 *   q    : bf16 [num_streams][n_new][num_q_heads][head_dim]
 *   k_new, v_new: bf16 [num_streams][n_new][num_kv_heads][head_dim]
 *   out  : bf16 [num_streams][n_new][num_q_heads][head_dim]
 *   lse  : float [num_streams][num_q_heads][n_new] natural-log sum-exp of the
 *          scaled scores, or NULL.
 * Query head h uses KV head h / (num_q_heads / num_kv_heads). Query i of
 * stream b is token L+i (L = seq_len[b]); its keys are the ring tokens still
 * held plus the own tokens L..L+n_new-1, filtered by `mask`. softmax_scale
 * <= 0 selects 1/sqrt(head_dim). The ring is not modified.
 * Host-checked: num_q_heads % num_kv_heads == 0; n_new <= capacity;
 * block-causal window*block <= capacity; causal window-1 <= capacity.
 * Caller contract: no visible key has been evicted (with an unlimited window
 * the stream must hold all its tokens, seq_len <= capacity).
 * Numerics: bf16 inputs, fp32 accumulation, bf16 output.
 */
frt_status frt_stream_attn_step(const frt_ring *ring, const frt_rope *rope,
                                const frt_mask *mask, const void *q,
                                const void *k_new, const void *v_new,
                                int32_t n_new, int32_t num_q_heads,
                                float softmax_scale, void *workspace,
                                size_t workspace_bytes, void *out, float *lse,
                                void *hip_stream);

/*
 * A whole streaming step: exactly frt_stream_attn_step followed by
 * frt_kv_append(k_new, v_new, n_new) on the same stream (same outputs, same
 * ring bytes and seq_len afterwards). The append copies the keys the step
 * has already rotated and rounded as the ring stores them from the workspace,
 * with the values from v_new, and advances seq_len in the same launch: three
 * launches instead of four, and no second rotation. The append
 * runs after the attention launch has finished reading the ring (the oldest
 * visible chunk may occupy the slots it overwrites). Arguments, workspace
 * and errors as for frt_stream_attn_step; n_new <= capacity.
 */
frt_status frt_stream_step(const frt_ring *ring, const frt_rope *rope,
                           const frt_mask *mask, const void *q,
                           const void *k_new, const void *v_new,
                           int32_t n_new, int32_t num_q_heads,
                           float softmax_scale, void *workspace,
                           size_t workspace_bytes, void *out, float *lse,
                           void *hip_stream);

/* Largest number of KV pieces a decode call splits the ring into (one
 * partial each): every (stream, KV head) is cut into pieces of consecutive
 * 32-token tiles, sized on the device so that the pieces spread evenly over
 * the waves that run at once. Depends on num_streams, num_kv_heads and
 * capacity only. */
int32_t frt_decode_max_splits(const frt_ring *ring);

/* Workspace bytes frt_decode_attn needs: an fp32 partial (max, sum, output
 * per query head of the group) for each of frt_decode_max_splits pieces and
 * one per (stream, KV head) holding the step's own token. Its contents need
 * no initialisation; calls sharing a workspace must be ordered on one
 * stream. */
size_t frt_decode_workspace_bytes(const frt_ring *ring, int32_t num_q_heads);

/*
 * One-token decode step for every stream: frt_stream_attn_step with
 * n_new = 1, computed as split-KV (each piece of the visible ring tokens, and
 * the own token on its own, yields a partial max/sum/output per query head)
 * followed by a combine pass, one block per (stream, KV head). Same tensor
 * layouts with n_new = 1. num_q_heads / num_kv_heads must be <= 16.
 */
frt_status frt_decode_attn(const frt_ring *ring, const frt_rope *rope,
                           const frt_mask *mask, const void *q,
                           const void *k_new, const void *v_new,
                           int32_t num_q_heads, float softmax_scale,
                           void *workspace, size_t workspace_bytes, void *out,
                           float *lse, void *hip_stream);

/*
 * A whole one-token decode step: exactly frt_decode_attn followed by
 * frt_kv_append(k_new, v_new, n_new = 1) on the same stream (same outputs,
 * same ring bytes and seq_len afterwards), in two launches instead of three:
 * the combine pass also writes each head's slot seq_len mod capacity and
 * advances seq_len, which is safe because every read of the ring and of
 * seq_len happens in the split pass before it. Arguments, workspace and
 * errors as for frt_decode_attn; on an error nothing is launched and the ring
 * is unchanged.
 */
frt_status frt_decode_step(const frt_ring *ring, const frt_rope *rope,
                           const frt_mask *mask, const void *q,
                           const void *k_new, const void *v_new,
                           int32_t num_q_heads, float softmax_scale,
                           void *workspace, size_t workspace_bytes, void *out,
                           float *lse, void *hip_stream);

/*
 * frt_decode_step without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation). The split partials live in a fixed
 * device array of FRT_NOALLOC_SCRATCH_BYTES bytes inside the library, one per
 * GPU, held until the process ends; the call allocates nothing. Calls on one
 * GPU share that array, so calls that overlap on one GPU (different streams
 * with no ordering between them) race and must not be made; calls ordered on
 * one stream are fine. The stream must belong to the current device.
 * Returns FRT_ERR_WORKSPACE when frt_decode_workspace_bytes(ring,
 * num_q_heads) exceeds FRT_NOALLOC_SCRATCH_BYTES (e.g. 32 streams x 4 KV
 * heads x 8 query heads per KV head at head_dim 128 need 9.6 MB), otherwise
 * behaves exactly as frt_decode_step.
 */
#define FRT_NOALLOC_SCRATCH_BYTES (32u << 20)
frt_status frt_decode_step_noalloc(const frt_ring *ring, const frt_rope *rope,
                                   const frt_mask *mask, const void *q,
                                   const void *k_new, const void *v_new,
                                   int32_t num_q_heads, float softmax_scale,
                                   void *out, float *lse, void *hip_stream);

/*
 * FP8 variant (the FP8 KV cache with FP8 Q.K^T and P.V). The ring holds
 * OCP e4m3fn codes (1 sign, 4 exponent bits with bias 7, 3 mantissa bits;
 * largest finite 448, 0x7f / 0xff NaN), same layouts as above with one-byte
 * elements. A code c of stream b, KV head h stands for value(c) * scale:
 *   k_scale, v_scale: fp32 [num_streams][num_kv_heads], device memory, > 0.
 * Coding: x / scale in fp32, clamped to +-448, rounded to nearest (ties to
 * the even code); keys are rotated as for the bf16 ring and rounded to fp32
 * before the division. Not a paper passage: the format and rounding follow
 * the OCP 8-bit floating point specification.
 */
typedef struct {
  const float *k_scale;
  const float *v_scale;
} frt_fp8_scales;

/* frt_kv_append for an FP8 ring: the same slots and seq_len update, the
 * values stored as codes. head_dim 64 or 128. */
frt_status frt_kv_append_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                             const frt_rope *rope, const void *k_new,
                             const void *v_new, int32_t n_new, void *hip_stream);

/* Workspace bytes frt_stream_attn_step_fp8 and frt_stream_step_fp8 need:
 * query codes and their row scales, the chunk's own key and value codes, and
 * each stream's starting position. */
size_t frt_stream_attn_fp8_workspace_bytes(const frt_ring *ring, int32_t n_new,
                                           int32_t num_q_heads);

/*
 * frt_stream_attn_step over an FP8 ring (head_dim 128). Queries are rotated
 * and scaled to base-2 score units in double, rounded to fp32 and coded with
 * a power-of-two scale per query row (the smallest 2^e with max|a| <= 448 *
 * 2^e); the chunk's own keys and values are coded as the append will store
 * them. Both contractions are FP8 MFMAs with fp32 accumulation; the
 * attention weights are coded too, p = code(2^(s - m + 7)) with m the
 * smallest integer >= the row's largest score (s in base-2 units), and
 * out = v_scale * sum(p v) / sum(p) with both sums over the coded weights. Same tensors, checks and errors as
 * frt_stream_attn_step, plus FRT_ERR_UNSUPPORTED for head_dim != 128.
 */
frt_status frt_stream_attn_step_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                                    const frt_rope *rope, const frt_mask *mask,
                                    const void *q, const void *k_new,
                                    const void *v_new, int32_t n_new,
                                    int32_t num_q_heads, float softmax_scale,
                                    void *workspace, size_t workspace_bytes,
                                    void *out, float *lse, void *hip_stream);

/*
 * A whole FP8 streaming step: exactly frt_stream_attn_step_fp8 followed by
 * frt_kv_append_fp8(k_new, v_new, n_new) on the same stream (same outputs,
 * same ring codes and seq_len afterwards). The append copies the key and
 * value codes the step has already computed from the workspace into the
 * ring's slots and advances seq_len in the same launch, after the attention
 * launch has finished reading the ring. Arguments, workspace and errors as
 * for frt_stream_attn_step_fp8; n_new <= capacity.
 */
frt_status frt_stream_step_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                               const frt_rope *rope, const frt_mask *mask,
                               const void *q, const void *k_new,
                               const void *v_new, int32_t n_new,
                               int32_t num_q_heads, float softmax_scale,
                               void *workspace, size_t workspace_bytes,
                               void *out, float *lse, void *hip_stream);

/* Workspace bytes frt_decode_attn_fp8 and frt_decode_step_fp8 need: one
 * partial per KV piece and one per (stream, KV head) for the step's own
 * token, which also carries the token's key and value codes. */
size_t frt_decode_fp8_workspace_bytes(const frt_ring *ring, int32_t num_q_heads);

/*
 * frt_decode_attn over an FP8 ring (head_dim 128): one token per stream,
 * the same arithmetic as frt_stream_attn_step_fp8 with n_new = 1 (query
 * codes with a power-of-two scale per query, FP8 contractions with fp32
 * accumulation, coded weights p = code(2^(s - m + 7))). The ring is cut
 * into KV pieces as in frt_decode_attn; each piece codes its weights against
 * its own integer reference max, and the pieces' partials are merged with
 * power-of-two rescaling. The step's own key and value are coded as
 * frt_kv_append_fp8 stores them. Tensors, checks and errors as
 * frt_decode_attn, plus FRT_ERR_UNSUPPORTED for head_dim != 128.
 */
frt_status frt_decode_attn_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                               const frt_rope *rope, const frt_mask *mask,
                               const void *q, const void *k_new, const void *v_new,
                               int32_t num_q_heads, float softmax_scale,
                               void *workspace, size_t workspace_bytes,
                               void *out, float *lse, void *hip_stream);

/*
 * A whole FP8 decode step: exactly frt_decode_attn_fp8 followed by
 * frt_kv_append_fp8(k_new, v_new, 1) on the same stream (same outputs, same
 * ring codes and seq_len afterwards). The combine pass stores the token's
 * key and value codes, which the split pass computed, and advances seq_len.
 */
frt_status frt_decode_step_fp8(const frt_ring *ring, const frt_fp8_scales *scales,
                               const frt_rope *rope, const frt_mask *mask,
                               const void *q, const void *k_new, const void *v_new,
                               int32_t num_q_heads, float softmax_scale,
                               void *workspace, size_t workspace_bytes,
                               void *out, float *lse, void *hip_stream);

/* Static description of a status code. */
const char *frt_status_str(frt_status status);

/* Detail of the last failure on the calling thread ("" if none). */
const char *frt_last_error(void);

/*
 * Built-in kernel timing. When enabled, every kernel the library launches
 * records its own start and end in a pair of HIP events on its stream.
 * frt_timing_query waits for the recorded events of `kernel` (a launch name:
 * "rope_append", "seq_advance", "chunk_prep", "chunk_attn", "chunk_append",
 * "decode_split", "decode_combine"; the FP8 calls use the names of their
 * bf16 counterparts) and returns their count and summed milliseconds. frt_timing_samples writes the duration of each of
 * them, in launch order, to ms_out (at most `capacity` values) and the number
 * recorded to *count. frt_timing_reset drops all records.
 */
frt_status frt_timing_enable(int32_t on);
frt_status frt_timing_query(const char *kernel, int32_t *count, double *total_ms);
frt_status frt_timing_samples(const char *kernel, float *ms_out, int32_t capacity,
                              int32_t *count);
void frt_timing_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* FRT_H_ */
