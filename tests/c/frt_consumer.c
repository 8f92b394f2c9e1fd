/* A plain C99 consumer of the C ABI: it compiles against include/frt.h alone,
 * links libfrt.so, and exercises the host-side calls that need no GPU: status
 * strings, workspace and table sizes, the rotary table, and argument
 * validation (every rejected call returns before touching the device). */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <stdint.h>

#include "frt.h"

static int fails = 0;
#define CHECK(cond)                                                            \
  do {                                                                         \
    if (!(cond)) {                                                             \
      printf("FAIL %s:%d %s (last error: %s)\n", __FILE__, __LINE__, #cond,    \
             frt_last_error());                                                \
      ++fails;                                                                 \
    }                                                                          \
  } while (0)

int main(void) {
  int s;
  for (s = FRT_OK; s <= FRT_ERR_HIP; ++s) {
    const char *str = frt_status_str((frt_status)s);
    CHECK(str != NULL && strlen(str) > 0);
  }

  /* a 1D rotary table for 64 positions of head_dim 128 */
  frt_rope rope;
  memset(&rope, 0, sizeof rope);
  rope.mode = FRT_ROPE_1D;
  rope.axis_dims[0] = 128;
  rope.max_pos[0] = 64;
  rope.base = 10000.0;
  size_t tb = frt_rope_table_bytes(&rope);
  CHECK(tb == (size_t)64 * 64 * 2 * sizeof(float));
  float *table = (float *)malloc(tb);
  CHECK(frt_rope_table_fill(&rope, table, tb) == FRT_OK);
  CHECK(table[0] == 1.0f && table[1] == 0.0f); /* position 0: cos 1, sin 0 */

  /* a ring description (no device memory behind it: only validated) */
  frt_ring ring;
  memset(&ring, 0, sizeof ring);
  ring.num_streams = 2;
  ring.num_kv_heads = 2;
  ring.head_dim = 128;
  ring.capacity = 256;
  CHECK(frt_stream_attn_workspace_bytes(&ring, 64, 8) > 0);
  CHECK(frt_decode_workspace_bytes(&ring, 8) > 0);

  frt_mask mask = {FRT_MASK_CAUSAL, 0, 0};
  void *fake = (void *)(uintptr_t)0x1000;
  rope.table = (const float *)fake;
  /* a NULL ring buffer is rejected on the host */
  CHECK(frt_kv_append(&ring, &rope, fake, fake, 8, NULL) == FRT_ERR_NULL);
  CHECK(strlen(frt_last_error()) > 0);
  ring.k_ring = fake;
  ring.v_ring = fake;
  ring.seq_len = (int64_t *)fake;
  /* 7 query heads over 2 KV heads */
  CHECK(frt_stream_attn_step(&ring, &rope, &mask, fake, fake, fake, 8, 7, 0.f, fake, 1 << 20,
                             fake, NULL, NULL) == FRT_ERR_SHAPE);
  /* head_dim 96 */
  ring.head_dim = 96;
  CHECK(frt_kv_append(&ring, &rope, fake, fake, 8, NULL) == FRT_ERR_UNSUPPORTED);
  ring.head_dim = 128;
  /* more new tokens than the ring holds */
  CHECK(frt_kv_append(&ring, &rope, fake, fake, 257, NULL) == FRT_ERR_CAPACITY);
  /* a workspace smaller than required */
  CHECK(frt_decode_attn(&ring, &rope, &mask, fake, fake, fake, 8, 0.f, fake, 16, fake, NULL,
                        NULL) == FRT_ERR_WORKSPACE);

  free(table);
  printf("%s: %d failure(s)\n", fails ? "FAIL" : "ok", fails);
  return fails ? 1 : 0;
}
