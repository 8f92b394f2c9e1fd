"""MI355X-native chunk-streamed attention over ring-buffer KV caches.

The compute lives in libfrt.so (HIP kernels for gfx950, C ABI in
include/frt.h); this package is its thin Python binding plus the in-tree
build script. Importing the package does not load the library; the first
call does, and raises ImportError if libfrt.so has not been built.
"""
from .binding import (FrtError, Ring, Rope, mask, kv_append, stream_attn_step,
                      stream_attn_workspace_bytes, stream_step, decode_attn,
                      RingFp8, kv_append_fp8, stream_attn_fp8_workspace_bytes,
                      stream_attn_step_fp8, stream_step_fp8, decode_fp8_workspace_bytes,
                      decode_attn_fp8, decode_step_fp8, decode_step, decode_step_noalloc,
                      decode_workspace_bytes,
                      decode_max_splits, timing_enable, timing_query, timing_samples, timing_reset,
                      load_library, ROPE_NONE, ROPE_1D, ROPE_3D, MASK_BLOCK_CAUSAL,
                      MASK_CAUSAL, EXPORTS, LIB_PATH)

__all__ = [
    "FrtError", "Ring", "Rope", "mask", "kv_append", "stream_attn_step",
    "stream_attn_workspace_bytes", "stream_step", "decode_attn", "RingFp8",
    "kv_append_fp8", "stream_attn_fp8_workspace_bytes", "stream_attn_step_fp8", "stream_step_fp8",
    "decode_fp8_workspace_bytes", "decode_attn_fp8", "decode_step_fp8",
    "decode_step", "decode_step_noalloc",
    "decode_workspace_bytes", "decode_max_splits",
    "timing_enable", "timing_query", "timing_samples", "timing_reset", "load_library", "ROPE_NONE", "ROPE_1D",
    "ROPE_3D", "MASK_BLOCK_CAUSAL", "MASK_CAUSAL", "EXPORTS", "LIB_PATH",
]
