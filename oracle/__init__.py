"""fp64 CPU oracle for chunk-streamed attention over a ring-buffer KV cache.

TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import this package. The product path (the
HIP library and its Python binding) never imports, calls or links it, and this
package never imports the product path: the two share no code. The only thing
both sides consume is the seeded input arrays drawn by `workloads`.

What is computed, and where it comes from
-----------------------------------------
The paper (FlashRT) defines the *state semantics* of a streaming step: batch j
of a node reads persistent state written by batch j-1 of the same node and
writes it for batch j+1 (Problem Formulation: cross-batch lambda=1 edges, with
a key/value cache carried between batches as the example; Chain-of-Program, IR design:
node-level persistent-state read/write annotations; App. "Formal Analysis of Pipeline Graphs";
App. "Application 2": independent per-denoising-step KV caches). It gives no
arithmetic for the attention itself. The arithmetic here is therefore the
plain textbook definition:

  * scaled dot-product attention softmax(q k^T * scale) V with max
    subtraction (Vaswani et al. 2017), evaluated in float64, no tiling, no
    online softmax, no split-KV;
  * rotary position embedding: rotate interleaved coordinate pairs
    (x[2i], x[2i+1]) by angle pos * theta_i, theta_i = base^(-2i/D)
    (Su et al., RoFormer 2021); a 3D variant applies it per axis (t, h, w)
    on disjoint slices of the head dimension;
  * a ring buffer of C slots per stream and KV head where token t lives in
    slot t mod C.

Readings chosen where the paper is silent:
interleaved pairs; per-axis theta with its own D_a; fp32 cos/sin tables from
float64 libm; stored K = bf16(fp32(rot_fp64(k))) with round-to-nearest-even at
both steps; attention reads the pre-step ring plus the chunk's own K/V (the
append happens after); scale 1/sqrt(d); GQA query head h uses KV head
h // (Hq/Hkv).

Modules: rope (tables, rotation, rounding), ring (append, slot map),
attention (masked attention, decode), brute (pure-Python loop twins), fp8
(the e4m3fn codec and the FP8 KV-cache / FP8 QK^T-PV variant of the step).
"""
from .rope import (rope_cos_sin, rope_positions, rotate_f64, round_f64_to_bf16,
                   bf16_to_f64, stored_k)
from .ring import RingState, new_ring, kv_append, slot_token, slots_of_tokens
from .attention import visible, stream_attn, decode_attn, attention_inputs

__all__ = [
    "rope_cos_sin", "rope_positions", "rotate_f64", "round_f64_to_bf16",
    "bf16_to_f64", "stored_k", "RingState", "new_ring", "kv_append",
    "slot_token", "slots_of_tokens", "visible", "stream_attn", "decode_attn",
    "attention_inputs",
]
