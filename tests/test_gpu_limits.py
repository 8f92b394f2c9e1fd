"""The largest ring the library admits, used at the top of its slot range.

A ring's per-head K (and V) storage must stay below 2^31 bytes; at head_dim
128 the largest admitted capacity is 8388600 slots (2147481600 bytes per head,
ending in a partial V block of 24 slots). Tokens are appended across the top
of such a ring, then a chunk step and a decode step run there. Under a causal
window of 100 keys only tokens of the last 100 positions are visible, and the
oracle's result depends on tokens and positions only, so a 128-slot oracle
ring fed the same tokens gives the expected values. Ring bytes are compared
bit for bit at every written slot; outputs to the attention tolerance.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_18171_amd as frt
from workloads import RopeSpec, MaskSpec, ROPE_3D, MASK_CAUSAL, draw_bf16
from gpu_helpers import to_dev, from_dev, bf16_dev_to_f64, check_close

pytestmark = pytest.mark.gpu

D = 128
C_MAX = (2 ** 31 - 1) // (D * 2) // 8 * 8
ROPE = RopeSpec(ROPE_3D, (44, 42, 42), (64, 64))  # positions near 2^23 stay small frame indices
MASK = MaskSpec(MASK_CAUSAL, 0, 100)
C_SMALL = 128


def written_slots_equal(ring, small, tokens):
    """The GPU ring's bytes for `tokens` equal the small oracle ring's."""
    slots = np.asarray(tokens, dtype=np.int64) % ring.C
    sslots = np.asarray(tokens, dtype=np.int64) % C_SMALL
    k = from_dev(ring.k[0, 0, torch.as_tensor(slots, device=ring.k.device)])
    v = from_dev(ring.v[0, 0, ring.v_index(slots).reshape(-1)]).reshape(len(slots), D)
    return np.array_equal(k, small.k[0, 0, sslots]) and np.array_equal(v, small.v[0, 0, sslots])


def test_max_capacity_ring_top():
    assert C_MAX == 8388600 and C_MAX * D * 2 < 2 ** 31 and C_MAX % 32 == 24
    B, Hq, Hkv = 1, 2, 1
    rng = np.random.default_rng(11)
    L0 = C_MAX - 40
    ring = frt.Ring(B, Hkv, D, C_MAX)
    ring.seq_len.fill_(L0)
    small = oracle.new_ring(B, Hkv, C_SMALL, D)
    small.seq_len[:] = L0
    rope = frt.Rope.for_tokens(ROPE.mode, ROPE.axis_dims, ROPE.frame_hw, C_MAX + 256, ROPE.base)
    msk = frt.mask(MASK.kind, MASK.block, MASK.window)

    # 64 tokens across the top: slots C-40 .. C-1 (the partial V block among
    # them), then 0 .. 23
    k1, v1 = draw_bf16(rng, (B, 64, Hkv, D)), draw_bf16(rng, (B, 64, Hkv, D))
    frt.kv_append(ring, rope, to_dev(k1), to_dev(v1))
    small = oracle.kv_append(small, k1, v1, ROPE)
    torch.cuda.synchronize()
    assert int(ring.seq_len[0]) == L0 + 64
    assert written_slots_equal(ring, small, np.arange(L0, L0 + 64))

    # a fused chunk step of 40 tokens at L = C + 24 (the window reaches back
    # to position C - 75: never-written zero slots, then the appended tokens)
    n = 40
    q, k2, v2 = (draw_bf16(rng, (B, n, Hq, D)), draw_bf16(rng, (B, n, Hkv, D)),
                 draw_bf16(rng, (B, n, Hkv, D)))
    qd = to_dev(q)
    out = torch.empty_like(qd)
    ws = torch.empty(frt.stream_attn_workspace_bytes(ring, n, Hq), dtype=torch.uint8,
                     device="cuda")
    frt.stream_step(ring, rope, msk, qd, to_dev(k2), to_dev(v2), out, ws)
    ref, _ = oracle.stream_attn(small, q, k2, v2, ROPE, MASK)
    small = oracle.kv_append(small, k2, v2, ROPE)
    torch.cuda.synchronize()
    vmax = float(max(np.abs(oracle.bf16_to_f64(v1)).max(), np.abs(oracle.bf16_to_f64(v2)).max()))
    check_close(bf16_dev_to_f64(out), ref, vmax, "chunk step at the top of the largest ring")
    assert int(ring.seq_len[0]) == L0 + 64 + n
    assert written_slots_equal(ring, small, np.arange(L0 + 64, L0 + 64 + n))

    # a decode step right after (window: positions C - 35 .. C + 64)
    q3, k3, v3 = (draw_bf16(rng, (B, 1, Hq, D)), draw_bf16(rng, (B, 1, Hkv, D)),
                  draw_bf16(rng, (B, 1, Hkv, D)))
    q3d = to_dev(q3)
    out3 = torch.empty_like(q3d)
    ws3 = torch.empty(frt.decode_workspace_bytes(ring, Hq), dtype=torch.uint8, device="cuda")
    frt.decode_step(ring, rope, msk, q3d, to_dev(k3), to_dev(v3), out3, ws3)
    ref3, _ = oracle.decode_attn(small, q3, k3, v3, ROPE, MASK)
    small = oracle.kv_append(small, k3, v3, ROPE)
    torch.cuda.synchronize()
    vmax3 = float(max(vmax, np.abs(oracle.bf16_to_f64(v3)).max()))
    check_close(bf16_dev_to_f64(out3), ref3, vmax3, "decode step at the top of the largest ring")
    L = L0 + 64 + n + 1
    assert int(ring.seq_len[0]) == L
    assert written_slots_equal(ring, small, [L - 1])

