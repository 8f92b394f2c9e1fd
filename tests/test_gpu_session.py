"""Long streaming sessions: the state a step leaves (ring bytes and lengths) is
the state the next step reads. Many consecutive fused steps run on the GPU
from an empty ring, each with a fresh query chunk and fresh keys and values,
the ring wrapping several times; after every step the output is checked
against the oracle's attention on the oracle's own ring, which the oracle then
advances with the same chunk, and at the end the two rings must be equal bit
for bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_18171_amd as frt
from workloads import (WORKLOADS, RopeSpec, MaskSpec, ROPE_1D, ROPE_3D, MASK_BLOCK_CAUSAL,
                       MASK_CAUSAL, shrink, draw_bf16)
from gpu_helpers import (to_dev, bf16_dev_to_f64, gpu_rope, gpu_mask, check_close,
                         ring_bytes_equal)

pytestmark = pytest.mark.gpu

SESSIONS = {
    # 3D rope, block-causal over 4 chunks of 72 tokens, a 4-chunk ring:
    # 14 steps wrap it three times
    "video": (shrink(WORKLOADS["video_1p3b"], Hq=2, Hkv=2, n=72, C=288,
                     rope=RopeSpec(ROPE_3D, (44, 42, 42), (4, 6)),
                     mask=MaskSpec(MASK_BLOCK_CAUSAL, 72, 4), prior_steps=0), 14),
    # GQA, a causal window of 200 over 100-token chunks, a ring of 256 that
    # is not a multiple of the chunk: the chunks straddle its end
    "swa": (shrink(WORKLOADS["prefill_swa"], B=2, Hq=8, Hkv=2, n=100, C=256,
                   mask=MaskSpec(MASK_CAUSAL, 0, 200)), 10),
}


def _vmax(oring, v_new):
    return float(np.abs(np.concatenate([oracle.bf16_to_f64(oring.v).ravel(),
                                        oracle.bf16_to_f64(v_new).ravel()])).max())


@pytest.mark.parametrize("name", sorted(SESSIONS))
def test_chunk_session_matches_oracle_every_step(name):
    wl, steps = SESSIONS[name]
    rope = gpu_rope(wl, steps * wl.n + 1)
    ring = frt.Ring(wl.B, wl.Hkv, wl.d, wl.C)
    oring = oracle.new_ring(wl.B, wl.Hkv, wl.C, wl.d)
    ws = torch.empty(frt.stream_attn_workspace_bytes(ring, wl.n, wl.Hq), dtype=torch.uint8,
                     device="cuda")
    rng = np.random.default_rng(40)
    for s in range(steps):
        q = draw_bf16(rng, (wl.B, wl.n, wl.Hq, wl.d), wl.qk_scale)
        k = draw_bf16(rng, (wl.B, wl.n, wl.Hkv, wl.d), wl.qk_scale)
        v = draw_bf16(rng, (wl.B, wl.n, wl.Hkv, wl.d))
        out = torch.empty((wl.B, wl.n, wl.Hq, wl.d), dtype=torch.bfloat16, device="cuda")
        frt.stream_step(ring, rope, gpu_mask(wl), to_dev(q), to_dev(k), to_dev(v), out, ws)
        torch.cuda.synchronize()
        ref, _ = oracle.stream_attn(oring, q, k, v, wl.rope, wl.mask)
        check_close(bf16_dev_to_f64(out), ref, _vmax(oring, v), "%s step %d" % (name, s))
        oring = oracle.kv_append(oring, k, v, wl.rope)
        assert np.array_equal(ring.seq_len.cpu().numpy(), oring.seq_len), (name, s)
    assert ring_bytes_equal(ring, oring)


def test_decode_session_matches_oracle_every_step():
    """Consecutive frt_decode_step calls on streams that start at different
    lengths, two of them passing the ring's capacity during the session (a
    300-token window, so the evicted tokens are out of every query's reach)."""
    wl = shrink(WORKLOADS["decode"], B=4, Hq=8, Hkv=2, C=320,
                rope=RopeSpec(ROPE_1D, (128, 0, 0)), mask=MaskSpec(MASK_CAUSAL, 0, 300))
    steps = 24
    start = [300, 0, 40, 310]
    rng = np.random.default_rng(41)
    rope = gpu_rope(wl, max(start) + steps + 1)
    ring = frt.Ring(wl.B, wl.Hkv, wl.d, wl.C)
    oring = oracle.new_ring(wl.B, wl.Hkv, wl.C, wl.d)
    for b, L in enumerate(start):
        if L:
            k = draw_bf16(rng, (1, L, wl.Hkv, wl.d))
            v = draw_bf16(rng, (1, L, wl.Hkv, wl.d))
            frt.kv_append(ring.view_stream(b), rope, to_dev(k), to_dev(v))
            oring = oracle.kv_append(oring, k, v, wl.rope, streams=[b])
    ws = torch.empty(frt.decode_workspace_bytes(ring, wl.Hq), dtype=torch.uint8, device="cuda")
    for s in range(steps):
        q = draw_bf16(rng, (wl.B, 1, wl.Hq, wl.d))
        k = draw_bf16(rng, (wl.B, 1, wl.Hkv, wl.d))
        v = draw_bf16(rng, (wl.B, 1, wl.Hkv, wl.d))
        out = torch.empty((wl.B, 1, wl.Hq, wl.d), dtype=torch.bfloat16, device="cuda")
        frt.decode_step(ring, rope, gpu_mask(wl), to_dev(q), to_dev(k), to_dev(v), out, ws)
        torch.cuda.synchronize()
        ref, _ = oracle.decode_attn(oring, q, k, v, wl.rope, wl.mask)
        check_close(bf16_dev_to_f64(out), ref, _vmax(oring, v), "decode step %d" % s)
        oring = oracle.kv_append(oring, k, v, wl.rope)
    assert ring_bytes_equal(ring, oring)
