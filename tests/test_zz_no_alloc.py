"""frt_decode_step_noalloc (the decode step on the library's fixed device
scratch, no workspace) against frt_decode_step with a workspace: identical
outputs, LSE, ring bytes and lengths, on two calls in a row, the second
smaller than the first."""
import numpy as np
import pytest
import torch

import paper_2607_18171_amd as frt
from workloads import WORKLOADS, RopeSpec, ROPE_1D, make_case, shrink
from gpu_helpers import to_dev, build_rings, gpu_mask

pytestmark = pytest.mark.gpu


def _twin(ring, wl):
    return frt.Ring(wl.B, wl.Hkv, wl.d, wl.C, k=ring.k.clone(), v=ring.v.clone(),
                    seq_len=ring.seq_len.clone())


@pytest.mark.parametrize("steps", [2])
def test_noalloc_decode_equals_workspace_decode(steps):
    big = WORKLOADS["decode"]
    small = shrink(WORKLOADS["decode"], B=5, Hq=8, Hkv=2, d=64, C=1024,
                   rope=RopeSpec(ROPE_1D, (64, 0, 0)))
    for wl, lengths, seed in ((big, None, 0), (small, [1023, 0, 1, 700, 64], 1)):
        assert frt.decode_workspace_bytes(frt.Ring(wl.B, wl.Hkv, wl.d, wl.C), wl.Hq) <= 32 << 20
        case = make_case(wl, seed, lengths=None if lengths is None else np.array(lengths))
        ring, _, rope = build_rings(case, extra_tokens=steps + 1)
        twin = _twin(ring, wl)
        ws = torch.empty(frt.decode_workspace_bytes(ring, wl.Hq), dtype=torch.uint8, device="cuda")
        q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
        for s in range(steps):
            out_a, out_b = torch.empty_like(q), torch.empty_like(q)
            lse_a = torch.empty((wl.B, wl.Hq, 1), dtype=torch.float32, device="cuda")
            lse_b = torch.empty_like(lse_a)
            frt.decode_step(twin, rope, gpu_mask(wl), q, k, v, out_a, ws, lse=lse_a)
            frt.decode_step_noalloc(ring, rope, gpu_mask(wl), q, k, v, out_b, lse=lse_b)
            torch.cuda.synchronize()
            what = "B%d step %d" % (wl.B, s)
            assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16)), what
            assert torch.equal(lse_a, lse_b), what
            assert torch.equal(ring.k.view(torch.int16), twin.k.view(torch.int16)), what
            assert torch.equal(ring.v.view(torch.int16), twin.v.view(torch.int16)), what
            assert torch.equal(ring.seq_len, twin.seq_len), what


def test_noalloc_rejects_rings_past_its_scratch():
    # 64 streams x 8 KV heads x 16 query heads per KV head at head_dim 128:
    # far more partials than the fixed scratch holds
    ring = frt.Ring(64, 8, 128, 8448)
    assert frt.decode_workspace_bytes(ring, 128) > 32 << 20
    rope = frt.Rope.for_tokens(ROPE_1D, (128, 0, 0), (0, 0), 16)
    q = torch.zeros((64, 1, 128, 128), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((64, 1, 8, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    with pytest.raises(frt.FrtError) as e:
        frt.decode_step_noalloc(ring, rope, frt.mask(2, 0, 0), q, kv, kv, out)
    assert e.value.status == 6
    assert torch.equal(ring.seq_len, torch.zeros_like(ring.seq_len))
