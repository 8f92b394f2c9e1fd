"""The steps (bf16 and FP8) under HIP graph capture: a serving loop captures one step and
replays it with new inputs copied into the captured buffers. Every replay must
equal the same step run eagerly, bit for bit (outputs, LSE, ring bytes and
lengths). The graphs hold only the library's kernels (no allocation, no
memset, no host synchronisation inside a step); each replay is followed by
eager work and a synchronisation before it is checked."""
import numpy as np
import pytest
import torch

import paper_2607_18171_amd as frt
from workloads import (WORKLOADS, RopeSpec, MaskSpec, ROPE_1D, MASK_BLOCK_CAUSAL, make_case,
                       shrink, draw_bf16)
from gpu_helpers import to_dev, build_rings, gpu_mask, gpu_rope as gpu_rope_for

pytestmark = pytest.mark.gpu

REPLAYS = 4


def _twin(ring, wl):
    return frt.Ring(wl.B, wl.Hkv, wl.d, wl.C, k=ring.k.clone(), v=ring.v.clone(),
                    seq_len=ring.seq_len.clone())


def _same_bits(a, b):
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


def _check(ring, twin, out_g, out_e, lse_g, lse_e, what):
    assert _same_bits(out_g, out_e), what
    assert torch.equal(lse_g, lse_e), what
    assert _same_bits(ring.k, twin.k), what
    assert _same_bits(ring.v, twin.v), what
    assert torch.equal(ring.seq_len, twin.seq_len), what


def _capture(fn):
    """Warm up on a side stream (first-call set-up stays out of the graph), then
    capture one call."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("noalloc", [False, True])
def test_decode_step_graph_replays(noalloc):
    wl = shrink(WORKLOADS["decode"], B=5, Hq=8, Hkv=2, C=1024)
    case = make_case(wl, 21, lengths=np.array([1023, 0, 1, 700, 64]))
    ring, _, rope = build_rings(case, extra_tokens=REPLAYS + 2)
    twin = _twin(ring, wl)
    m = gpu_mask(wl)
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.Hq, 1), dtype=torch.float32, device="cuda")
    ws = torch.empty(frt.decode_workspace_bytes(ring, wl.Hq), dtype=torch.uint8, device="cuda")
    ws_e = torch.empty_like(ws)

    def step():
        if noalloc:
            frt.decode_step_noalloc(ring, rope, m, q, k, v, out, lse=lse)
        else:
            frt.decode_step(ring, rope, m, q, k, v, out, ws, lse=lse)

    if noalloc:  # the scratch address is looked up once per device, before capture
        probe = _twin(ring, wl)
        frt.decode_step_noalloc(probe, rope, m, q, k, v, torch.empty_like(q),
                                lse=torch.empty_like(lse))
        torch.cuda.synchronize()
        del probe
    g = _capture(step)  # captured, not run: the ring is unchanged
    assert torch.equal(ring.seq_len, twin.seq_len)
    rng = np.random.default_rng(5)
    for r in range(REPLAYS):
        qb, kb, vb = (draw_bf16(rng, case.q.shape), draw_bf16(rng, case.k_new.shape),
                      draw_bf16(rng, case.v_new.shape))
        q.copy_(to_dev(qb))
        k.copy_(to_dev(kb))
        v.copy_(to_dev(vb))
        g.replay()
        out_e = torch.empty_like(q)
        lse_e = torch.empty_like(lse)
        frt.decode_step(twin, rope, m, to_dev(qb), to_dev(kb), to_dev(vb), out_e, ws_e,
                        lse=lse_e)
        torch.cuda.synchronize()
        _check(ring, twin, out, out_e, lse, lse_e, "decode replay %d" % r)


def test_stream_step_graph_replays():
    wl = shrink(WORKLOADS["tiny"], B=2, Hq=4, Hkv=2, d=128, n=48, C=192,
                rope=RopeSpec(ROPE_1D, (128, 0, 0)), mask=MaskSpec(MASK_BLOCK_CAUSAL, 48, 3),
                prior_steps=5)
    case = make_case(wl, 22)
    ring, _, rope = build_rings(case, extra_tokens=(REPLAYS + 2) * wl.n)
    twin = _twin(ring, wl)
    m = gpu_mask(wl)
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.Hq, wl.n), dtype=torch.float32, device="cuda")
    ws = torch.empty(frt.stream_attn_workspace_bytes(ring, wl.n, wl.Hq), dtype=torch.uint8,
                     device="cuda")
    ws_e = torch.empty_like(ws)
    g = _capture(lambda: frt.stream_step(ring, rope, m, q, k, v, out, ws, lse=lse))
    assert torch.equal(ring.seq_len, twin.seq_len)
    rng = np.random.default_rng(6)
    for r in range(REPLAYS):
        qb, kb, vb = (draw_bf16(rng, case.q.shape), draw_bf16(rng, case.k_new.shape),
                      draw_bf16(rng, case.v_new.shape))
        q.copy_(to_dev(qb))
        k.copy_(to_dev(kb))
        v.copy_(to_dev(vb))
        g.replay()
        out_e = torch.empty_like(q)
        lse_e = torch.empty_like(lse)
        frt.stream_step(twin, rope, m, to_dev(qb), to_dev(kb), to_dev(vb), out_e, ws_e, lse=lse_e)
        torch.cuda.synchronize()
        _check(ring, twin, out, out_e, lse, lse_e, "stream replay %d" % r)


def _fp8_pair(wl, lengths, seed):
    """An FP8 ring filled with `lengths` tokens per stream, and an identical twin."""
    ks = np.full((wl.B, wl.Hkv), 0.02, np.float32)
    vs = np.full((wl.B, wl.Hkv), 0.02, np.float32)
    rope = gpu_rope_for(wl, max(lengths) + 8 * wl.n + 1)
    ring = frt.RingFp8(wl.B, wl.Hkv, wl.d, wl.C, torch.from_numpy(ks), torch.from_numpy(vs))
    rng = np.random.default_rng(seed)
    for b, L in enumerate(lengths):
        for s in range(0, L, wl.C):
            e = min(L, s + wl.C)
            k = draw_bf16(rng, (1, e - s, wl.Hkv, wl.d))
            v = draw_bf16(rng, (1, e - s, wl.Hkv, wl.d))
            frt.kv_append_fp8(ring.view_stream(b), rope, to_dev(k), to_dev(v))
    twin = frt.RingFp8(wl.B, wl.Hkv, wl.d, wl.C, torch.from_numpy(ks), torch.from_numpy(vs))
    twin.k.copy_(ring.k)
    twin.v.copy_(ring.v)
    twin.seq_len.copy_(ring.seq_len)
    torch.cuda.synchronize()
    return ring, twin, rope


def _same_fp8_rings(ring, twin):
    return (torch.equal(ring.k, twin.k) and torch.equal(ring.v, twin.v)
            and torch.equal(ring.seq_len, twin.seq_len))


@pytest.mark.parametrize("decode", [True, False])
def test_fp8_step_graph_replays(decode):
    """frt_decode_step_fp8 / frt_stream_step_fp8 captured once and replayed with new
    inputs: every replay equals the eager step bit for bit (outputs, ring codes,
    lengths)."""
    if decode:
        wl = shrink(WORKLOADS["decode"], B=5, Hq=8, Hkv=2, C=1024)
        lengths = [1023, 0, 1, 700, 64]
    else:
        wl = shrink(WORKLOADS["tiny"], B=2, Hq=4, Hkv=2, d=128, n=48, C=192,
                    rope=RopeSpec(ROPE_1D, (128, 0, 0)),
                    mask=MaskSpec(MASK_BLOCK_CAUSAL, 48, 3))
        lengths = [240, 96]
    ring, twin, rope = _fp8_pair(wl, lengths, 23)
    m = gpu_mask(wl)
    shape_q = (wl.B, wl.n, wl.Hq, wl.d)
    shape_kv = (wl.B, wl.n, wl.Hkv, wl.d)
    q = torch.zeros(shape_q, dtype=torch.bfloat16, device="cuda")
    k = torch.zeros(shape_kv, dtype=torch.bfloat16, device="cuda")
    v = torch.zeros(shape_kv, dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    if decode:
        ws = torch.empty(frt.decode_fp8_workspace_bytes(ring, wl.Hq), dtype=torch.uint8,
                         device="cuda")
        step = frt.decode_step_fp8
    else:
        ws = torch.empty(frt.stream_attn_fp8_workspace_bytes(ring, wl.n, wl.Hq),
                         dtype=torch.uint8, device="cuda")
        step = frt.stream_step_fp8
    ws_e = torch.empty_like(ws)
    g = _capture(lambda: step(ring, rope, m, q, k, v, out, ws))
    assert _same_fp8_rings(ring, twin)
    rng = np.random.default_rng(7)
    for r in range(REPLAYS):
        qb, kb, vb = draw_bf16(rng, shape_q), draw_bf16(rng, shape_kv), draw_bf16(rng, shape_kv)
        q.copy_(to_dev(qb))
        k.copy_(to_dev(kb))
        v.copy_(to_dev(vb))
        g.replay()
        out_e = torch.empty_like(q)
        step(twin, rope, m, to_dev(qb), to_dev(kb), to_dev(vb), out_e, ws_e)
        torch.cuda.synchronize()
        assert _same_bits(out, out_e), ("fp8", decode, r)
        assert _same_fp8_rings(ring, twin), ("fp8", decode, r)
