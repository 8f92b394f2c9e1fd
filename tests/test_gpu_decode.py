"""frt_decode_attn (split-KV + combine) and frt_decode_step on the GPU against the fp64
oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_18171_amd as frt
from workloads import (WORKLOADS, RopeSpec, MaskSpec, ROPE_1D, MASK_CAUSAL, MASK_BLOCK_CAUSAL,
                       make_case, shrink, draw_bf16)
from gpu_helpers import (to_dev, bf16_dev_to_f64, build_rings, gpu_mask, visible_vmax,
                         check_close, ring_bytes_equal)

pytestmark = pytest.mark.gpu


def run_decode(case, ring, rope):
    wl = case.wl
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.Hq, 1), dtype=torch.float32, device="cuda")
    ws = torch.empty(frt.decode_workspace_bytes(ring, wl.Hq), dtype=torch.uint8, device="cuda")
    frt.decode_attn(ring, rope, gpu_mask(wl), q, k, v, out, ws, lse=lse)
    torch.cuda.synchronize()
    return out, lse


CASES = {
    "decode": (WORKLOADS["decode"], None),
    "split_edges": (shrink(WORKLOADS["decode"], B=6, C=1024), [0, 1, 255, 256, 257, 1023]),
    "wrapped_window": (shrink(WORKLOADS["decode"], B=3, Hq=8, Hkv=1, C=512,
                              mask=MaskSpec(MASK_CAUSAL, 0, 300)), [1000, 299, 512]),
    "g16_d64": (shrink(WORKLOADS["decode"], B=2, Hq=32, Hkv=2, d=64, C=328,
                       rope=RopeSpec(ROPE_1D, (64, 0, 0))), [327, 40]),
    "mha": (shrink(WORKLOADS["decode"], B=2, Hq=4, Hkv=4, C=264), [100, 263]),
    "block_causal": (shrink(WORKLOADS["decode"], B=2, Hq=8, Hkv=2, C=512,
                            mask=MaskSpec(MASK_BLOCK_CAUSAL, 128, 2)), [300, 511]),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_decode_matches_oracle(name):
    wl, lengths = CASES[name]
    case = make_case(wl, 0, lengths=None if lengths is None else np.array(lengths))
    ring, oring, rope = build_rings(case)
    out, lse = run_decode(case, ring, rope)
    ref, ref_lse = oracle.decode_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
    check_close(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), name)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2


def test_decode_equals_stream_step_with_one_token():
    wl, lengths = CASES["split_edges"]
    case = make_case(wl, 2, lengths=np.array(lengths))
    ring, oring, rope = build_rings(case)
    a, _ = run_decode(case, ring, rope)
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    b = torch.empty_like(q)
    ws = torch.empty(frt.stream_attn_workspace_bytes(ring, 1, wl.Hq), dtype=torch.uint8,
                     device="cuda")
    frt.stream_attn_step(ring, rope, gpu_mask(wl), q, k, v, b, ws)
    torch.cuda.synchronize()
    check_close(bf16_dev_to_f64(a), bf16_dev_to_f64(b), visible_vmax(oring, case), "decode vs step")


@pytest.mark.parametrize("name", ["split_edges", "mha", "g16_d64", "wrapped_window"])
def test_decode_step_equals_attn_then_append(name):
    """frt_decode_step over consecutive steps: the same outputs and lse as
    frt_decode_attn + frt_kv_append, bit for bit, and the same ring bytes and
    lengths, which also match the oracle's ring exactly."""
    wl, lengths = CASES[name]
    case = make_case(wl, 3, lengths=np.array(lengths))
    steps = 4
    ring, oring, rope = build_rings(case, extra_tokens=steps + 1)
    twin = frt.Ring(wl.B, wl.Hkv, wl.d, wl.C, k=ring.k.clone(), v=ring.v.clone(),
                    seq_len=ring.seq_len.clone())
    ws = torch.empty(frt.decode_workspace_bytes(ring, wl.Hq), dtype=torch.uint8, device="cuda")
    ws2 = torch.empty_like(ws)
    rng = np.random.default_rng(11)
    for s in range(steps):
        kn = draw_bf16(rng, case.k_new.shape)  # a fresh token each step
        vn = draw_bf16(rng, case.v_new.shape)
        q, k, v = to_dev(case.q), to_dev(kn), to_dev(vn)
        out_a, out_b = torch.empty_like(q), torch.empty_like(q)
        lse_a = torch.empty((wl.B, wl.Hq, 1), dtype=torch.float32, device="cuda")
        lse_b = torch.empty_like(lse_a)
        frt.decode_attn(twin, rope, gpu_mask(wl), q, k, v, out_a, ws2, lse=lse_a)
        frt.kv_append(twin, rope, k, v)
        frt.decode_step(ring, rope, gpu_mask(wl), q, k, v, out_b, ws, lse=lse_b)
        torch.cuda.synchronize()
        assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16)), (name, s)
        assert torch.equal(lse_a, lse_b), (name, s)
        assert torch.equal(ring.k.view(torch.int16), twin.k.view(torch.int16)), (name, s)
        assert torch.equal(ring.v.view(torch.int16), twin.v.view(torch.int16)), (name, s)
        assert torch.equal(ring.seq_len, twin.seq_len), (name, s)
        oring = oracle.kv_append(oring, kn, vn, wl.rope)
    assert ring_bytes_equal(ring, oring)


def test_decode_v_all_ones_gives_ones():
    """V = 1 everywhere: the output is a convex combination of ones, so 1 within one bf16
    step (the sum uses the same rounded weights as the P.V product)."""
    wl, lengths = CASES["split_edges"]
    case = make_case(wl, 7, lengths=np.array(lengths))
    case.v_new[:] = 0x3F80
    for _, v in case.prior_fills:
        v[:] = 0x3F80
    ring, oring, rope = build_rings(case)
    out, _ = run_decode(case, ring, rope)
    assert np.abs(bf16_dev_to_f64(out) - 1.0).max() <= 4e-3


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("Hq,Hkv", [(3, 3), (4, 2), (6, 2), (8, 2), (10, 2), (16, 2), (32, 2)])
def test_decode_group_sizes(Hq, Hkv, d):
    """Every query-group size G = Hq/Hkv from 1 to 16 (the combining wave splits its
    lanes over the G x d outputs by G), at both head dims."""
    wl = shrink(WORKLOADS["decode"], B=3, Hq=Hq, Hkv=Hkv, d=d, C=704,
                rope=RopeSpec(ROPE_1D, (d, 0, 0)))
    case = make_case(wl, Hq + d, lengths=np.array([703, 0, 333]))
    ring, oring, rope = build_rings(case)
    out, lse = run_decode(case, ring, rope)
    ref, ref_lse = oracle.decode_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
    check_close(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), "G%d d%d" % (Hq // Hkv, d))
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2


def _pieces_per_head(wl, lengths):
    """Pieces the decode pass cuts each (stream, KV head) of these lengths into: the
    visible ring tokens as 32-token tiles (causal, no window: tokens 0 .. L-1), `per`
    tiles a piece with per = clamp(ceil(T / slots), 4, 12), T the tiles of every head
    and slots the 2048 resident waves less one per head."""
    tiles = [(L + 31) // 32 for L in lengths]
    heads = len(lengths) * wl.Hkv
    T = sum(tiles) * wl.Hkv
    slots = max(2048 - heads, 1024)
    per = min(max(-(-T // slots), 4), 12)
    return [-(-t // per) for t in tiles]


def test_decode_split_count_independence():
    """The same stream decoded alone and inside batches whose total work cuts its
    ring into different numbers of pieces: each result within tolerance of the
    oracle (the split is an exact rewrite of the definition)."""
    L0 = 6000
    base = shrink(WORKLOADS["decode"], B=1, C=8448)
    one = make_case(base, 21, lengths=np.array([L0]))
    splits = set()
    for B in (1, 12, 24):
        wl = shrink(WORKLOADS["decode"], B=B, C=8448)
        lengths = np.array([L0] + [8000] * (B - 1))
        case = make_case(wl, 22 + B, lengths=lengths)
        # stream 0 carries exactly the single-stream case's data
        case.prior_fills[0] = one.prior_fills[0]
        case.q[0] = one.q[0]
        case.k_new[0] = one.k_new[0]
        case.v_new[0] = one.v_new[0]
        splits.add(_pieces_per_head(wl, lengths)[0])
        ring, oring, rope = build_rings(case)
        out, lse = run_decode(case, ring, rope)
        ref, ref_lse = oracle.decode_attn(oring, case.q[:1], case.k_new[:1], case.v_new[:1],
                                          wl.rope, wl.mask)
        got = bf16_dev_to_f64(out)[:1]
        check_close(got, ref, visible_vmax(oring, case), "B%d" % B)
        assert np.abs(lse.cpu().numpy()[:1] - ref_lse).max() < 2e-2
    assert len(splits) == 3, splits


@pytest.mark.parametrize("B", [65, 130])
def test_decode_more_than_64_streams(B):
    """The decode pass finds each wave's stream and piece range with wave-wide
    scans over groups of 64 streams: batches past one and two groups, with
    lengths from empty to a full ring, against the oracle; then the fused step's
    ring and lengths against the oracle's."""
    wl = shrink(WORKLOADS["decode"], B=B, Hq=4, Hkv=2, C=256,
                mask=MaskSpec(MASK_CAUSAL, 0, 0))
    rng = np.random.default_rng(B)
    lengths = rng.integers(0, 256, B)
    lengths[0], lengths[-1], lengths[B // 2] = 0, 255, 1
    case = make_case(wl, B, lengths=lengths)
    ring, oring, rope = build_rings(case, extra_tokens=2)
    out, lse = run_decode(case, ring, rope)
    ref, ref_lse = oracle.decode_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
    check_close(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), "B%d" % B)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2
    ws = torch.empty(frt.decode_workspace_bytes(ring, wl.Hq), dtype=torch.uint8, device="cuda")
    step_out = torch.empty_like(out)
    frt.decode_step(ring, rope, gpu_mask(wl), to_dev(case.q), to_dev(case.k_new),
                    to_dev(case.v_new), step_out, ws)
    torch.cuda.synchronize()
    assert torch.equal(step_out.view(torch.int16), out.view(torch.int16))
    oring = oracle.kv_append(oring, case.k_new, case.v_new, wl.rope)
    assert ring_bytes_equal(ring, oring)
