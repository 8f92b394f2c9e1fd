"""frt_stream_attn_step on the GPU against the fp64 oracle.

Tolerance (bf16 inputs, fp32 accumulation): max|err| <= 1e-2 * max|V| and
mean|err| <= 1e-3, per case, over every output element computed.
"""
import functools

import numpy as np
import pytest
import torch

import oracle
import paper_2607_18171_amd as frt
from workloads import (WORKLOADS, RopeSpec, MaskSpec, ROPE_1D, ROPE_3D, ROPE_NONE,
                       MASK_BLOCK_CAUSAL, MASK_CAUSAL, make_case, shrink, draw_bf16)
from gpu_helpers import (to_dev, from_dev, bf16_dev_to_f64, build_rings, gpu_mask,
                         visible_vmax, check_close, ring_bytes_equal)

pytestmark = pytest.mark.gpu


def lse_tol(wl):
    """LSE tolerance (natural log): 2e-2 for unit-variance Q and K. The LSE moves by
    the probability-weighted change of the scores, and the bf16 rounding of the
    rotated query changes a score in proportion to its size, so the bound grows
    with the logit scale (qk_scale^2: 3x for the 14B-like workload)."""
    return 2e-2 * wl.qk_scale ** 2


def run_step(case, ring, rope, with_lse=True):
    wl = case.wl
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.Hq, wl.n), dtype=torch.float32, device="cuda") if with_lse else None
    ws = torch.empty(frt.stream_attn_workspace_bytes(ring, wl.n, wl.Hq), dtype=torch.uint8,
                     device="cuda")
    frt.stream_attn_step(ring, rope, gpu_mask(wl), q, k, v, out, ws, lse=lse)
    torch.cuda.synchronize()
    return out, lse


SMALL = {
    "video_small": shrink(WORKLOADS["video_1p3b"], Hq=2, Hkv=2, n=72, C=288,
                          rope=RopeSpec(ROPE_3D, (44, 42, 42), (4, 6)),
                          mask=MaskSpec(MASK_BLOCK_CAUSAL, 72, 4), prior_steps=6),
    "video_partial": shrink(WORKLOADS["video_1p3b"], Hq=3, Hkv=3, n=40, C=96,
                            rope=RopeSpec(ROPE_3D, (44, 42, 42), (2, 4)),
                            mask=MaskSpec(MASK_BLOCK_CAUSAL, 40, 2), prior_steps=1),
    # capacity 16 past a multiple of 32 (a partial last V block, as in the
    # 28080-slot ring), wrapped, window of 6 chunks. Unit-variance Q and K: over
    # a 280-key window the 3x sharper scores of the full-size draw push the
    # bf16 Q/P rounding alone to a mean error of 1.2e-3 (same at C = 256).
    "video_vpart": shrink(WORKLOADS["video_14b"], Hq=2, Hkv=2, n=40, C=240,
                          rope=RopeSpec(ROPE_3D, (44, 42, 42), (2, 4)),
                          mask=MaskSpec(MASK_BLOCK_CAUSAL, 40, 6), prior_steps=9,
                          qk_scale=1.0),
    "gqa_swa": shrink(WORKLOADS["prefill_swa"], B=3, Hq=8, Hkv=2, n=100, C=256,
                      mask=MaskSpec(MASK_CAUSAL, 0, 200), len_lo=0, len_hi=800),
    "mha_causal": shrink(WORKLOADS["prefill_swa"], B=2, Hq=4, Hkv=4, n=37, C=512,
                         mask=MaskSpec(MASK_CAUSAL, 0, 0), len_lo=0, len_hi=400),
    "gqa_d64": shrink(WORKLOADS["prefill_swa"], B=2, Hq=6, Hkv=3, d=64, n=65, C=136,
                      rope=RopeSpec(ROPE_1D, (64, 0, 0)), mask=MaskSpec(MASK_CAUSAL, 0, 120),
                      len_lo=0, len_hi=500),
    # G = 8 at head_dim 64 (the wide preparation blocks at the small head
    # size), a chunk that ends 6 tokens into its second 64-token block
    "gqa8_d64": shrink(WORKLOADS["prefill_swa"], B=2, Hq=16, Hkv=2, d=64, n=70, C=192,
                       rope=RopeSpec(ROPE_1D, (64, 0, 0)), mask=MaskSpec(MASK_CAUSAL, 0, 150),
                       len_lo=0, len_hi=600),
    "g8_block": shrink(WORKLOADS["prefill_swa"], B=1, Hq=16, Hkv=2, n=48, C=96,
                       mask=MaskSpec(MASK_BLOCK_CAUSAL, 48, 2), len_lo=96, len_hi=96),
    "rope_none": shrink(WORKLOADS["prefill_swa"], B=2, Hq=2, Hkv=1, n=33, C=64,
                        rope=RopeSpec(ROPE_NONE), mask=MaskSpec(MASK_CAUSAL, 0, 50),
                        len_lo=0, len_hi=300),
}


@pytest.mark.parametrize("name", ["tiny"] + sorted(SMALL))
@pytest.mark.parametrize("seed", [0, 1])
def test_small_cases_all_rows(name, seed):
    wl = WORKLOADS[name] if name in WORKLOADS else SMALL[name]
    case = make_case(wl, seed)
    ring, oring, rope = build_rings(case)
    out, lse = run_step(case, ring, rope)
    ref, ref_lse = oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
    check_close(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), name)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < lse_tol(wl)
    # attention reads the ring, never writes it
    assert np.array_equal(from_dev(ring.k), oring.k)


def test_straddle_chunk_causal():
    wl = shrink(WORKLOADS["prefill_swa"], B=1, Hq=4, Hkv=2, n=64, C=192,
                mask=MaskSpec(MASK_CAUSAL, 0, 150))
    case = make_case(wl, 3, lengths=np.array([160]))
    ring, oring, rope = build_rings(case)
    out, _ = run_step(case, ring, rope)
    ref, _ = oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
    check_close(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), "straddle")


# Full-size steps, computed once on the GPU and compared with the oracle head
# group by head group (each group's oracle run takes seconds on the host).
_FULL = {}


def _full_size(name, wl, lengths=None):
    if name not in _FULL:
        case = make_case(wl, 0, lengths=lengths)
        ring, oring, rope = build_rings(case)
        out, lse = run_step(case, ring, rope)
        _FULL.clear()  # keep one workload's tensors at a time
        _FULL[name] = (case, oring, bf16_dev_to_f64(out), lse.cpu().numpy(),
                       visible_vmax(oring, case))
    return _FULL[name]


def _oracle_heads(case, oring, kv0, kv1, rows=None):
    """The oracle's output and LSE for KV heads [kv0, kv1) and their query heads."""
    G = case.wl.G
    sub = oracle.RingState(oring.k[:, kv0:kv1], oring.v[:, kv0:kv1], oring.seq_len)
    return oracle.stream_attn(sub, case.q[:, :, kv0 * G:kv1 * G], case.k_new[:, :, kv0:kv1],
                              case.v_new[:, :, kv0:kv1], case.wl.rope, case.wl.mask, rows=rows)


# (workload, stream lengths or None, KV heads per group)
FULL = {
    "video_1p3b": (WORKLOADS["video_1p3b"], None, 6),
    "video_14b": (WORKLOADS["video_14b"], None, 8),
    # the 14B-like step before its ring fills: steps 0 and 1 (4680 and 9360 keys)
    "video_14b_step0": (shrink(WORKLOADS["video_14b"], prior_steps=0), None, 20),
    "video_14b_step1": (shrink(WORKLOADS["video_14b"], prior_steps=1), None, 20),
    "prefill_swa": (WORKLOADS["prefill_swa"], None, 8),
}
FULL_CASES = [(name, g) for name, (wl, _, per) in FULL.items() for g in range(wl.Hkv // per)]


@pytest.mark.parametrize("name,group", FULL_CASES)
def test_full_size_all_rows(name, group):
    """Every output row of the full-size steps, one group of KV heads per case."""
    wl, lengths, per = FULL[name]
    case, oring, got, lse, vmax = _full_size(name, wl, lengths)
    kv0, kv1 = group * per, (group + 1) * per
    ref, ref_lse = _oracle_heads(case, oring, kv0, kv1)
    G = wl.G
    check_close(got[:, :, kv0 * G:kv1 * G], ref, vmax, "%s heads %d-%d" % (name, kv0, kv1))
    assert np.abs(lse[:, kv0 * G:kv1 * G] - ref_lse).max() < lse_tol(wl)


def test_full_size_sampled_rows_pp4():
    """The four-cache step-pipeline layout: sampled rows of every head."""
    wl = WORKLOADS["video_1p3b_pp4"]
    case = make_case(wl, 0)
    ring, oring, rope = build_rings(case)
    out, lse = run_step(case, ring, rope)
    rng = np.random.default_rng(1)
    rows = {0, wl.n - 1, wl.n // 2, 255, 256, 511}
    rows |= set(int(x) for x in rng.integers(0, wl.n, 24))
    rows = np.array(sorted(rows))
    ref, ref_lse = oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                      rows=rows)
    got = bf16_dev_to_f64(out)
    check_close(got[:, rows], ref[:, rows], visible_vmax(oring, case), "pp4")
    assert np.abs(lse.cpu().numpy()[:, :, rows] - ref_lse[:, :, rows]).max() < lse_tol(wl)
    assert np.all(np.isfinite(got))


def test_v_all_ones_gives_ones():
    wl = SMALL["gqa_swa"]
    case = make_case(wl, 4)
    case.v_new[:] = 0x3F80
    for k, v in case.prior_fills:
        v[:] = 0x3F80
    ring, oring, rope = build_rings(case)
    out, _ = run_step(case, ring, rope)
    assert np.abs(bf16_dev_to_f64(out) - 1.0).max() <= 4e-3


def test_poisoned_invisible_slots_do_not_change_output():
    """Never-written and out-of-window slots filled with +-3e4: output bitwise unchanged."""
    wl = SMALL["gqa_swa"]
    case = make_case(wl, 5, lengths=np.array([0, 120, 700]))
    ring, oring, rope = build_rings(case)
    base, _ = run_step(case, ring, rope)
    k = ring.k.clone()
    v = ring.v.clone()
    # stream 0: nothing written; stream 1: slots >= 120 never written;
    # stream 2: L=700, window 200: tokens < 700-199 are invisible to every query
    poison = torch.tensor(29952.0, dtype=torch.bfloat16)
    ring.k[0] = poison
    ring.v[0] = -poison
    ring.k[1, :, 120:] = poison
    ring.v[1, :, ring.v_index(np.arange(120, wl.C)).reshape(-1)] = -poison
    slots = np.arange(700 - 256, 700 - 199) % 256
    ring.k[2, :, torch.from_numpy(slots).cuda()] = poison
    ring.v[2, :, ring.v_index(slots).reshape(-1)] = -poison
    out, _ = run_step(case, ring, rope)
    assert torch.equal(out.view(torch.int16), base.view(torch.int16))
    ring.k.copy_(k)
    ring.v.copy_(v)


def test_deterministic_and_checkpoint_restore():
    """Two identical steps give identical bits; a ring copied mid-stream continues identically."""
    wl = SMALL["video_small"]
    case = make_case(wl, 6)
    ring, oring, rope = build_rings(case, extra_tokens=2 * wl.n)
    a, _ = run_step(case, ring, rope)
    b, _ = run_step(case, ring, rope)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    saved = frt.Ring(wl.B, wl.Hkv, wl.d, wl.C, k=ring.k.clone(), v=ring.v.clone(),
                     seq_len=ring.seq_len.clone())
    for r in (ring, saved):
        frt.kv_append(r, rope, to_dev(case.k_new), to_dev(case.v_new))
    x, _ = run_step(case, ring, rope)
    y, _ = run_step(case, saved, rope)
    assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    assert torch.equal(ring.k.view(torch.int16), saved.k.view(torch.int16))
    assert torch.equal(ring.v.view(torch.int16), saved.v.view(torch.int16))


@pytest.mark.parametrize("name", ["video_small", "video_vpart", "gqa_swa", "gqa_d64", "gqa8_d64"])
def test_stream_step_equals_attn_then_append(name):
    """frt_stream_step over consecutive steps: the same outputs and lse as
    frt_stream_attn_step + frt_kv_append, bit for bit, the same ring bytes and
    lengths, and a ring equal to the oracle's."""
    wl = SMALL[name]
    case = make_case(wl, 4)
    steps = 3
    ring, oring, rope = build_rings(case, extra_tokens=steps * wl.n)
    twin = frt.Ring(wl.B, wl.Hkv, wl.d, wl.C, k=ring.k.clone(), v=ring.v.clone(),
                    seq_len=ring.seq_len.clone())
    nbytes = frt.stream_attn_workspace_bytes(ring, wl.n, wl.Hq)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    ws2 = torch.empty_like(ws)
    rng = np.random.default_rng(12)
    for s in range(steps):
        kn = draw_bf16(rng, case.k_new.shape)  # a fresh chunk each step
        vn = draw_bf16(rng, case.v_new.shape)
        q, k, v = to_dev(case.q), to_dev(kn), to_dev(vn)
        out_a, out_b = torch.empty_like(q), torch.empty_like(q)
        lse_a = torch.empty((wl.B, wl.Hq, wl.n), dtype=torch.float32, device="cuda")
        lse_b = torch.empty_like(lse_a)
        frt.stream_attn_step(twin, rope, gpu_mask(wl), q, k, v, out_a, ws2, lse=lse_a)
        frt.kv_append(twin, rope, k, v)
        frt.stream_step(ring, rope, gpu_mask(wl), q, k, v, out_b, ws, lse=lse_b)
        torch.cuda.synchronize()
        assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16)), (name, s)
        assert torch.equal(lse_a, lse_b), (name, s)
        assert torch.equal(ring.k.view(torch.int16), twin.k.view(torch.int16)), (name, s)
        assert torch.equal(ring.v.view(torch.int16), twin.v.view(torch.int16)), (name, s)
        assert torch.equal(ring.seq_len, twin.seq_len), (name, s)
        oring = oracle.kv_append(oring, kn, vn, wl.rope)
    assert ring_bytes_equal(ring, oring)


def test_very_negative_first_tile():
    """Every row's first visible tile scores below -128 in base-2 units (its keys
    point against the query), the later keys are ordinary: the output is the
    oracle's, not the 0 * inf of rescaling an empty accumulator by exp2(-max)."""
    wl = shrink(WORKLOADS["prefill_swa"], B=1, Hq=2, Hkv=1, n=64, C=256,
                rope=RopeSpec(ROPE_NONE), mask=MaskSpec(MASK_CAUSAL, 0, 0))
    case = make_case(wl, 9, lengths=np.array([160]))
    four = 0x4080  # bf16 4.0
    case.q[:] = four
    k0, _ = case.prior_fills[0]
    k0[:, :64] = four | 0x8000  # tokens 0..63: -4 in every dim, q.k*scale = -181
    small = draw_bf16(np.random.default_rng(3), k0[:, 64:].shape, 0.05)
    k0[:, 64:] = small
    case.k_new[:] = draw_bf16(np.random.default_rng(4), case.k_new.shape, 0.05)
    ring, oring, rope = build_rings(case)
    out, lse = run_step(case, ring, rope)
    ref, ref_lse = oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
    check_close(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), "negative first tile")
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < lse_tol(wl)


@pytest.mark.parametrize("name,j", [("gqa_swa", 57), ("mha_causal", 20), ("gqa_d64", 64)])
def test_future_own_token_has_no_influence(name, j):
    """Causal mask: changing the chunk's own token j (its key and value) leaves the
    outputs and LSE of every query i < j bit for bit unchanged."""
    wl = SMALL[name]
    case = make_case(wl, 13)
    ring, oring, rope = build_rings(case)
    out_a, lse_a = run_step(case, ring, rope)
    rng = np.random.default_rng(14)
    case.k_new[:, j] = draw_bf16(rng, case.k_new[:, j].shape, 3.0)
    case.v_new[:, j] = draw_bf16(rng, case.v_new[:, j].shape, 3.0)
    out_b, lse_b = run_step(case, ring, rope)
    a, b = out_a.view(torch.int16), out_b.view(torch.int16)
    assert torch.equal(a[:, :j], b[:, :j])
    assert torch.equal(lse_a[:, :, :j], lse_b[:, :, :j])
    assert not torch.equal(a[:, j:], b[:, j:])  # the later queries do see it


@pytest.mark.parametrize("C2", [264, 333 - 333 % 8])
def test_ring_capacity_does_not_change_the_result(C2):
    """The same token stream in rings of 256 and of C2 slots (the tokens sit at other
    physical slots, and the tiles cut the visible keys elsewhere): both results
    within tolerance of the oracle, and the oracle's two results equal up to fp64
    rounding (the larger ring holds more, invisible, tokens)."""
    outs = []
    for C in (256, C2):
        wl = shrink(SMALL["gqa_swa"], C=C)
        case = make_case(wl, 15, lengths=np.array([0, 300, 750]))
        ring, oring, rope = build_rings(case)
        out, _ = run_step(case, ring, rope)
        ref, _ = oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
        check_close(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), "C%d" % C)
        outs.append(ref)
    assert np.abs(outs[0] - outs[1]).max() <= 1e-12
