"""FP8 (e4m3fn) ring append and step attention on the GPU against the FP8
oracle: ring bytes bit for bit, attention outputs within tolerance."""
import numpy as np
import pytest
import torch

import oracle
from oracle import fp8
import paper_2607_18171_amd as frt
from workloads import (WORKLOADS, RopeSpec, MaskSpec, ROPE_3D, MASK_BLOCK_CAUSAL, MASK_CAUSAL,
                       make_case, shrink, draw_bf16)
from gpu_helpers import to_dev, from_dev, bf16_dev_to_f64, gpu_rope, gpu_mask

pytestmark = pytest.mark.gpu


def scales(wl, seed):
    """Per-(stream, KV head) scales putting N(0, 1)-sized values well inside +-448."""
    rng = np.random.default_rng(100 + seed)
    ks = rng.uniform(0.01, 0.04, (wl.B, wl.Hkv)).astype(np.float32) * wl.qk_scale
    vs = rng.uniform(0.01, 0.04, (wl.B, wl.Hkv)).astype(np.float32)
    return ks, vs


def build_fp8_rings(case, ks, vs, extra_tokens=0):
    wl = case.wl
    max_tok = int(case.prior_lengths.max()) + wl.n + extra_tokens + 1
    rope = gpu_rope(wl, max_tok)
    ring = frt.RingFp8(wl.B, wl.Hkv, wl.d, wl.C, torch.from_numpy(ks), torch.from_numpy(vs))
    oring = fp8.RingFP8(wl.B, wl.Hkv, wl.C, wl.d)
    for k, v in case.prior_steps:
        frt.kv_append_fp8(ring, rope, to_dev(k), to_dev(v))
        fp8.kv_append_fp8(oring, k, v, wl.rope, ks, vs)
    for b, (k, v) in enumerate(case.prior_fills):
        n = k.shape[1]
        for s in range(0, n, wl.C):
            e = min(n, s + wl.C)
            frt.kv_append_fp8(ring.view_stream(b), rope, to_dev(k[:, s:e]), to_dev(v[:, s:e]))
            fp8.kv_append_fp8(oring, k[:, s:e], v[:, s:e], wl.rope, ks, vs, streams=[b])
    return ring, oring, rope


def ring_codes_equal(ring, oring):
    k = ring.k.cpu().numpy()
    v = ring.v[:, :, ring.v_index().reshape(-1)].reshape(ring.B, ring.Hkv, ring.C, ring.d)
    return (np.array_equal(k, oring.k) and np.array_equal(v.cpu().numpy(), oring.v)
            and np.array_equal(ring.seq_len.cpu().numpy(), oring.seq_len))


def run_fp8_step(case, ring, rope, rows_lse=True):
    wl = case.wl
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.Hq, wl.n), dtype=torch.float32, device="cuda")
    ws = torch.empty(frt.stream_attn_fp8_workspace_bytes(ring, wl.n, wl.Hq), dtype=torch.uint8,
                     device="cuda")
    frt.stream_attn_step_fp8(ring, rope, gpu_mask(wl), q, k, v, out, ws, lse=lse)
    torch.cuda.synchronize()
    return out, lse


SMALL = {
    "video_small": shrink(WORKLOADS["video_1p3b"], Hq=2, Hkv=2, n=72, C=288,
                          rope=RopeSpec(ROPE_3D, (44, 42, 42), (4, 6)),
                          mask=MaskSpec(MASK_BLOCK_CAUSAL, 72, 4), prior_steps=6),
    # unit-variance Q and K: see the note on the tolerance below
    "video_vpart": shrink(WORKLOADS["video_14b"], Hq=2, Hkv=2, n=40, C=240,
                          rope=RopeSpec(ROPE_3D, (44, 42, 42), (2, 4)),
                          mask=MaskSpec(MASK_BLOCK_CAUSAL, 40, 6), prior_steps=9,
                          qk_scale=1.0),
    "gqa_swa": shrink(WORKLOADS["prefill_swa"], B=3, Hq=8, Hkv=2, n=100, C=256,
                      mask=MaskSpec(MASK_CAUSAL, 0, 200), len_lo=0, len_hi=800),
    "mha_causal": shrink(WORKLOADS["prefill_swa"], B=2, Hq=4, Hkv=4, n=37, C=512,
                         mask=MaskSpec(MASK_CAUSAL, 0, 0), len_lo=0, len_hi=400),
    "rope_none": shrink(WORKLOADS["prefill_swa"], B=2, Hq=2, Hkv=1, n=33, C=64,
                        rope=RopeSpec(0), mask=MaskSpec(MASK_CAUSAL, 0, 50),
                        len_lo=0, len_hi=300),
}

# Error sources between the kernel and the FP8 oracle: fp32 accumulation of
# the exact code products, the hardware exp2, and so the rare weight whose
# exact value lies within that error of a rounding boundary of the code (one
# code step is 1/8 to 1/16 of the weight); bf16 rounding of the output. And
# one of definition: the oracle codes weights against m = ceil(row max), the
# kernel against its running integer max, at most one below it between
# raises, so only weights in the subnormal codes (2^-13 of the largest and
# less) can round differently; on the full-size 14B-like step (32760 keys of
# 3x unit logits, the widest spread of mass here) that is 0.5% of max|V| at
# most and 3e-4 on average.
MAX_REL_V = 1e-2   # of max |v_scale * value(code)| over the visible values
MEAN_ABS = 1e-3


def vmax_fp8(oring, case, vs):
    wl = case.wl
    vals = [np.abs(fp8.e4m3_decode(fp8.stored_v8(case.v_new[b, :, h, :], vs[b, h])) * vs[b, h]).max()
            for b in range(wl.B) for h in range(wl.Hkv)]
    vals.append(max(np.abs(fp8.e4m3_decode(oring.v[b, h]) * vs[b, h]).max()
                    for b in range(wl.B) for h in range(wl.Hkv)))
    return float(max(vals))


def check_fp8(got, ref, vmax, what):
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got)), what
    mx, mean = float(err.max()), float(err.mean())
    print("%s: max|err| %.3g (%.3g of max|V|) mean %.3g" % (what, mx, mx / vmax, mean))
    assert mx <= MAX_REL_V * vmax, "%s: max|err| %.3g > %.3g" % (what, mx, MAX_REL_V * vmax)
    assert mean <= MEAN_ABS, "%s: mean|err| %.3g" % (what, mean)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_fp8_append_codes_match_oracle(name):
    wl = SMALL[name]
    case = make_case(wl, 0)
    ks, vs = scales(wl, 0)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    assert ring_codes_equal(ring, oring)


@pytest.mark.parametrize("name", sorted(SMALL))
@pytest.mark.parametrize("seed", [0, 1])
def test_fp8_attention_small(name, seed):
    wl = SMALL[name]
    case = make_case(wl, seed)
    ks, vs = scales(wl, seed)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    out, lse = run_fp8_step(case, ring, rope)
    ref, ref_lse = fp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                       ks, vs)
    check_fp8(bf16_dev_to_f64(out), ref, vmax_fp8(oring, case, vs), name)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2
    assert ring_codes_equal(ring, oring)  # attention reads the ring only


@pytest.mark.parametrize("name", ["video_1p3b", "video_14b"])
def test_fp8_attention_full_size_sampled_rows(name):
    wl = WORKLOADS[name]
    case = make_case(wl, 0)
    ks, vs = scales(wl, 0)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    out, lse = run_fp8_step(case, ring, rope)
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([[0, 255, 256, wl.n - 1], rng.integers(0, wl.n, 12)]))
    ref, ref_lse = fp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                       ks, vs, rows=rows)
    check_fp8(bf16_dev_to_f64(out)[:, rows], ref[:, rows], vmax_fp8(oring, case, vs), name)
    assert np.abs(lse.cpu().numpy()[:, :, rows] - ref_lse[:, :, rows]).max() < 2e-2


@pytest.mark.parametrize("name", ["video_small", "video_vpart", "gqa_swa", "mha_causal"])
def test_fp8_stream_step_equals_attn_then_append(name):
    """frt_stream_step_fp8 over consecutive steps: the same outputs and lse as
    frt_stream_attn_step_fp8 + frt_kv_append_fp8, bit for bit, the same ring
    codes and lengths, and ring codes equal to the FP8 oracle's."""
    wl = SMALL[name]
    case = make_case(wl, 4)
    ks, vs = scales(wl, 4)
    steps = 3
    ring, oring, rope = build_fp8_rings(case, ks, vs, extra_tokens=steps * wl.n)
    twin = frt.RingFp8(wl.B, wl.Hkv, wl.d, wl.C, torch.from_numpy(ks), torch.from_numpy(vs))
    twin.k.copy_(ring.k)
    twin.v.copy_(ring.v)
    twin.seq_len.copy_(ring.seq_len)
    nbytes = frt.stream_attn_fp8_workspace_bytes(ring, wl.n, wl.Hq)
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
        frt.stream_attn_step_fp8(twin, rope, gpu_mask(wl), q, k, v, out_a, ws2, lse=lse_a)
        frt.kv_append_fp8(twin, rope, k, v)
        frt.stream_step_fp8(ring, rope, gpu_mask(wl), q, k, v, out_b, ws, lse=lse_b)
        torch.cuda.synchronize()
        assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16)), (name, s)
        assert torch.equal(lse_a, lse_b), (name, s)
        assert torch.equal(ring.k, twin.k), (name, s)
        assert torch.equal(ring.v, twin.v), (name, s)
        assert torch.equal(ring.seq_len, twin.seq_len), (name, s)
        fp8.kv_append_fp8(oring, kn, vn, wl.rope, ks, vs)
    assert ring_codes_equal(ring, oring)


def test_fp8_saturating_scales():
    """Scales small enough that many values lie beyond +-448 codes: the ring
    holds the clamped codes bit for bit as the oracle does, and attention
    over them (and the step's own clamped codes) stays within tolerance."""
    wl = SMALL["gqa_swa"]
    case = make_case(wl, 5)
    ks = np.full((wl.B, wl.Hkv), 2e-3, np.float32)  # |k| > 0.9 saturates
    vs = np.full((wl.B, wl.Hkv), 3e-3, np.float32)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    codes = ring.k.cpu().numpy()
    assert np.isin(codes, [0x7e, 0xfe]).mean() > 0.1  # the clamp is exercised
    assert ring_codes_equal(ring, oring)
    out, lse = run_fp8_step(case, ring, rope)
    ref, ref_lse = fp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                       ks, vs)
    check_fp8(bf16_dev_to_f64(out), ref, vmax_fp8(oring, case, vs), "saturating")
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2


def test_fp8_attention_rejects_head_dim_64():
    wl = shrink(WORKLOADS["prefill_swa"], B=1, Hq=2, Hkv=1, d=64, n=8, C=64,
                rope=RopeSpec(0), mask=MaskSpec(MASK_CAUSAL, 0, 0), len_lo=8, len_hi=8)
    case = make_case(wl, 0)
    ks, vs = scales(wl, 0)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    assert ring_codes_equal(ring, oring)  # the append supports head_dim 64
    with pytest.raises(frt.FrtError):
        run_fp8_step(case, ring, rope)


# ---- FP8 decode: the FP8 step's attention with one token per stream ----

DECODE = {
    "decode": (WORKLOADS["decode"], None),
    "split_edges": (shrink(WORKLOADS["decode"], B=6, C=1024), [0, 1, 255, 256, 257, 1023]),
    "wrapped_window": (shrink(WORKLOADS["decode"], B=3, Hq=8, Hkv=1, C=512,
                              mask=MaskSpec(MASK_CAUSAL, 0, 300)), [1000, 299, 512]),
    "mha_g1": (shrink(WORKLOADS["decode"], B=2, Hq=4, Hkv=4, C=264), [100, 263]),
    "g16": (shrink(WORKLOADS["decode"], B=2, Hq=32, Hkv=2, C=328), [327, 40]),
    "block_causal": (shrink(WORKLOADS["decode"], B=2, Hq=8, Hkv=2, C=512,
                            mask=MaskSpec(MASK_BLOCK_CAUSAL, 128, 2)), [300, 511]),
    # more streams than one 64-lane scan group (twice over), empty to full rings
    "streams_130": (shrink(WORKLOADS["decode"], B=130, Hq=4, Hkv=2, C=256),
                    [0, 255, 1] + [(37 * b + 5) % 256 for b in range(3, 130)]),
}


def decode_case(name, seed):
    wl, lengths = DECODE[name]
    case = make_case(wl, seed, lengths=None if lengths is None else np.array(lengths))
    ks, vs = scales(wl, seed)
    return wl, case, ks, vs


def run_decode_fp8(wl, case, ring, rope, step=False):
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.Hq, 1), dtype=torch.float32, device="cuda")
    ws = torch.empty(frt.decode_fp8_workspace_bytes(ring, wl.Hq), dtype=torch.uint8,
                     device="cuda")
    fn = frt.decode_step_fp8 if step else frt.decode_attn_fp8
    fn(ring, rope, gpu_mask(wl), q, k, v, out, ws, lse=lse)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("name", sorted(DECODE))
def test_fp8_decode_matches_oracle(name):
    wl, case, ks, vs = decode_case(name, 0)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    out, lse = run_decode_fp8(wl, case, ring, rope)
    ref, ref_lse = fp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                       ks, vs)
    check_fp8(bf16_dev_to_f64(out), ref, vmax_fp8(oring, case, vs), name)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2
    assert ring_codes_equal(ring, oring)  # decode attention reads the ring only


@pytest.mark.parametrize("name", ["split_edges", "wrapped_window", "g16"])
def test_fp8_decode_step_equals_attn_then_append(name):
    """frt_decode_step_fp8 over consecutive steps: the same outputs and lse as
    frt_decode_attn_fp8 + frt_kv_append_fp8, bit for bit, the same ring codes
    and lengths, and ring codes equal to the FP8 oracle's."""
    wl, case, ks, vs = decode_case(name, 3)
    steps = 3
    ring, oring, rope = build_fp8_rings(case, ks, vs, extra_tokens=steps)
    twin = frt.RingFp8(wl.B, wl.Hkv, wl.d, wl.C, torch.from_numpy(ks), torch.from_numpy(vs))
    twin.k.copy_(ring.k)
    twin.v.copy_(ring.v)
    twin.seq_len.copy_(ring.seq_len)
    nbytes = frt.decode_fp8_workspace_bytes(ring, wl.Hq)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    ws2 = torch.empty_like(ws)
    rng = np.random.default_rng(13)
    for s in range(steps):
        qn = draw_bf16(rng, case.q.shape)
        kn = draw_bf16(rng, case.k_new.shape)
        vn = draw_bf16(rng, case.v_new.shape)
        q, k, v = to_dev(qn), to_dev(kn), to_dev(vn)
        out_a, out_b = torch.empty_like(q), torch.empty_like(q)
        lse_a = torch.empty((wl.B, wl.Hq, 1), dtype=torch.float32, device="cuda")
        lse_b = torch.empty_like(lse_a)
        frt.decode_attn_fp8(twin, rope, gpu_mask(wl), q, k, v, out_a, ws2, lse=lse_a)
        frt.kv_append_fp8(twin, rope, k, v)
        frt.decode_step_fp8(ring, rope, gpu_mask(wl), q, k, v, out_b, ws, lse=lse_b)
        torch.cuda.synchronize()
        assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16)), (name, s)
        assert torch.equal(lse_a, lse_b), (name, s)
        assert torch.equal(ring.k, twin.k), (name, s)
        assert torch.equal(ring.v, twin.v), (name, s)
        assert torch.equal(ring.seq_len, twin.seq_len), (name, s)
        ref, _ = fp8.stream_attn_fp8(oring, qn, kn, vn, wl.rope, wl.mask, ks, vs)
        vmax = max(vmax_fp8(oring, case, vs),
                   max(np.abs(fp8.e4m3_decode(fp8.stored_v8(vn[b, :, h, :], vs[b, h])) * vs[b, h]).max()
                       for b in range(wl.B) for h in range(wl.Hkv)))
        check_fp8(bf16_dev_to_f64(out_b), ref, vmax, "%s step %d" % (name, s))
        fp8.kv_append_fp8(oring, kn, vn, wl.rope, ks, vs)
    assert ring_codes_equal(ring, oring)


def test_fp8_decode_rejects_head_dim_64():
    wl = shrink(WORKLOADS["decode"], B=1, Hq=2, Hkv=1, d=64, C=64,
                rope=RopeSpec(0), mask=MaskSpec(MASK_CAUSAL, 0, 0))
    case = make_case(wl, 0, lengths=np.array([10]))
    ks, vs = scales(wl, 0)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    with pytest.raises(frt.FrtError):
        run_decode_fp8(wl, case, ring, rope)


# ---- the FP8 step against exact attention (the fp64 oracle on the same inputs) ----
from _helpers import FP8_MAX_REL_V, FP8_MEAN, e4m3_exact_case_values  # noqa: E402
from gpu_helpers import visible_vmax, check_close, MAX_ERR_REL_V, MEAN_ERR  # noqa: E402

EXACT_SMALL = dict(SMALL)
# the 14B-like step's logit scale (Q and K drawn with std sqrt(3)) over a short window
EXACT_SMALL["video_vpart_std3"] = shrink(SMALL["video_vpart"], qk_scale=float(np.sqrt(3.0)))


def exact_oracle_ring(case):
    wl = case.wl
    oring = oracle.new_ring(wl.B, wl.Hkv, wl.C, wl.d)
    for k, v in case.prior_steps:
        oring = oracle.kv_append(oring, k, v, wl.rope)
    for b, (k, v) in enumerate(case.prior_fills):
        for s in range(0, k.shape[1], wl.C):
            e = min(k.shape[1], s + wl.C)
            oring = oracle.kv_append(oring, k[:, s:e], v[:, s:e], wl.rope, streams=[b])
    return oring


def check_fp8_vs_exact(got, ref, vmax, what):
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got)), what
    mx, mean = float(err.max()), float(err.mean())
    print("%s vs exact: max|err| %.3g of max|V|, mean %.3g" % (what, mx / vmax, mean))
    assert mx <= FP8_MAX_REL_V * vmax, "%s: max|err| %.3g of max|V|" % (what, mx / vmax)
    assert mean <= FP8_MEAN, "%s: mean|err| %.3g" % (what, mean)


@pytest.mark.parametrize("name", sorted(EXACT_SMALL))
def test_fp8_attention_small_against_exact(name):
    wl = EXACT_SMALL[name]
    case = make_case(wl, 2)
    ks, vs = scales(wl, 2)
    ring, _, rope = build_fp8_rings(case, ks, vs)
    out, _ = run_fp8_step(case, ring, rope)
    oring = exact_oracle_ring(case)
    ref, _ = oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
    check_fp8_vs_exact(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), name)


@pytest.mark.parametrize("name", ["video_1p3b", "video_14b", "prefill_swa", "decode"])
def test_fp8_full_size_against_exact(name):
    wl = WORKLOADS[name]
    case = make_case(wl, 0)
    ks, vs = scales(wl, 0)
    ring, _, rope = build_fp8_rings(case, ks, vs)
    if wl.n == 1:
        out, _ = run_decode_fp8(wl, case, ring, rope)
        rows = np.array([0])
    else:
        out, _ = run_fp8_step(case, ring, rope)
        rows = np.unique(np.linspace(0, wl.n - 1, 64).astype(np.int64))
    oring = exact_oracle_ring(case)
    ref, _ = oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                rows=rows)
    check_fp8_vs_exact(bf16_dev_to_f64(out)[:, rows], ref[:, rows], visible_vmax(oring, case),
                       name)


def test_fp8_equals_exact_attention_on_inputs_the_format_represents():
    """No rotation, softmax scale ln 2 (base-2 scores equal q.k), scales 1, integer
    queries and keys and quarter-integer values e4m3 represents, scores within 8 of
    each row's maximum (so every weight is a normal e4m3 code): every operand and
    weight the FP8 kernel codes is exact, so its result is exact attention up to
    fp32 accumulation and the bf16 output rounding."""
    wl = shrink(WORKLOADS["prefill_swa"], B=2, Hq=4, Hkv=2, n=70, C=192, rope=RopeSpec(0),
                mask=MaskSpec(MASK_CAUSAL, 0, 150), len_lo=0, len_hi=400)
    case = make_case(wl, 6, lengths=np.array([130, 300]))
    rng = np.random.default_rng(7)
    for i, (k, v) in enumerate(case.prior_fills):
        case.prior_fills[i] = (e4m3_exact_case_values(rng, k.shape, -1, 1, 1),
                               e4m3_exact_case_values(rng, v.shape, -4, 4, 0.25))
    case.k_new[:] = e4m3_exact_case_values(rng, case.k_new.shape, -1, 1, 1)
    case.v_new[:] = e4m3_exact_case_values(rng, case.v_new.shape, -4, 4, 0.25)
    case.q[:] = 0
    for b in range(wl.B):
        for i in range(wl.n):
            for h in range(wl.Hq):
                dims = rng.choice(wl.d, 4, replace=False)
                case.q[b, i, h, dims] = e4m3_exact_case_values(rng, 4, -1, 1, 2) | 0x3f80
    ones = np.ones((wl.B, wl.Hkv), np.float32)
    ring, oring8, rope = build_fp8_rings(case, ones, ones)
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    out = torch.empty_like(q)
    ws = torch.empty(frt.stream_attn_fp8_workspace_bytes(ring, wl.n, wl.Hq), dtype=torch.uint8,
                     device="cuda")
    ln2 = float(np.float32(np.log(2.0)))
    frt.stream_attn_step_fp8(ring, rope, gpu_mask(wl), q, k, v, out, ws, softmax_scale=ln2)
    torch.cuda.synchronize()
    oring = exact_oracle_ring(case)
    ref, _ = oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                scale=ln2)
    got = bf16_dev_to_f64(out)
    check_close(got, ref, visible_vmax(oring, case), "exact inputs")
    # the rounding of the output to bf16 is the only error left
    excess = np.abs(got - ref) - (np.abs(ref) * 2.0 ** -8 + 1e-6)
    w = np.unravel_index(np.argmax(excess), excess.shape)
    assert excess.max() <= 0, (w, got[w], ref[w])


def test_fp8_very_negative_first_tile():
    """Every row's first visible tile scores far below the row's later keys: the FP8
    kernel's first raise of its reference max must not turn the empty accumulator
    into 0 * inf."""
    wl = shrink(WORKLOADS["prefill_swa"], B=1, Hq=2, Hkv=1, n=64, C=256, rope=RopeSpec(0),
                mask=MaskSpec(MASK_CAUSAL, 0, 0))
    case = make_case(wl, 9, lengths=np.array([160]))
    case.q[:] = 0x4080  # 4.0
    k0, _ = case.prior_fills[0]
    k0[:, :64] = 0x4080 | 0x8000
    k0[:, 64:] = draw_bf16(np.random.default_rng(3), k0[:, 64:].shape, 0.05)
    case.k_new[:] = draw_bf16(np.random.default_rng(4), case.k_new.shape, 0.05)
    ks = np.full((1, 1), 0.02, np.float32)
    vs = np.full((1, 1), 0.02, np.float32)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    out, lse = run_fp8_step(case, ring, rope)
    ref, ref_lse = fp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                       ks, vs)
    check_fp8(bf16_dev_to_f64(out), ref, vmax_fp8(oring, case, vs), "negative first tile")
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2


@pytest.mark.parametrize("slope", [0.0175, 0.245])
def test_fp8_reference_max_climbing_along_the_row(slope):
    """Scores that rise steadily along the keys (by about 8, or about 100, base-2
    units over a row): the reference max is raised tile after tile, the PV
    products carry 2^(m - m0) in the MFMA's B scale, and past 64 units the row
    re-bases once. Against the FP8 oracle within its tolerance, LSE included."""
    wl = shrink(WORKLOADS["prefill_swa"], B=1, Hq=2, Hkv=1, n=64, C=256, rope=RopeSpec(0),
                mask=MaskSpec(MASK_CAUSAL, 0, 0))
    L = 160
    case = make_case(wl, 11, lengths=np.array([L]))
    rng = np.random.default_rng(12)

    def bf16_bits(x):
        b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
        return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)

    q = rng.standard_normal(case.q.shape).astype(np.float32) * 0.05
    q[..., 0] = 16.0
    case.q[:] = bf16_bits(q)
    k0, _ = case.prior_fills[0]
    kp = rng.standard_normal(k0.shape).astype(np.float32) * 0.05
    kp[0, :, 0, 0] = slope * np.arange(L)
    k0[:] = bf16_bits(kp)
    kn = rng.standard_normal(case.k_new.shape).astype(np.float32) * 0.05
    kn[0, :, 0, 0] = slope * np.arange(L, L + wl.n)
    case.k_new[:] = bf16_bits(kn)
    ks = np.full((1, 1), 0.125, np.float32)
    vs = np.full((1, 1), 0.02, np.float32)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    out, lse = run_fp8_step(case, ring, rope)
    ref, ref_lse = fp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                       ks, vs)
    check_fp8(bf16_dev_to_f64(out), ref, vmax_fp8(oring, case, vs), "slope %g" % slope)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2
