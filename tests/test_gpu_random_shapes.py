"""Seeded random shapes against the oracles: stream counts, GQA groups, head
sizes, ring capacities, chunk lengths, mask kinds and windows, rotary modes and
ring fills (empty, partial, wrapped several times) drawn from a fixed list of
seeds, so every run checks the same cases. Each bf16 case runs the attention
step against the fp64 oracle and the fused step (attention and append) against
the oracle's ring, bit for bit; each FP8 case (head_dim 128) runs the FP8 step
against the FP8 oracle."""
import numpy as np
import pytest
import torch

import oracle
from oracle import fp8
import paper_2607_18171_amd as frt
from workloads import (WORKLOADS, RopeSpec, MaskSpec, ROPE_NONE, ROPE_1D, ROPE_3D,
                       MASK_BLOCK_CAUSAL, MASK_CAUSAL, make_case, shrink)
from gpu_helpers import (to_dev, bf16_dev_to_f64, build_rings, gpu_mask, visible_vmax,
                         check_close, ring_bytes_equal)

pytestmark = pytest.mark.gpu

BF16_SEEDS = list(range(100, 220))
FP8_SEEDS = list(range(300, 348))


def random_workload(seed, d=None):
    """A valid workload drawn from `seed`: capacity a multiple of 8, the chunk no
    longer than the ring, and any window the ring can hold."""
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 4))
    Hkv = int(rng.integers(1, 3))
    G = int(rng.choice([1, 2, 4, 8]))
    d = int(rng.choice([64, 128])) if d is None else d
    C = 8 * int(rng.integers(8, 65))
    n = int(rng.integers(1, min(C, 160) + 1))
    if rng.random() < 0.5:
        window = 0 if rng.random() < 0.3 else int(rng.integers(1, C + 2))
        mask = MaskSpec(MASK_CAUSAL, 0, window)
    else:
        block = int(rng.integers(1, n + 1)) if rng.random() < 0.5 else n
        window = 0 if rng.random() < 0.3 else int(rng.integers(1, C // block + 1))
        mask = MaskSpec(MASK_BLOCK_CAUSAL, block, window)
    mode = int(rng.choice([ROPE_NONE, ROPE_1D, ROPE_3D]))
    if mode == ROPE_NONE:
        rope = RopeSpec(ROPE_NONE)
    elif mode == ROPE_1D:
        rope = RopeSpec(ROPE_1D, (d, 0, 0))
    else:
        dims = (44, 42, 42) if d == 128 else (24, 20, 20)
        rope = RopeSpec(ROPE_3D, dims, (int(rng.integers(1, 7)), int(rng.integers(1, 7))))
    wl = shrink(WORKLOADS["prefill_swa"], B=B, Hq=G * Hkv, Hkv=Hkv, d=d, n=n, C=C, rope=rope,
                mask=mask, len_lo=0, len_hi=3 * C)
    lengths = rng.integers(0, 3 * C + 1, B)
    lengths[int(rng.integers(0, B))] = int(rng.choice([0, C - n // 2, C, 2 * C + 3]))
    return wl, np.maximum(lengths, 0)


def describe(wl):
    m = wl.mask
    kind = "causal" if m.kind == MASK_CAUSAL else "block%d" % m.block
    return "B%d H%d/%d d%d n%d C%d %s w%d rope%d" % (wl.B, wl.Hq, wl.Hkv, wl.d, wl.n, wl.C,
                                                      kind, m.window, wl.rope.mode)


@pytest.mark.parametrize("seed", BF16_SEEDS)
def test_random_shape_matches_oracle(seed):
    wl, lengths = random_workload(seed)
    what = "seed %d: %s" % (seed, describe(wl))
    case = make_case(wl, seed, lengths=lengths)
    ring, oring, rope = build_rings(case, extra_tokens=wl.n)
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    ws = torch.empty(frt.stream_attn_workspace_bytes(ring, wl.n, wl.Hq), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.Hq, wl.n), dtype=torch.float32, device="cuda")
    frt.stream_step(ring, rope, gpu_mask(wl), q, k, v, out, ws, lse=lse)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
    check_close(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), what)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2, what
    oring = oracle.kv_append(oring, case.k_new, case.v_new, wl.rope)
    assert ring_bytes_equal(ring, oring), what


@pytest.mark.parametrize("seed", FP8_SEEDS)
def test_random_shape_fp8_matches_oracle(seed):
    from test_gpu_fp8 import build_fp8_rings, run_fp8_step, check_fp8, vmax_fp8, scales
    wl, lengths = random_workload(seed, d=128)
    what = "seed %d: %s" % (seed, describe(wl))
    case = make_case(wl, seed, lengths=lengths)
    ks, vs = scales(wl, seed)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    out, lse = run_fp8_step(case, ring, rope)
    ref, ref_lse = fp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                       ks, vs)
    check_fp8(bf16_dev_to_f64(out), ref, vmax_fp8(oring, case, vs), what)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2, what


DECODE_SEEDS = list(range(400, 460))
DECODE_FP8_SEEDS = list(range(500, 524))


def random_decode_workload(seed, d=None):
    """A valid one-token decode workload drawn from `seed` (G up to 16: the query
    heads of a KV head are the columns of one 16-wide MFMA)."""
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 20))
    Hkv = int(rng.integers(1, 5))
    G = int(rng.choice([1, 2, 4, 8, 16]))
    d = int(rng.choice([64, 128])) if d is None else d
    C = 8 * int(rng.integers(4, 65))
    if rng.random() < 0.7:
        window = 0 if rng.random() < 0.5 else int(rng.integers(1, C + 2))
        mask = MaskSpec(MASK_CAUSAL, 0, window)
    else:
        block = int(rng.integers(1, min(64, C) + 1))
        window = 0 if rng.random() < 0.3 else int(rng.integers(1, C // block + 1))
        mask = MaskSpec(MASK_BLOCK_CAUSAL, block, window)
    rope = RopeSpec(ROPE_1D, (d, 0, 0)) if rng.random() < 0.8 else RopeSpec(ROPE_NONE)
    wl = shrink(WORKLOADS["decode"], B=B, Hq=G * Hkv, Hkv=Hkv, d=d, C=C, rope=rope, mask=mask,
                len_lo=0, len_hi=3 * C)
    lengths = rng.integers(0, 3 * C + 1, B)
    lengths[int(rng.integers(0, B))] = int(rng.choice([0, 1, C - 1, C, 2 * C + 5]))
    return wl, lengths


@pytest.mark.parametrize("seed", DECODE_SEEDS)
def test_random_decode_matches_oracle(seed):
    wl, lengths = random_decode_workload(seed)
    what = "seed %d: %s" % (seed, describe(wl))
    case = make_case(wl, seed, lengths=lengths)
    ring, oring, rope = build_rings(case, extra_tokens=1)
    q, k, v = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    ws = torch.empty(frt.decode_workspace_bytes(ring, wl.Hq), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(q)
    lse = torch.empty((wl.B, wl.Hq, 1), dtype=torch.float32, device="cuda")
    frt.decode_step(ring, rope, gpu_mask(wl), q, k, v, out, ws, lse=lse)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.decode_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
    check_close(bf16_dev_to_f64(out), ref, visible_vmax(oring, case), what)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2, what
    oring = oracle.kv_append(oring, case.k_new, case.v_new, wl.rope)
    assert ring_bytes_equal(ring, oring), what


@pytest.mark.parametrize("seed", DECODE_FP8_SEEDS)
def test_random_decode_fp8_matches_oracle(seed):
    from test_gpu_fp8 import build_fp8_rings, run_decode_fp8, check_fp8, vmax_fp8, scales
    wl, lengths = random_decode_workload(seed, d=128)
    what = "seed %d: %s" % (seed, describe(wl))
    case = make_case(wl, seed, lengths=lengths)
    ks, vs = scales(wl, seed)
    ring, oring, rope = build_fp8_rings(case, ks, vs)
    out, lse = run_decode_fp8(wl, case, ring, rope)
    ref, ref_lse = fp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                                       ks, vs)
    check_fp8(bf16_dev_to_f64(out), ref, vmax_fp8(oring, case, vs), what)
    assert np.abs(lse.cpu().numpy() - ref_lse).max() < 2e-2, what
