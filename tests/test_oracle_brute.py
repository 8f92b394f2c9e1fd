"""The vectorised oracle against its pure-Python loop twin on small cases (CPU only)."""
import numpy as np
import pytest

import oracle
from oracle import brute
from workloads import (RopeSpec, MaskSpec, ROPE_1D, ROPE_3D, ROPE_NONE,
                       MASK_BLOCK_CAUSAL, MASK_CAUSAL, WORKLOADS, make_case)
from _helpers import rand_bits

CASES = [
    # (rope, mask, B, Hq, Hkv, C, d, prior steps, n)
    (RopeSpec(ROPE_1D, (16, 0, 0)), MaskSpec(MASK_BLOCK_CAUSAL, 4, 0), 1, 2, 2, 12, 16, [4, 4], 4),
    (RopeSpec(ROPE_1D, (16, 0, 0)), MaskSpec(MASK_BLOCK_CAUSAL, 4, 2), 2, 2, 1, 8, 16, [4, 4, 4], 4),
    (RopeSpec(ROPE_3D, (8, 4, 4), (2, 3)), MaskSpec(MASK_BLOCK_CAUSAL, 6, 1), 1, 2, 2, 12, 16, [6, 6, 6], 6),
    (RopeSpec(ROPE_1D, (16, 0, 0)), MaskSpec(MASK_CAUSAL, 0, 0), 2, 4, 2, 16, 16, [3, 5], 3),
    (RopeSpec(ROPE_1D, (16, 0, 0)), MaskSpec(MASK_CAUSAL, 0, 7), 1, 4, 1, 8, 16, [5, 5], 3),
    (RopeSpec(ROPE_NONE), MaskSpec(MASK_CAUSAL, 0, 0), 1, 1, 1, 10, 8, [4, 4, 4], 1),
]


@pytest.mark.parametrize("case", CASES)
def test_vectorised_matches_loops(case):
    rope, mask, B, Hq, Hkv, C, d, steps, n = case
    rng = np.random.default_rng(30)
    ring = oracle.new_ring(B, Hkv, C, d)
    model = brute.ListRing(B, Hkv, C, d)
    for s in steps:
        k = rand_bits(rng, (B, s, Hkv, d))
        v = rand_bits(rng, (B, s, Hkv, d))
        ring = oracle.kv_append(ring, k, v, rope)
        model.append(k.tolist(), v.tolist(), rope)
    q = rand_bits(rng, (B, n, Hq, d), 2.0)
    k = rand_bits(rng, (B, n, Hkv, d), 2.0)
    v = rand_bits(rng, (B, n, Hkv, d))
    out, _ = oracle.stream_attn(ring, q, k, v, rope, mask)
    ref = np.array(brute.attend(model, q.tolist(), k.tolist(), v.tolist(), rope, mask, Hq))
    assert np.allclose(out, ref, rtol=0, atol=1e-12)


def test_tiny_workload_matches_loops():
    wl = WORKLOADS["tiny"]
    c = make_case(wl, 0)
    ring = oracle.new_ring(wl.B, wl.Hkv, wl.C, wl.d)
    model = brute.ListRing(wl.B, wl.Hkv, wl.C, wl.d)
    for k, v in c.prior_steps:
        ring = oracle.kv_append(ring, k, v, wl.rope)
        model.append(k.tolist(), v.tolist(), wl.rope)
    out, _ = oracle.stream_attn(ring, c.q, c.k_new, c.v_new, wl.rope, wl.mask)
    ref = np.array(brute.attend(model, c.q.tolist(), c.k_new.tolist(), c.v_new.tolist(),
                                wl.rope, wl.mask, wl.Hq))
    assert np.allclose(out, ref, rtol=0, atol=1e-12)
