"""Pins for the oracle's masked attention (CPU only)."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import brute
from workloads import (RopeSpec, MaskSpec, ROPE_1D, ROPE_3D, ROPE_NONE,
                       MASK_BLOCK_CAUSAL, MASK_CAUSAL)
from _helpers import golden_lines, rand_bits

NONE = RopeSpec(ROPE_NONE)
R1D = RopeSpec(ROPE_1D, (32, 0, 0))


def _filled_ring(rng, B, Hkv, C, d, steps, rope, per_stream=None):
    ring = oracle.new_ring(B, Hkv, C, d)
    for n in steps:
        ring = oracle.kv_append(ring, rand_bits(rng, (B, n, Hkv, d)),
                                rand_bits(rng, (B, n, Hkv, d)), rope)
    return ring


def test_uniform_scores_give_mean_of_visible_v():
    rng = np.random.default_rng(20)
    B, Hq, Hkv, C, d, n = 2, 4, 2, 24, 32, 6
    ring = _filled_ring(rng, B, Hkv, C, d, [10, 10, 9], R1D)     # L = 29 > C: wrapped
    q = np.zeros((B, n, Hq, d), np.uint16)                      # all scores 0
    k = rand_bits(rng, (B, n, Hkv, d))
    v = rand_bits(rng, (B, n, Hkv, d))
    mask = MaskSpec(MASK_CAUSAL, 0, 20)
    out, lse = oracle.stream_attn(ring, q, k, v, R1D, mask)
    for b in range(B):
        L = int(ring.seq_len[b])
        for i in range(n):
            p = L + i
            for hq in range(Hq):
                h = hq // 2
                rows = []
                for t in range(max(0, p - 19), p + 1):
                    if t < L:
                        assert t >= L - C
                        rows.append(oracle.bf16_to_f64(ring.v[b, h, t % C]))
                    else:
                        rows.append(oracle.bf16_to_f64(v[b, t - L, h]))
                assert np.allclose(out[b, i, hq], np.mean(rows, axis=0), rtol=0, atol=1e-12)
                assert abs(lse[b, hq, i] - math.log(len(rows))) < 1e-12


def test_single_dominant_key_gives_its_v_row():
    rng = np.random.default_rng(21)
    B, H, C, d, n = 1, 1, 40, 32, 4
    ring = _filled_ring(rng, B, H, C, d, [16, 16], NONE)
    q = np.zeros((B, n, H, d), np.uint16)
    q[..., 0] = 0x4000                                  # q = 2 e_0
    ring.k[0, 0, :, :] = 0
    ring.k[0, 0, 7, 0] = 0x4300                         # key token 7: k = 128 e_0, score 256/sqrt(32)
    k = np.zeros((B, n, H, d), np.uint16)
    v = rand_bits(rng, (B, n, H, d))
    out, _ = oracle.stream_attn(ring, q, k, v, NONE, MaskSpec(MASK_BLOCK_CAUSAL, 4, 0))
    target = oracle.bf16_to_f64(ring.v[0, 0, 7])
    for i in range(n):
        assert np.allclose(out[0, i, 0], target, rtol=0, atol=1e-12)


def test_softmax_golden_012():
    w = [float(x) for x in golden_lines("softmax_012.txt")]
    B, H, C, d, n = 1, 1, 8, 4, 1
    ring = oracle.new_ring(B, H, C, d)
    # keys 0,1 cached with k = (0,..), (1,..); own key k = (2,..); q = (1,0,0,0); scale 1
    ring.k[0, 0, 1, 0] = 0x3F80
    ring.seq_len[:] = 2
    rng = np.random.default_rng(22)
    ring.v[0, 0, :2] = rand_bits(rng, (2, d))
    k = np.zeros((B, n, H, d), np.uint16)
    k[0, 0, 0, 0] = 0x4000
    v = rand_bits(rng, (B, n, H, d))
    q = np.zeros((B, n, H, d), np.uint16)
    q[0, 0, 0, 0] = 0x3F80
    out, lse = oracle.stream_attn(ring, q, k, v, NONE, MaskSpec(MASK_CAUSAL, 0, 0), scale=1.0)
    V = np.stack([oracle.bf16_to_f64(ring.v[0, 0, 0]), oracle.bf16_to_f64(ring.v[0, 0, 1]),
                  oracle.bf16_to_f64(v[0, 0, 0])])
    assert np.allclose(out[0, 0, 0], np.array(w) @ V, rtol=0, atol=1e-15)
    assert abs(lse[0, 0, 0] - (2.0 - math.log(w[2]))) < 1e-14


def test_masked_slots_have_no_influence():
    """Poison never-written, evicted-by-window and future-block slots: output unchanged."""
    rng = np.random.default_rng(23)
    B, Hq, Hkv, C, d, n = 2, 2, 1, 32, 32, 8
    ring = _filled_ring(rng, B, Hkv, C, d, [8, 8], R1D)         # L = 16 of 32: 16 slots unwritten
    q = rand_bits(rng, (B, n, Hq, d))
    k = rand_bits(rng, (B, n, Hkv, d))
    v = rand_bits(rng, (B, n, Hkv, d))
    mask = MaskSpec(MASK_BLOCK_CAUSAL, 8, 1)                   # only the previous block is visible
    base, _ = oracle.stream_attn(ring, q, k, v, R1D, mask)
    poisoned = ring.copy()
    poisoned.k[:, :, 16:] = 0x46EA     # 29952.0: never-written slots
    poisoned.v[:, :, 16:] = 0xC6EA
    poisoned.k[:, :, 0:8] = 0x46EA     # tokens 0..7: two blocks back, outside the window
    poisoned.v[:, :, 0:8] = 0xC6EA
    out, _ = oracle.stream_attn(poisoned, q, k, v, R1D, mask)
    assert np.array_equal(out, base)


def test_causal_future_own_tokens_have_no_influence():
    rng = np.random.default_rng(24)
    B, H, C, d, n = 1, 2, 16, 32, 8
    ring = _filled_ring(rng, B, H, C, d, [5], R1D)
    q = rand_bits(rng, (B, n, H, d))
    k = rand_bits(rng, (B, n, H, d))
    v = rand_bits(rng, (B, n, H, d))
    mask = MaskSpec(MASK_CAUSAL, 0, 0)
    base, _ = oracle.stream_attn(ring, q, k, v, R1D, mask)
    k2, v2 = k.copy(), v.copy()
    k2[0, 5:] ^= 0x1234
    v2[0, 5:] ^= 0x0F0F
    out, _ = oracle.stream_attn(ring, q, k2, v2, R1D, mask)
    assert np.array_equal(out[0, :5], base[0, :5])
    assert not np.array_equal(out[0, 5:], base[0, 5:])


def test_rows_sum_to_one():
    rng = np.random.default_rng(25)
    B, Hq, Hkv, C, d, n = 1, 4, 2, 20, 32, 6
    ring = _filled_ring(rng, B, Hkv, C, d, [6, 6, 6, 6], R1D)
    q = rand_bits(rng, (B, n, Hq, d), 3.0)
    k = rand_bits(rng, (B, n, Hkv, d), 3.0)
    v = rand_bits(rng, (B, n, Hkv, d))
    _, _, probs = oracle.stream_attn(ring, q, k, v, R1D, MaskSpec(MASK_BLOCK_CAUSAL, 6, 2),
                                     return_probs=True)
    for (_, _), (P, _) in probs.items():
        assert np.all(np.abs(P.sum(axis=1) - 1.0) < 1e-12)
        assert np.all(P >= 0)


@pytest.mark.parametrize("mask", [MaskSpec(MASK_BLOCK_CAUSAL, 5, 0), MaskSpec(MASK_BLOCK_CAUSAL, 5, 2),
                                  MaskSpec(MASK_CAUSAL, 0, 0), MaskSpec(MASK_CAUSAL, 0, 9)])
def test_matches_torch_sdpa_float64(mask):
    """torch's scaled_dot_product_attention (float64, CPU, explicit boolean mask)."""
    rng = np.random.default_rng(26)
    B, Hq, Hkv, C, d, n = 2, 4, 2, 16, 32, 5
    ring = _filled_ring(rng, B, Hkv, C, d, [5, 5, 5, 5], R1D)
    q = rand_bits(rng, (B, n, Hq, d))
    k = rand_bits(rng, (B, n, Hkv, d))
    v = rand_bits(rng, (B, n, Hkv, d))
    out, _ = oracle.stream_attn(ring, q, k, v, R1D, mask)
    for b in range(B):
        L = int(ring.seq_len[b])
        ptok = L + np.arange(n)
        for hq in range(Hq):
            h = hq // 2
            ktok, K, V = oracle.attention_inputs(ring, b, h, k, v, R1D)
            qh = oracle.rotate_f64(q[b, :, hq], ptok, R1D)
            allowed = oracle.visible(mask, ptok[:, None], ktok[None, :])
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(qh)[None], torch.from_numpy(K)[None], torch.from_numpy(V)[None],
                attn_mask=torch.from_numpy(allowed)[None])[0].numpy()
            assert np.allclose(out[b, :, hq], ref, rtol=0, atol=1e-12)


def test_gqa_equals_mha_with_replicated_kv():
    rng = np.random.default_rng(27)
    B, Hq, Hkv, C, d, n = 1, 6, 2, 16, 32, 4
    ring = _filled_ring(rng, B, Hkv, C, d, [4, 4, 4], R1D)
    q = rand_bits(rng, (B, n, Hq, d))
    k = rand_bits(rng, (B, n, Hkv, d))
    v = rand_bits(rng, (B, n, Hkv, d))
    mask = MaskSpec(MASK_CAUSAL, 0, 0)
    out, _ = oracle.stream_attn(ring, q, k, v, R1D, mask)
    rep = oracle.RingState(np.repeat(ring.k, 3, axis=1), np.repeat(ring.v, 3, axis=1),
                           ring.seq_len.copy())
    out2, _ = oracle.stream_attn(rep, q, np.repeat(k, 3, axis=2), np.repeat(v, 3, axis=2), R1D, mask)
    assert np.array_equal(out, out2)


def test_row_subset_equals_full():
    rng = np.random.default_rng(28)
    B, H, C, d, n = 1, 2, 32, 32, 12
    ring = _filled_ring(rng, B, H, C, d, [12, 12], R1D)
    q = rand_bits(rng, (B, n, H, d))
    k = rand_bits(rng, (B, n, H, d))
    v = rand_bits(rng, (B, n, H, d))
    mask = MaskSpec(MASK_CAUSAL, 0, 0)
    full, lse = oracle.stream_attn(ring, q, k, v, R1D, mask, row_block=5)
    rows = np.array([0, 3, 11])
    sub, lse2 = oracle.stream_attn(ring, q, k, v, R1D, mask, rows=rows)
    assert np.array_equal(sub[:, rows], full[:, rows])
    assert np.array_equal(lse2[:, :, rows], lse[:, :, rows])


@pytest.mark.parametrize("shift", [1, 7, 23])
def test_physical_ring_rotation_does_not_change_the_result(shift):
    """The same visible keys at another physical offset: ring B first takes `shift`
    tokens that end up outside the causal window, then the same token values as
    ring A, so every slot holds A's value `shift` slots further on. Without RoPE
    and under a relative (causal-window) mask, the step's result is the same up to
    fp64 rounding; an error in the slot <-> token map reads other keys in one of
    the two rings and breaks it."""
    rng = np.random.default_rng(30)
    B, H, C, d, n, W = 1, 2, 24, 32, 5, 16
    mask = MaskSpec(MASK_CAUSAL, 0, W)
    toks_k = rand_bits(rng, (B, 40, H, d))
    toks_v = rand_bits(rng, (B, 40, H, d))
    junk_k = rand_bits(rng, (B, shift, H, d))
    junk_v = rand_bits(rng, (B, shift, H, d))
    q = rand_bits(rng, (B, n, H, d))
    k = rand_bits(rng, (B, n, H, d))
    v = rand_bits(rng, (B, n, H, d))
    ra = oracle.new_ring(B, H, C, d)
    for s in range(0, 40, 8):
        ra = oracle.kv_append(ra, toks_k[:, s:s + 8], toks_v[:, s:s + 8], NONE)
    rb = oracle.kv_append(oracle.new_ring(B, H, C, d), junk_k, junk_v, NONE)
    for s in range(0, 40, 8):
        rb = oracle.kv_append(rb, toks_k[:, s:s + 8], toks_v[:, s:s + 8], NONE)
    # same values, slots rotated by `shift`
    assert np.array_equal(np.roll(ra.k, shift, axis=2), rb.k)
    oa, la = oracle.stream_attn(ra, q, k, v, NONE, mask)
    ob, lb = oracle.stream_attn(rb, q, k, v, NONE, mask)
    assert np.abs(oa - ob).max() <= 1e-12
    assert np.abs(la - lb).max() <= 1e-12


def test_ring_capacity_beyond_the_window_does_not_change_the_result():
    """One token stream in rings of C = window - 1 (the least a causal window of W
    keys needs) and of larger capacities: equal results up to fp64 rounding."""
    rng = np.random.default_rng(31)
    B, H, d, n, W = 2, 2, 32, 6, 20
    mask = MaskSpec(MASK_CAUSAL, 0, W)
    kk = rand_bits(rng, (B, 50, H, d))
    vv = rand_bits(rng, (B, 50, H, d))
    q = rand_bits(rng, (B, n, H, d))
    k = rand_bits(rng, (B, n, H, d))
    v = rand_bits(rng, (B, n, H, d))
    outs = []
    for C in (W - 1, W + 5, 64):
        ring = oracle.new_ring(B, H, C, d)
        for s in range(0, 50, 10):
            ring = oracle.kv_append(ring, kk[:, s:s + 10], vv[:, s:s + 10], R1D)
        outs.append(oracle.stream_attn(ring, q, k, v, R1D, mask))
    for o, l in outs[1:]:
        assert np.abs(o - outs[0][0]).max() <= 1e-12
        assert np.abs(l - outs[0][1]).max() <= 1e-12
