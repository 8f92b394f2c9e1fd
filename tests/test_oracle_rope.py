"""Pins for the oracle's rotary embedding and rounding (CPU only)."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import rope as orope
from workloads import RopeSpec, ROPE_1D, ROPE_3D, ROPE_NONE, f32_to_bf16_bits
from _helpers import golden_lines, rand_bits

R1D64 = RopeSpec(ROPE_1D, (64, 0, 0))
R1D128 = RopeSpec(ROPE_1D, (128, 0, 0))
R3D = RopeSpec(ROPE_3D, (44, 42, 42), (30, 52))


@pytest.mark.parametrize("rope,d", [(R1D64, 64), (R1D128, 128), (R3D, 128)])
def test_position_zero_is_identity(rope, d):
    rng = np.random.default_rng(1)
    k = rand_bits(rng, (7, d))
    out = oracle.stored_k(k, np.zeros(7, np.int64), rope)
    assert np.array_equal(out, k)


@pytest.mark.parametrize("d", [64, 128])
def test_1d_matches_roformer_library(d):
    """transformers' RoFormer rotary (interleaved pairs, base 10000) in float64."""
    from transformers.models.roformer.modeling_roformer import (
        RoFormerSinusoidalPositionalEmbedding, RoFormerSelfAttention)
    npos = 3000
    emb = RoFormerSinusoidalPositionalEmbedding(npos, d)
    w = emb.create_weight().to(torch.float64)          # [npos][d]: sin | cos halves
    rng = np.random.default_rng(2)
    pos = rng.integers(0, npos, 64)
    x = rand_bits(rng, (64, d))
    xf = torch.from_numpy(oracle.bf16_to_f64(x))
    sp = w[torch.from_numpy(pos)]
    ref, _ = RoFormerSelfAttention.apply_rotary_position_embeddings(
        sp, xf, xf.clone())
    ours = oracle.rotate_f64(x, pos, RopeSpec(ROPE_1D, (d, 0, 0)))
    ref = ref.numpy()
    # the library rounds its fp64 sin/cos to fp32 too; only the libm used may differ
    assert np.allclose(ours, ref, rtol=0, atol=1e-6 * np.abs(x).max())
    assert np.mean(ours == ref) > 0.99


def test_3d_slices_reduce_to_1d():
    """Each 3D axis slice is 1D RoPE (its own D_a) at that axis coordinate."""
    rng = np.random.default_rng(3)
    toks = np.array([0, 51, 52, 1559, 1560, 1613, 4679, 28080, 32759, 46799])
    x = rand_bits(rng, (len(toks), 128))
    y = oracle.rotate_f64(x, toks, R3D)
    t, rem = np.divmod(toks, 1560)
    h, w = np.divmod(rem, 52)
    for (lo, D, coord) in [(0, 44, t), (44, 42, h), (86, 42, w)]:
        ref = oracle.rotate_f64(x[:, lo:lo + D], coord, RopeSpec(ROPE_1D, (D, 0, 0)))
        assert np.array_equal(y[:, lo:lo + D], ref)


def test_3d_coordinates_golden():
    for line in golden_lines("rope3d_coords.txt"):
        tok, thw = line.split("->")
        tok = int(tok)
        expect = [int(v) for v in thw.split()]
        coords = [int(c[2]) for c in orope.rope_positions(R3D, np.array(tok))]
        assert coords == expect, (tok, coords, expect)


@pytest.mark.parametrize("rope,d", [(R1D128, 128), (R3D, 128)])
def test_norm_preserved_per_pair(rope, d):
    rng = np.random.default_rng(4)
    toks = rng.integers(0, 40000, 50)
    x = rand_bits(rng, (50, d))
    xf = oracle.bf16_to_f64(x)
    y = oracle.rotate_f64(x, toks, rope)
    n_in = xf[:, 0::2] ** 2 + xf[:, 1::2] ** 2
    n_out = y[:, 0::2] ** 2 + y[:, 1::2] ** 2
    # cos/sin are fp32-rounded: c^2 + s^2 = 1 within a few 2^-24
    assert np.all(np.abs(n_out - n_in) <= 4 * 2.0 ** -24 * n_in + 1e-300)


@pytest.mark.parametrize("rope", [R1D128, R3D])
def test_relative_position_property(rope):
    """rot(q,p).rot(k,t) depends on p - t only (up to table rounding)."""
    rng = np.random.default_rng(5)
    q = rand_bits(rng, (20, 128))
    k = rand_bits(rng, (20, 128))
    p = rng.integers(0, 2000, 20)
    t = rng.integers(0, 2000, 20)
    if rope.mode == ROPE_3D:
        shift = 1560 * 7          # whole frames: shifts t only, keeps (h, w)
    else:
        shift = 977
    a = np.sum(oracle.rotate_f64(q, p, rope) * oracle.rotate_f64(k, t, rope), axis=1)
    b = np.sum(oracle.rotate_f64(q, p + shift, rope) * oracle.rotate_f64(k, t + shift, rope), axis=1)
    scale = np.sum(np.abs(oracle.bf16_to_f64(q)) * np.abs(oracle.bf16_to_f64(k)), axis=1)
    assert np.all(np.abs(a - b) <= 1e-6 * scale)


def test_table_close_to_exact_cos_sin():
    pos = np.arange(0, 5000, 7)
    c, s = oracle.rope_cos_sin(128, 10000.0, pos)
    th = 10000.0 ** (-np.arange(64) * 2.0 / 128)
    ang = pos[:, None] * th[None, :]
    assert np.all(np.abs(c - np.cos(ang)) <= 2.0 ** -24 * 1.01)
    assert np.all(np.abs(s - np.sin(ang)) <= 2.0 ** -24 * 1.01)


def test_round_to_bf16_matches_torch_including_ties():
    rng = np.random.default_rng(6)
    y = rng.standard_normal(200000) * np.exp(rng.uniform(-20, 20, 200000))
    # exact fp32 ties for the bf16 step: low 16 bits == 0x8000
    t = rng.integers(0, 2 ** 31, 4096, dtype=np.uint64).astype(np.uint32)
    t = (t & np.uint32(0x7FFF0000)) | np.uint32(0x8000)
    t = t[(t >> 23) & 0xFF != 0xFF]
    ties = t.view(np.float32).astype(np.float64)
    y = np.concatenate([y, ties, -ties])
    ours = oracle.round_f64_to_bf16(y)
    ref = torch.from_numpy(y).to(torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_generator_bf16_rounding_is_rne():
    rng = np.random.default_rng(7)
    x = rng.standard_normal(100000).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(f32_to_bf16_bits(x), ref)


def test_rope_none_is_plain_decode():
    rng = np.random.default_rng(8)
    x = rand_bits(rng, (5, 64))
    assert np.array_equal(oracle.rotate_f64(x, np.arange(5) * 1000, RopeSpec(ROPE_NONE)),
                          oracle.bf16_to_f64(x))
