"""Rotary position embedding and bf16 rounding, float64 reference.

Test infrastructure only (see the package docstring). Parity pins:
tests/test_oracle_rope.py (identity at position 0, recovered rotation angles
and their geometric frequency ladder, interleaved pairing, 3D axis split,
relative-position property, agreement with the RoFormer implementation in
`transformers`).

Definition (RoFormer, Su et al. 2021, pairwise rotation form): for a head
vector x of length D and a position p, pair i (coordinates 2i and 2i+1) is
rotated by angle p * theta_i with theta_i = base^(-2i/D):
    y[2i]   = x[2i] cos(p theta_i) - x[2i+1] sin(p theta_i)
    y[2i+1] = x[2i] sin(p theta_i) + x[2i+1] cos(p theta_i)
The 3D form splits the head dimension into consecutive axis slices of sizes
(D_t, D_h, D_w) and rotates slice a with its own D_a by that axis coordinate
of the token: (t, h, w) = (p div (H*W), (p mod (H*W)) div W, p mod W) for a
latent frame of H x W tokens in raster order.

cos and sin are evaluated in float64 by the C library (`math.cos`,
`math.sin`) and rounded to float32 (the table precision). The rotation is then
done in float64: each product of a bf16 value (8 significant bits) and a
float32 table value (24 bits) is exact in float64, so the only rounding is the
final add/subtract. Stored keys are rounded float64 -> float32 -> bf16, each
step round-to-nearest-even.
"""
from __future__ import annotations

import math
from functools import lru_cache

import numpy as np

ROPE_NONE, ROPE_1D, ROPE_3D = 0, 1, 2


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64 (exact: bf16 -> fp32 is a 16-bit shift)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def round_f64_to_bf16(y: np.ndarray) -> np.ndarray:
    """float64 -> float32 (IEEE round-to-nearest-even) -> bf16 (RNE on the bits).

    Inputs are finite. Returns uint16 bit patterns.
    """
    f = np.asarray(y, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


@lru_cache(maxsize=64)
def _axis_table(axis_dim: int, base: float, npos: int):
    """cos/sin (float32) for positions 0..npos-1 and pairs 0..axis_dim/2-1."""
    npairs = axis_dim // 2
    thetas = [math.pow(base, -(2.0 * i) / axis_dim) for i in range(npairs)]
    cos = np.empty((npos, npairs), dtype=np.float32)
    sin = np.empty((npos, npairs), dtype=np.float32)
    for p in range(npos):
        cos[p] = [math.cos(p * th) for th in thetas]
        sin[p] = [math.sin(p * th) for th in thetas]
    cos.flags.writeable = False
    sin.flags.writeable = False
    return cos, sin


def rope_cos_sin(axis_dim: int, base: float, positions: np.ndarray):
    """Float32 cos/sin of positions * theta_i, shapes [len(positions)][axis_dim/2]."""
    positions = np.asarray(positions, dtype=np.int64)
    if positions.size == 0:
        z = np.zeros((0, axis_dim // 2), dtype=np.float32)
        return z, z
    npos = int(positions.max()) + 1
    cos, sin = _axis_table(int(axis_dim), float(base), npos)
    return cos[positions], sin[positions]


def rope_positions(rope, tokens: np.ndarray):
    """Per-axis coordinates of token indices: list of (slice_start, D_a, coords)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    if rope.mode == ROPE_1D:
        return [(0, rope.axis_dims[0], tokens)]
    if rope.mode == ROPE_3D:
        fh, fw = rope.frame_hw
        per_frame = fh * fw
        t = tokens // per_frame
        h = (tokens % per_frame) // fw
        w = tokens % fw
        dt, dh, dw = rope.axis_dims
        return [(0, dt, t), (dt, dh, h), (dt + dh, dw, w)]
    return []


def rotate_f64(x_bits: np.ndarray, tokens: np.ndarray, rope) -> np.ndarray:
    """Rotate bf16 vectors x_bits[..., N, D] at token indices tokens[N]; float64 result.

    Leading dimensions broadcast; `tokens` indexes the second-to-last axis.
    Coordinates outside every axis slice are returned unchanged.
    """
    x = bf16_to_f64(x_bits)
    if rope.mode == ROPE_NONE:
        return x
    y = x.copy()
    for start, dim, coord in rope_positions(rope, tokens):
        c, s = rope_cos_sin(dim, rope.base, coord)
        c = c.astype(np.float64)
        s = s.astype(np.float64)
        x0 = x[..., start:start + dim:2]
        x1 = x[..., start + 1:start + dim:2]
        y[..., start:start + dim:2] = x0 * c - x1 * s
        y[..., start + 1:start + dim:2] = x0 * s + x1 * c
    return y


def stored_k(k_bits: np.ndarray, tokens: np.ndarray, rope) -> np.ndarray:
    """The bf16 bits a ring slot holds for raw key k at token index `tokens`."""
    return round_f64_to_bf16(rotate_f64(k_bits, tokens, rope))
