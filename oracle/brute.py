"""Pure-Python loop twins of the oracle for tiny inputs.

Test infrastructure only (see the package docstring). These are written
directly from the definitions (RoFormer pair rotation, textbook softmax
attention, token t in slot t mod C) with Python floats and integers and no
numpy arithmetic, so that tests can pin the vectorised oracle against an
implementation that shares none of its code. Used by
tests/test_oracle_brute.py on small cases only.
"""
from __future__ import annotations

import math
import struct


def f32(x: float) -> float:
    """Round a Python float (binary64) to binary32, nearest-even."""
    return struct.unpack("<f", struct.pack("<f", x))[0]


def bf16_from_float(x: float) -> int:
    """binary64 -> binary32 (RNE) -> bf16 (RNE) bit pattern."""
    u = struct.unpack("<I", struct.pack("<f", x))[0]
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u & 0xFFFF


def bf16_value(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def axis_coords(rope, token: int):
    """[(slice_start, D_a, coordinate)] for one token."""
    if rope.mode == 1:
        return [(0, rope.axis_dims[0], token)]
    if rope.mode == 2:
        fh, fw = rope.frame_hw
        t, rem = divmod(token, fh * fw)
        h, w = divmod(rem, fw)
        dt, dh, dw = rope.axis_dims
        return [(0, dt, t), (dt, dh, h), (dt + dh, dw, w)]
    return []


def rotate(vec_bits, token: int, rope):
    """Rotate one bf16 vector (list of bit patterns); returns list of Python floats."""
    x = [bf16_value(b) for b in vec_bits]
    y = list(x)
    for start, dim, pos in axis_coords(rope, token):
        for i in range(dim // 2):
            theta = math.pow(rope.base, -(2.0 * i) / dim)
            c = f32(math.cos(pos * theta))
            s = f32(math.sin(pos * theta))
            a, b = x[start + 2 * i], x[start + 2 * i + 1]
            y[start + 2 * i] = a * c - b * s
            y[start + 2 * i + 1] = a * s + b * c
    return y


class ListRing:
    """A ring as a Python list of slots, each slot a dict head -> (token, k_bits, v_bits)."""

    def __init__(self, B, Hkv, C, d):
        self.B, self.Hkv, self.C, self.d = B, Hkv, C, d
        self.slots = [[[None] * C for _ in range(Hkv)] for _ in range(B)]
        self.seq_len = [0] * B

    def append(self, k_new, v_new, rope):
        """k_new, v_new: nested lists [B][n][Hkv][d] of bf16 bit patterns."""
        for b in range(self.B):
            L = self.seq_len[b]
            for i in range(len(k_new[b])):
                tok = L + i
                slot = tok % self.C
                for h in range(self.Hkv):
                    kb = [bf16_from_float(v) for v in rotate(k_new[b][i][h], tok, rope)]
                    self.slots[b][h][slot] = (tok, kb, list(v_new[b][i][h]))
            self.seq_len[b] = L + len(k_new[b])

    def present(self, b, h):
        """[(token, k_bits, v_bits)] for tokens still held, any order."""
        return [e for e in self.slots[b][h] if e is not None]


def is_visible(mask, p: int, k: int) -> bool:
    if mask.kind == 1:
        bp, bk = p // mask.block, k // mask.block
        return bk <= bp and (mask.window == 0 or bp - bk <= mask.window)
    return k <= p and (mask.window == 0 or p - k < mask.window)


def attend(ring: ListRing, q, k_new, v_new, rope, mask, Hq, scale=None):
    """Loop attention. q: nested [B][n][Hq][d]; returns out [B][n][Hq][d] floats."""
    Hkv = ring.Hkv
    G = Hq // Hkv
    d = ring.d
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = []
    for b in range(ring.B):
        L = ring.seq_len[b]
        n = len(q[b])
        rows = []
        for i in range(n):
            p = L + i
            heads = []
            for hq in range(Hq):
                h = hq // G
                keys = []
                for tok, kb, vb in ring.present(b, h):
                    keys.append((tok, [bf16_value(x) for x in kb], [bf16_value(x) for x in vb]))
                for j in range(n):
                    tok = L + j
                    kb = [bf16_from_float(v) for v in rotate(k_new[b][j][h], tok, rope)]
                    keys.append((tok, [bf16_value(x) for x in kb],
                                 [bf16_value(x) for x in v_new[b][j][h]]))
                qv = rotate(q[b][i][hq], p, rope)
                scores = []
                for tok, kv, vv in keys:
                    if is_visible(mask, p, tok):
                        scores.append((sum(qv[t] * kv[t] for t in range(d)) * scale, vv))
                m = max(s for s, _ in scores)
                w = [math.exp(s - m) for s, _ in scores]
                tot = sum(w)
                o = [0.0] * d
                for wk, (_, vv) in zip(w, scores):
                    for t in range(d):
                        o[t] += wk * vv[t]
                heads.append([x / tot for x in o])
            rows.append(heads)
        out.append(rows)
    return out
