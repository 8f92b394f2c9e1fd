"""FP8 (OCP e4m3fn) variant of the streaming step, reference model.

Test infrastructure only (see the package docstring). This is the FP8 KV
cache / FP8 QK^T-PV variant of the step: the same attention, with the ring
holding 8-bit codes and the two contractions taking 8-bit operands. The paper
fixes no low-precision arithmetic, so everything below is a stated reading,
listed with the others in the design notes:

  * format: e4m3fn (1 sign, 4 exponent bits with bias 7, 3 mantissa bits,
    subnormals at exponent field 0, no infinities, 0x7f / 0xff are NaN,
    largest finite 448);
  * rounding to the format: to nearest, ties to the even code, after
    clamping to [-448, 448];
  * ring contents: K8 = q8(fp32(rot(k)) / s_k) and V8 = q8(v / s_v), with
    per-(stream, KV head) fp32 scales s_k, s_v given by the caller and the
    division done in fp32;
  * queries: a = fp32(rot(q) * scale * log2(e)) (the base-2 score units of
    the bf16 path), quantised per query row with a power-of-two scale 2^e,
    e the smallest integer with max|a| <= 448 * 2^e;
  * scores s = 2^e * s_k * (q8 . k8) in base-2 units; with m the smallest
    integer >= the row's largest visible score, the weights are
    p = q8(2^(s - m + 7)) and out = s_v * sum(p * v8) / sum(p), so the sum
    and the product use the same quantised weights. The factor 2^7 puts the
    largest weight in [64, 128] and the first subnormal code 2^-13 below it:
    a row whose softmax mass is spread (3x unit logits over tens of
    thousands of keys leave the top key a few percent of it) keeps that mass
    in normal codes instead of flushing it to zero.

Pins: tests/test_oracle_fp8.py (every code against the format's definition,
rounding ties, the closed forms of uniform and one-hot attention, and the
bf16 oracle on inputs the format represents exactly).
"""
from __future__ import annotations

import math

import numpy as np

from .rope import rotate_f64, bf16_to_f64
from .ring import slots_of_tokens
from .attention import visible

E4M3_MAX = 448.0
P_SHIFT = 7  # weights are coded at 2^P_SHIFT times their ratio to 2^m


def e4m3_value(code: int) -> float:
    """The real number an e4m3fn code stands for (NaN for 0x7f / 0xff)."""
    code = int(code) & 0xff
    sign = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xf
    m = code & 0x7
    if e == 0xf and m == 0x7:
        return math.nan
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** -6
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


_DECODE = np.array([e4m3_value(c) for c in range(256)], dtype=np.float64)
# the 127 finite non-negative values in increasing order with their codes
_POS_CODES = np.arange(0x00, 0x7f, dtype=np.int64)
_POS_VALS = _DECODE[_POS_CODES]


def e4m3_decode(codes) -> np.ndarray:
    return _DECODE[np.asarray(codes, dtype=np.uint8)]


def e4m3_encode(x) -> np.ndarray:
    """float64 values -> e4m3fn codes: clamp to +-448, round to nearest, ties
    to the even code (codes are in value order, so even code = even mantissa);
    the sign bit is the input's, zero included."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    hi = np.searchsorted(_POS_VALS, a, side="left")        # first value >= a
    hi = np.minimum(hi, len(_POS_VALS) - 1)
    lo = np.maximum(hi - 1, 0)
    dlo = a - _POS_VALS[lo]
    dhi = _POS_VALS[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (_POS_CODES[hi] % 2 == 0) & (hi != lo))
    code = np.where(pick_hi, _POS_CODES[hi], _POS_CODES[lo])
    code = np.where(a == _POS_VALS[hi], _POS_CODES[hi], code)
    # the sign is kept, also when the magnitude rounds to zero (-0 is 0x80)
    return (code | np.where(np.signbit(x), 0x80, 0)).astype(np.uint8)


def quantize(x_f32, scale) -> np.ndarray:
    """q8(x / s): the division in fp32 (IEEE, round to nearest), then e4m3."""
    xf = np.asarray(x_f32, dtype=np.float32)
    s = np.asarray(scale, dtype=np.float32)
    return e4m3_encode((xf / s).astype(np.float64))


def pow2_row_exponent(a_f32) -> np.ndarray:
    """Smallest integer e with max|a| <= 448 * 2^e per row (last axis); 0 for a zero row."""
    m = np.max(np.abs(np.asarray(a_f32, dtype=np.float64)), axis=-1)
    e = np.zeros(m.shape, dtype=np.int64)
    nz = m > 0
    e[nz] = np.ceil(np.log2(m[nz] / E4M3_MAX)).astype(np.int64)
    # log2 rounding guard: step e to the exact smallest value
    e = np.where(nz & (m > E4M3_MAX * np.exp2(e.astype(np.float64))), e + 1, e)
    e = np.where(nz & (m <= E4M3_MAX * np.exp2(e.astype(np.float64) - 1)), e - 1, e)
    return e


class RingFP8:
    """Ring of e4m3 codes: k, v uint8 [B][Hkv][C][d] (slot-major), seq_len int64 [B]."""

    def __init__(self, B, Hkv, C, d):
        self.k = np.zeros((B, Hkv, C, d), np.uint8)
        self.v = np.zeros((B, Hkv, C, d), np.uint8)
        self.seq_len = np.zeros(B, np.int64)

    @property
    def C(self):
        return self.k.shape[2]


def stored_k8(k_bits, tokens, rope, s_k) -> np.ndarray:
    """Codes a slot holds for raw bf16 key k at token indices `tokens`."""
    return quantize(rotate_f64(k_bits, tokens, rope).astype(np.float32), s_k)


def stored_v8(v_bits, s_v) -> np.ndarray:
    return quantize(bf16_to_f64(v_bits).astype(np.float32), s_v)


def kv_append_fp8(ring: RingFP8, k_new, v_new, rope, k_scale, v_scale, streams=None):
    """Append k_new / v_new (bf16 bits [B][n][Hkv][d]) to the FP8 ring, in place.

    k_scale, v_scale: fp32 [B][Hkv] for the whole ring (indexed by stream)."""
    B = ring.k.shape[0]
    sel = list(range(B)) if streams is None else list(streams)
    n = k_new.shape[1]
    assert n <= ring.C
    for row, b in enumerate(sel):
        L = int(ring.seq_len[b])
        toks = L + np.arange(n, dtype=np.int64)
        slots = slots_of_tokens(toks, ring.C)
        for h in range(ring.k.shape[1]):
            ring.k[b, h, slots] = stored_k8(k_new[row, :, h, :], toks, rope, k_scale[b, h])
            ring.v[b, h, slots] = stored_v8(v_new[row, :, h, :], v_scale[b, h])
        ring.seq_len[b] = L + n
    return ring


def query_codes(q_bits, tokens, rope, scale):
    """(codes [N][d], e [N]) of rotated queries in base-2 score units."""
    mul = scale * math.log2(math.e)
    a = (rotate_f64(q_bits, tokens, rope) * mul).astype(np.float32)
    e = pow2_row_exponent(a)
    scaled = a.astype(np.float64) * np.exp2(-e.astype(np.float64))[..., None]
    return e4m3_encode(scaled), e


def stream_attn_fp8(ring: RingFP8, q, k_new, v_new, rope, mask, k_scale, v_scale,
                    scale=None, rows=None):
    """FP8 step attention. Returns (out [B][n][Hq][d] f64, lse [B][Hq][n] f64).

    Reads the pre-step ring plus the chunk's own keys and values quantised as
    the append stores them."""
    B, n, Hq, d = q.shape
    Hkv = k_new.shape[2]
    G = Hq // Hkv
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(d)
    sel = np.arange(n, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.full((B, n, Hq, d), np.nan)
    lse = np.full((B, Hq, n), np.nan)
    for b in range(B):
        L = int(ring.seq_len[b])
        C = ring.C
        cached = np.arange(max(0, L - C), L, dtype=np.int64)
        own = L + np.arange(n, dtype=np.int64)
        ktok = np.concatenate([cached, own])
        ptok = L + sel
        for kvh in range(Hkv):
            sk = float(np.float32(k_scale[b, kvh]))
            sv = float(np.float32(v_scale[b, kvh]))
            slots = slots_of_tokens(cached, C)
            K = np.concatenate([e4m3_decode(ring.k[b, kvh][slots]),
                                e4m3_decode(stored_k8(k_new[b, :, kvh, :], own, rope, sk))])
            V = np.concatenate([e4m3_decode(ring.v[b, kvh][slots]),
                                e4m3_decode(stored_v8(v_new[b, :, kvh, :], sv))])
            for g in range(G):
                hq = kvh * G + g
                q8, e = query_codes(q[b, sel, hq, :], ptok, rope, scale)
                s = (e4m3_decode(q8) @ K.T) * (np.exp2(e.astype(np.float64))[:, None] * sk)
                vis = visible(mask, ptok[:, None], ktok[None, :])
                s = np.where(vis, s, -np.inf)
                m = np.ceil(s.max(axis=1, keepdims=True))
                p = e4m3_decode(e4m3_encode(np.exp2(s - m + P_SHIFT)))
                l = p.sum(axis=1, keepdims=True)
                out[b, sel, hq, :] = sv * (p @ V) / l
                lse[b, hq, sel] = ((m - P_SHIFT + np.log2(l)) * math.log(2.0))[:, 0]
    return out, lse
