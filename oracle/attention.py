"""Masked attention over (pre-step ring) + (own chunk), float64 reference.

Test infrastructure only (see the package docstring). Parity pins:
tests/test_oracle_attention.py (uniform scores give the mean of V, a dominant
key gives its V row, masked keys have no influence, softmax rows sum to 1,
the worked softmax example in tests/golden/softmax_012.txt, agreement with
torch's scaled_dot_product_attention in float64 under an explicit mask, a
pure-Python loop twin on small cases, invariance to the ring's physical
rotation, GQA reduction to MHA).

Definition. For stream b with L = seq_len[b] before the step and query token
p = L + i (i < n), query head hq uses KV head hq // G (G = Hq / Hkv). Its key
set is every key token k that is present and visible:
    present: cached k in [max(0, L - C), L) (read from the ring) or own
             k in [L, L + n) (from the step's k_new / v_new);
    visible: block-causal (block Bc, window w blocks, 0 = unlimited):
                 k div Bc <= p div Bc  and  (w = 0 or p div Bc - k div Bc <= w)
             causal (window W keys including self, 0 = unlimited):
                 k <= p  and  (W = 0 or p - k < W)
Scores are s_k = (rot(q, p) . K_k) * scale with rot in float64 (q is not
rounded after rotation) and K_k the bf16 value the ring holds for k (for own
keys: the value the append will store, stored_k). Output
    O = sum_k softmax(s)_k V_k,  LSE = log sum_k exp(s_k)   (natural log)
evaluated in float64 with the row max subtracted. Attention only reads the
ring; the chunk is appended afterwards by kv_append.
"""
from __future__ import annotations

import math

import numpy as np

from .rope import bf16_to_f64, rotate_f64, stored_k
from .ring import RingState, slots_of_tokens

MASK_BLOCK_CAUSAL, MASK_CAUSAL = 1, 2


def visible(mask, p, k):
    """Boolean visibility of key token(s) k for query token(s) p (broadcasting)."""
    p = np.asarray(p, dtype=np.int64)
    k = np.asarray(k, dtype=np.int64)
    if mask.kind == MASK_BLOCK_CAUSAL:
        bp = p // mask.block
        bk = k // mask.block
        ok = bk <= bp
        if mask.window:
            ok = ok & (bp - bk <= mask.window)
        return ok
    if mask.kind == MASK_CAUSAL:
        ok = k <= p
        if mask.window:
            ok = ok & (p - k < mask.window)
        return ok
    raise ValueError("unknown mask kind %r" % (mask.kind,))


def attention_inputs(ring: RingState, b: int, kvh: int, k_new, v_new, rope):
    """Key tokens (logical order), K (float64), V (float64) visible-candidate set of one head.

    Cached tokens [max(0, L-C), L) then own tokens [L, L+n).
    """
    L = int(ring.seq_len[b])
    C = ring.C
    n = k_new.shape[1]
    cached = np.arange(max(0, L - C), L, dtype=np.int64)
    own = L + np.arange(n, dtype=np.int64)
    slots = slots_of_tokens(cached, C)
    k_c = bf16_to_f64(ring.k[b, kvh][slots])
    v_c = bf16_to_f64(ring.v[b, kvh][slots])
    k_o = bf16_to_f64(stored_k(k_new[b, :, kvh, :], own, rope))
    v_o = bf16_to_f64(v_new[b, :, kvh, :])
    return (np.concatenate([cached, own]), np.concatenate([k_c, k_o]),
            np.concatenate([v_c, v_o]))


def stream_attn(ring: RingState, q, k_new, v_new, rope, mask, scale=None,
                rows=None, row_block: int = 512, return_probs: bool = False):
    """Attention of one streaming step. Returns (out [B][n][Hq][d] f64, lse [B][Hq][n] f64).

    q: bf16 bits [B][n][Hq][d]; k_new, v_new: bf16 bits [B][n][Hkv][d].
    rows: optional sorted array of query indices i to evaluate (others are NaN).
    return_probs: also return {(b, hq): P [len(rows)][num_keys]} with key tokens.
    """
    B, n, Hq, d = q.shape
    Hkv = k_new.shape[2]
    G = Hq // Hkv
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(d)
    sel = np.arange(n, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.full((B, n, Hq, d), np.nan)
    lse = np.full((B, Hq, n), np.nan)
    probs = {}
    for b in range(B):
        L = int(ring.seq_len[b])
        ptok = L + sel
        for kvh in range(Hkv):
            ktok, K, V = attention_inputs(ring, b, kvh, k_new, v_new, rope)
            for g in range(G):
                hq = kvh * G + g
                qh = rotate_f64(q[b, sel, hq, :], ptok, rope)
                for r0 in range(0, len(sel), row_block):
                    r1 = min(len(sel), r0 + row_block)
                    s = (qh[r0:r1] @ K.T) * scale
                    vis = visible(mask, ptok[r0:r1, None], ktok[None, :])
                    s = np.where(vis, s, -np.inf)
                    m = s.max(axis=1, keepdims=True)
                    e = np.exp(s - m)
                    l = e.sum(axis=1, keepdims=True)
                    p = e / l
                    out[b, sel[r0:r1], hq, :] = p @ V
                    lse[b, hq, sel[r0:r1]] = (m + np.log(l))[:, 0]
                    if return_probs:
                        probs.setdefault((b, hq), []).append(p)
                if return_probs:
                    probs[(b, hq)] = (np.concatenate(probs[(b, hq)]), ktok)
    if return_probs:
        return out, lse, probs
    return out, lse


def decode_attn(ring: RingState, q, k_new, v_new, rope, mask, scale=None):
    """One-token decode step: the same definition with n = 1."""
    assert q.shape[1] == 1 and k_new.shape[1] == 1
    return stream_attn(ring, q, k_new, v_new, rope, mask, scale)
