"""Ring-buffer KV cache state and append, reference model.

Test infrastructure only (see the package docstring). Parity pins:
tests/test_oracle_ring.py (a list-of-slots model written independently, the
worked slot examples in tests/golden/ring_slots.txt, untouched-slot and
byte-copy invariants).

The persistent state of one stream is what the paper calls state inherited
across batches (Problem Formulation: lambda=1 edges, whose example is an
attention key/value cache carried from one batch to the next; Chain-of-Program,
IR design: a node's persistent state reads and writes). Here that state is, per stream b and KV head h, C
slots of K and V plus a counter seq_len[b] of tokens ever appended. Token t
lives in slot t mod C, so slot s holds token
    k(s) = L - 1 - ((L - 1 - s) mod C)       (L = seq_len, mod non-negative)
which is a real token iff L >= 1 and k(s) >= 0. The tokens still present are
[max(0, L - C), L).

Appending n tokens writes, for i < n, K = stored_k(k_new[i], L + i) and
V = v_new[i] (bytes copied) into slot (L + i) mod C, then sets seq_len = L + n.
Slots not written keep their bytes. The append requires n <= C.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .rope import stored_k


@dataclasses.dataclass
class RingState:
    k: np.ndarray        # uint16 bf16 bits [B][Hkv][C][d]  (logical layout: slot-major)
    v: np.ndarray        # uint16 bf16 bits [B][Hkv][C][d]
    seq_len: np.ndarray  # int64 [B]

    @property
    def C(self) -> int:
        return self.k.shape[2]

    def copy(self) -> "RingState":
        return RingState(self.k.copy(), self.v.copy(), self.seq_len.copy())


def new_ring(B: int, Hkv: int, C: int, d: int) -> RingState:
    """A zero-filled ring with no tokens (never-written slots hold +0.0)."""
    return RingState(np.zeros((B, Hkv, C, d), np.uint16),
                     np.zeros((B, Hkv, C, d), np.uint16),
                     np.zeros(B, np.int64))


def slot_token(L: int, s, C: int):
    """Token index held by slot s when seq_len = L (negative: never written)."""
    s = np.asarray(s, dtype=np.int64)
    return L - 1 - np.mod(L - 1 - s, C)


def slots_of_tokens(tokens, C: int):
    return np.mod(np.asarray(tokens, dtype=np.int64), C)


def kv_append(ring: RingState, k_new: np.ndarray, v_new: np.ndarray, rope,
              streams=None) -> RingState:
    """Append k_new/v_new [B][n][Hkv][d] (bf16 bits) to every stream; returns a new state.

    `streams` optionally restricts the append to a subset of streams (their
    rows of k_new/v_new are used in order).
    """
    out = ring.copy()
    B = ring.k.shape[0]
    C = ring.C
    idx = list(range(B)) if streams is None else list(streams)
    n = k_new.shape[1]
    assert n <= C, "an append of more than C tokens would overwrite its own tokens"
    for row, b in enumerate(idx):
        L = int(ring.seq_len[b])
        tokens = L + np.arange(n, dtype=np.int64)
        slots = slots_of_tokens(tokens, C)
        # k_new[row]: [n][Hkv][d] -> per head [n][d]
        kh = np.transpose(k_new[row], (1, 0, 2))
        vh = np.transpose(v_new[row], (1, 0, 2))
        out.k[b][:, slots, :] = stored_k(kh, tokens, rope)
        out.v[b][:, slots, :] = vh
        out.seq_len[b] = L + n
    return out
