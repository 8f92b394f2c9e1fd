"""Pins for the oracle's ring-buffer append and slot map (CPU only)."""
import numpy as np
import pytest

import oracle
from oracle import brute
from workloads import RopeSpec, ROPE_1D, ROPE_3D
from _helpers import golden_lines, rand_bits

R1D = RopeSpec(ROPE_1D, (16, 0, 0))
R3D_SMALL = RopeSpec(ROPE_3D, (8, 4, 4), (2, 3))


def test_slot_golden():
    for line in golden_lines("ring_slots.txt"):
        if "->" in line:
            lhs, rhs = line.split("->")
            C, L, n = (int(v) for v in lhs.split())
            expect = [int(v) for v in rhs.split()]
            got = oracle.slots_of_tokens(L + np.arange(n), C).tolist()
            assert got == expect, line
        else:
            lhs, rhs = line.split("=>")
            C, L, s = (int(v) for v in lhs.split())
            assert int(oracle.slot_token(L, s, C)) == int(rhs), line


def _to_lists(a):
    return a.tolist()


@pytest.mark.parametrize("rope", [R1D, R3D_SMALL])
@pytest.mark.parametrize("C,chunks", [(12, [5, 5, 5, 3, 12, 1]), (8, [8, 8, 3, 7]), (20, [4, 4])])
def test_append_matches_list_model(rope, C, chunks):
    B, Hkv, d = 2, 2, 16
    rng = np.random.default_rng(10 + C)
    ring = oracle.new_ring(B, Hkv, C, d)
    model = brute.ListRing(B, Hkv, C, d)
    for n in chunks:
        k = rand_bits(rng, (B, n, Hkv, d))
        v = rand_bits(rng, (B, n, Hkv, d))
        ring = oracle.kv_append(ring, k, v, rope)
        model.append(_to_lists(k), _to_lists(v), rope)
        assert ring.seq_len.tolist() == model.seq_len
        for b in range(B):
            for h in range(Hkv):
                for s in range(C):
                    e = model.slots[b][h][s]
                    if e is None:
                        assert not ring.k[b, h, s].any() and not ring.v[b, h, s].any()
                        assert oracle.slot_token(int(ring.seq_len[b]), s, C) < 0
                        continue
                    tok, kb, vb = e
                    assert int(oracle.slot_token(int(ring.seq_len[b]), s, C)) == tok
                    assert ring.k[b, h, s].tolist() == kb
                    assert ring.v[b, h, s].tolist() == vb


def test_untouched_slots_and_v_bytes():
    B, Hkv, C, d, n = 1, 3, 64, 16, 10
    rng = np.random.default_rng(11)
    ring = oracle.new_ring(B, Hkv, C, d)
    ring.k[:] = rand_bits(rng, ring.k.shape)
    ring.v[:] = rand_bits(rng, ring.v.shape)
    ring.seq_len[:] = 60
    k = rand_bits(rng, (B, n, Hkv, d))
    v = rand_bits(rng, (B, n, Hkv, d))
    out = oracle.kv_append(ring, k, v, R1D)
    written = oracle.slots_of_tokens(60 + np.arange(n), C)
    other = np.setdiff1d(np.arange(C), written)
    assert np.array_equal(out.k[:, :, other], ring.k[:, :, other])
    assert np.array_equal(out.v[:, :, other], ring.v[:, :, other])
    assert np.array_equal(out.v[0][:, written, :], np.transpose(v[0], (1, 0, 2)))
    assert out.seq_len[0] == 70


def test_full_ring_rewrite():
    B, Hkv, C, d = 1, 1, 16, 16
    rng = np.random.default_rng(12)
    ring = oracle.new_ring(B, Hkv, C, d)
    ring.seq_len[:] = 5
    k = rand_bits(rng, (B, C, Hkv, d))
    v = rand_bits(rng, (B, C, Hkv, d))
    out = oracle.kv_append(ring, k, v, R1D)
    toks = 5 + np.arange(C)
    assert np.array_equal(out.v[0, 0][toks % C], v[0, :, 0])
    assert np.array_equal(out.k[0, 0][toks % C], oracle.stored_k(k[0, :, 0], toks, R1D))
