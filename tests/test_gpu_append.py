"""frt_kv_append on the GPU: ring bytes and seq_len bit-exact against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_18171_amd as frt
from workloads import (WORKLOADS, RopeSpec, MaskSpec, ROPE_1D, ROPE_3D, ROPE_NONE,
                       MASK_CAUSAL, make_case, shrink, draw_bf16)
from gpu_helpers import to_dev, from_dev, build_rings, ring_bytes_equal, gpu_rope

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "video_1p3b", "decode"])
def test_workload_fill_bit_exact(name):
    case = make_case(name, 0)
    ring, oring, rope = build_rings(case)
    torch.cuda.synchronize()
    assert ring_bytes_equal(ring, oring)
    # then append the measured chunk
    frt.kv_append(ring, rope, to_dev(case.k_new), to_dev(case.v_new))
    oring = oracle.kv_append(oring, case.k_new, case.v_new, case.wl.rope)
    torch.cuda.synchronize()
    assert ring_bytes_equal(ring, oring)


@pytest.mark.parametrize("rope,d", [
    (RopeSpec(ROPE_1D, (64, 0, 0)), 64),
    (RopeSpec(ROPE_1D, (96, 0, 0)), 128),          # pairs beyond the rotated slice pass through
    (RopeSpec(ROPE_3D, (44, 42, 42), (4, 6)), 128),
    (RopeSpec(ROPE_NONE), 128),
])
@pytest.mark.parametrize("C,chunks", [(56, [16, 16, 16, 16, 16]), (64, [64, 64, 1, 63]),
                                      (72, [70, 5, 1, 1, 72])])
def test_append_sequences_wrap_and_straddle(rope, d, C, chunks):
    B, Hkv = 3, 2
    rng = np.random.default_rng(C + d)
    total = sum(chunks) + 1
    if rope.mode == ROPE_3D:
        fh, fw = rope.frame_hw
        max_pos = ((total + fh * fw - 1) // (fh * fw), fh, fw)
    else:
        max_pos = (total, 0, 0)
    grope = frt.Rope(rope.mode, rope.axis_dims, rope.frame_hw, max_pos, rope.base)
    ring = frt.Ring(B, Hkv, d, C)
    oring = oracle.new_ring(B, Hkv, C, d)
    for n in chunks:
        k = draw_bf16(rng, (B, n, Hkv, d))
        v = draw_bf16(rng, (B, n, Hkv, d))
        frt.kv_append(ring, grope, to_dev(k), to_dev(v))
        oring = oracle.kv_append(oring, k, v, rope)
        torch.cuda.synchronize()
        assert ring_bytes_equal(ring, oring), (C, n)


def test_prefill_chunk_straddles_ring_end():
    """A 512-token chunk at L = 8000 in an 8192-slot ring crosses the physical end."""
    wl = WORKLOADS["prefill_swa"]
    case = make_case(wl, 1, lengths=np.array([8000, 100, 16384, 0]))
    ring, oring, rope = build_rings(case)
    frt.kv_append(ring, rope, to_dev(case.k_new), to_dev(case.v_new))
    oring = oracle.kv_append(oring, case.k_new, case.v_new, wl.rope)
    torch.cuda.synchronize()
    assert ring_bytes_equal(ring, oring)


def test_rope_table_matches_oracle_cos_sin():
    """The library's fp32 cos/sin table equals the oracle's, bit for bit (same libm)."""
    r = frt.Rope(ROPE_3D, (44, 42, 42), (30, 52), (31, 30, 52))
    tab = r.host_table.numpy()
    off = 0
    for D, npos in ((44, 31), (42, 30), (42, 52)):
        c, s = oracle.rope_cos_sin(D, 10000.0, np.arange(npos))
        blk = tab[off:off + npos * (D // 2) * 2].reshape(npos, D // 2, 2)
        assert np.array_equal(blk[..., 0], c) and np.array_equal(blk[..., 1], s)
        off += npos * (D // 2) * 2
