"""The algorithmic work bench.py divides by: visible (query, key) pairs and
the minimum K/V bytes of a step, against a brute-force count with the
oracle's visibility rule and against the closed forms of the video steps."""
import dataclasses

import numpy as np
import pytest

import bench
from oracle.attention import visible
from workloads import WORKLOADS, MaskSpec, MASK_CAUSAL, MASK_BLOCK_CAUSAL


def brute_work(wl, lengths, kv_elem_bytes=2):
    """Count every visible pair of every stream, key by key."""
    pairs = 0
    kv_bytes = 0
    for L in lengths:
        L = int(L)
        keys = np.arange(max(0, L - wl.C), L + wl.n, dtype=np.int64)
        seen = np.zeros(keys.shape, dtype=bool)
        for i in range(wl.n):
            vis = visible(wl.mask, L + i, keys)
            pairs += int(vis.sum())
            seen |= vis
        kv_bytes += int(seen.sum()) * wl.Hkv * wl.d * 2 * kv_elem_bytes
    qo_bytes = 2 * wl.B * wl.n * wl.Hq * wl.d * 2
    return pairs * 4 * wl.d * wl.Hq, kv_bytes + qo_bytes


SMALL = [
    # block-causal, window 2 blocks, ring of 3 blocks (wrapped), chunk = block
    (dataclasses.replace(WORKLOADS["tiny"], n=16, C=48,
                         mask=MaskSpec(MASK_BLOCK_CAUSAL, 16, 2)), [0, 16, 80, 96]),
    # block-causal, blocks smaller than the chunk, unlimited window
    (dataclasses.replace(WORKLOADS["tiny"], n=24, C=64,
                         mask=MaskSpec(MASK_BLOCK_CAUSAL, 8, 0)), [0, 40, 64, 100]),
    # causal sliding window wider than the chunk, ring shorter than the window
    (dataclasses.replace(WORKLOADS["tiny"], n=20, C=40,
                         mask=MaskSpec(MASK_CAUSAL, 0, 50)), [0, 7, 39, 40, 123]),
    # causal, unlimited window, one query (decode shape)
    (dataclasses.replace(WORKLOADS["tiny"], n=1, C=32,
                         mask=MaskSpec(MASK_CAUSAL, 0, 0)), [0, 1, 31, 32, 77]),
]


@pytest.mark.parametrize("wl,lengths", SMALL)
@pytest.mark.parametrize("kv_elem_bytes", [2, 1])
def test_step_work_matches_brute_force(wl, lengths, kv_elem_bytes):
    assert bench.step_work(wl, lengths, kv_elem_bytes) == brute_work(wl, lengths, kv_elem_bytes)


def test_video_steps_closed_forms():
    # every query of the chunk sees the whole window: (window + 1) chunks
    for name, chunks in (("video_1p3b", 5), ("video_14b", 7)):
        wl = WORKLOADS[name]
        L = wl.prior_steps * wl.n
        flops, by = bench.step_work(wl, [L])
        assert flops == 4 * wl.d * wl.Hq * wl.n * chunks * wl.n
        assert by == chunks * wl.n * wl.Hkv * wl.d * 2 * 2 + 2 * wl.n * wl.Hq * wl.d * 2
    assert bench.step_work(WORKLOADS["video_1p3b"], [6 * 4680])[0] == 672_841_728_000
    assert bench.step_work(WORKLOADS["video_14b"], [9 * 4680])[0] == 3_139_928_064_000


def test_sliding_window_union_exceeds_one_query_range():
    # causal window W over an n-token chunk: the chunk reads W + n - 1 keys
    # once the stream is long enough, more than any single query's W
    wl = dataclasses.replace(WORKLOADS["prefill_swa"], B=1)
    L = 3 * wl.C
    _, by = bench.step_work(wl, [L])
    keys = wl.mask.window + wl.n - 1
    assert by == keys * wl.Hkv * wl.d * 2 * 2 + 2 * wl.n * wl.Hq * wl.d * 2
