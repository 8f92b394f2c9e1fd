"""Seeded synthetic inputs for chunk-streamed attention over ring-buffer KV caches.

This module only *draws* inputs: shapes, lengths and bf16 bit patterns. It
holds none of the method's arithmetic (no rotation, no attention, no ring
indexing), so both the fp64 oracle and the HIP path can consume the same
arrays without sharing any code that computes a result.

The five workloads stand in for the attention inputs of the streaming steps
the paper deploys (autoregressive video DiTs and multimodal LLMs; the paper
describes them as pipelines with persistent KV-cache state carried from batch
j-1 to batch j, Problem Formulation and App. "Pipeline graph"). The paper gives
no tensor dimensions, so the shapes are fixed here:

  tiny          B1, H2, d64, 16-token chunk after 48 cached tokens, ring of 64
  video_1p3b    B1, H12, d128, 3-frame chunks of 30x52 latents (4680 tokens),
                4 chunks cached in an 18720-slot ring, measured at step 6
  video_14b     B1, H40, d128, 4680-token chunks, 6 chunks cached in a
                28080-slot ring, measured at step 9, logits std ~3
  decode        32 streams x 1 token, GQA 32/4, per-stream context ~U[512,8192]
  prefill_swa   4 streams x 512-token chunk, GQA 32/8, cached ~U[0,16384],
                sliding window 8192 in an 8192-slot ring

Draw order for every workload (numpy.random.default_rng(seed)):
  1. lengths, if the workload has per-stream lengths;
  2. prior fill: for each prior step (or, for per-stream fills, each stream)
     k_raw then v_raw;
  3. the measured step: k_raw, v_raw, then q.
Each draw is rng.standard_normal(shape, float32) * scale, then rounded to
bf16 by round-to-nearest-even on the fp32 bit pattern.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

MASK_BLOCK_CAUSAL = 1
MASK_CAUSAL = 2
ROPE_NONE = 0
ROPE_1D = 1
ROPE_3D = 2


@dataclasses.dataclass(frozen=True)
class RopeSpec:
    mode: int                      # ROPE_NONE / ROPE_1D / ROPE_3D
    axis_dims: tuple = (0, 0, 0)   # 1D: (d,0,0); 3D: (44,42,42)
    frame_hw: tuple = (0, 0)       # 3D: latent frame (H, W)
    base: float = 10000.0


@dataclasses.dataclass(frozen=True)
class MaskSpec:
    kind: int      # MASK_BLOCK_CAUSAL or MASK_CAUSAL
    block: int     # block-causal: tokens per block (= chunk length)
    window: int    # block-causal: blocks (0 = unlimited); causal: keys incl. self (0 = unlimited)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    n: int                 # tokens per measured step
    C: int                 # ring slots per stream per KV head
    rope: RopeSpec
    mask: MaskSpec
    prior_steps: int = 0   # uniform prior steps of n tokens (video / tiny)
    len_lo: int = -1       # per-stream prior lengths ~ U{len_lo..len_hi}
    len_hi: int = -1
    qk_scale: float = 1.0  # Q and K drawn N(0,1)*qk_scale
    stagger: int = 0       # stream b holds prior_steps + stagger*(B-1-b) chunks
    description: str = ""

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def per_stream_lengths(self) -> bool:
        return self.len_lo >= 0 or self.stagger > 0


WORKLOADS = {
    "tiny": Workload(
        "tiny", B=1, Hq=2, Hkv=2, d=64, n=16, C=64,
        rope=RopeSpec(ROPE_1D, (64, 0, 0)),
        mask=MaskSpec(MASK_BLOCK_CAUSAL, 16, 0), prior_steps=3,
        description="B1 H2 d64, 16-token chunk after 48 cached, 64-slot ring"),
    "video_1p3b": Workload(
        "video_1p3b", B=1, Hq=12, Hkv=12, d=128, n=4680, C=18720,
        rope=RopeSpec(ROPE_3D, (44, 42, 42), (30, 52)),
        mask=MaskSpec(MASK_BLOCK_CAUSAL, 4680, 4), prior_steps=6,
        description="B1 H12 d128, 4680-token chunk vs 18720 cached + own, block-causal"),
    "video_14b": Workload(
        "video_14b", B=1, Hq=40, Hkv=40, d=128, n=4680, C=28080,
        rope=RopeSpec(ROPE_3D, (44, 42, 42), (30, 52)),
        mask=MaskSpec(MASK_BLOCK_CAUSAL, 4680, 6), prior_steps=9,
        qk_scale=float(np.sqrt(3.0)),
        description="B1 H40 d128, 4680-token chunk vs 28080 cached + own, wrapped ring"),
    "video_1p3b_pp4": Workload(
        "video_1p3b_pp4", B=4, Hq=12, Hkv=12, d=128, n=4680, C=18720,
        rope=RopeSpec(ROPE_3D, (44, 42, 42), (30, 52)),
        mask=MaskSpec(MASK_BLOCK_CAUSAL, 4680, 4), prior_steps=6, stagger=1,
        description="4 denoising-step caches of the 1.3B-like step as 4 streams, one "
                    "chunk apart (the stages of a step pipeline), one launch"),
    "decode": Workload(
        "decode", B=32, Hq=32, Hkv=4, d=128, n=1, C=8448,
        rope=RopeSpec(ROPE_1D, (128, 0, 0)),
        mask=MaskSpec(MASK_CAUSAL, 0, 0), len_lo=512, len_hi=8192,
        description="32 streams x 1 token, GQA 32/4, context ~U[512,8192]"),
    "prefill_swa": Workload(
        "prefill_swa", B=4, Hq=32, Hkv=8, d=128, n=512, C=8192,
        rope=RopeSpec(ROPE_1D, (128, 0, 0)),
        mask=MaskSpec(MASK_CAUSAL, 0, 8192), len_lo=0, len_hi=16384,
        description="4 streams x 512-token chunk, GQA 32/8, cached ~U[0,16384], window 8192"),
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest-even), returned as uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def draw_bf16(rng: np.random.Generator, shape, scale: float = 1.0) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        x = x * np.float32(scale)
    return f32_to_bf16_bits(x)


@dataclasses.dataclass
class Case:
    """One drawn instance of a workload. All tensors are bf16 bit patterns (uint16)."""
    wl: Workload
    seed: int
    prior_lengths: np.ndarray          # int64 [B]: tokens appended before the measured step
    # uniform prior steps: list of (k_raw [B][n][Hkv][d], v_raw) per step
    prior_steps: List[tuple]
    # per-stream prior fills: list over streams of (k_raw [1][n_b][Hkv][d], v_raw)
    prior_fills: List[tuple]
    k_new: np.ndarray                  # [B][n][Hkv][d]
    v_new: np.ndarray                  # [B][n][Hkv][d]
    q: np.ndarray                      # [B][n][Hq][d]


def make_case(wl, seed: int = 0, lengths: Optional[np.ndarray] = None) -> Case:
    """Draw a seeded instance of `wl` (a Workload or its name).

    `lengths` overrides the per-stream prior lengths (used by edge-case tests,
    e.g. a chunk that straddles the physical end of the ring).
    """
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    rng = np.random.default_rng(seed)
    s = wl.qk_scale
    if wl.per_stream_lengths:
        if wl.stagger > 0:
            drawn = np.array([(wl.prior_steps + wl.stagger * (wl.B - 1 - b)) * wl.n
                              for b in range(wl.B)], dtype=np.int64)
        else:
            drawn = rng.integers(wl.len_lo, wl.len_hi, wl.B, endpoint=True).astype(np.int64)
        if lengths is not None:
            drawn = np.asarray(lengths, dtype=np.int64)
        fills = []
        for b in range(wl.B):
            nb = int(drawn[b])
            fills.append((draw_bf16(rng, (1, nb, wl.Hkv, wl.d), s),
                          draw_bf16(rng, (1, nb, wl.Hkv, wl.d))))
        prior = drawn
        steps = []
    else:
        steps = []
        for _ in range(wl.prior_steps):
            steps.append((draw_bf16(rng, (wl.B, wl.n, wl.Hkv, wl.d), s),
                          draw_bf16(rng, (wl.B, wl.n, wl.Hkv, wl.d))))
        prior = np.full(wl.B, wl.prior_steps * wl.n, dtype=np.int64)
        fills = []
    k_new = draw_bf16(rng, (wl.B, wl.n, wl.Hkv, wl.d), s)
    v_new = draw_bf16(rng, (wl.B, wl.n, wl.Hkv, wl.d))
    q = draw_bf16(rng, (wl.B, wl.n, wl.Hq, wl.d), s)
    return Case(wl, seed, prior, steps, fills, k_new, v_new, q)




def shrink(wl: Workload, **kw) -> Workload:
    """A copy of `wl` with some fields replaced (small parity variants)."""
    return dataclasses.replace(wl, **kw)
