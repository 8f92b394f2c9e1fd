"""Helpers for GPU parity tests: device transfer of bf16 bit arrays, ring setup
on both sides, tolerance checks. No method arithmetic lives here."""
import numpy as np
import torch

import oracle
import paper_2607_18171_amd as frt
from workloads import Workload, Case, make_case

# Tolerance for attention outputs (bf16 in, fp32 accumulate):
# max|err| <= 1e-2 * max|V| and mean|err| <= 1e-3.
MAX_ERR_REL_V = 1e-2
MEAN_ERR = 1e-3


def to_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def from_dev(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_dev_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def gpu_rope(wl: Workload, max_tokens: int) -> "frt.Rope":
    r = wl.rope
    return frt.Rope.for_tokens(r.mode, r.axis_dims, r.frame_hw, max_tokens, r.base)


def gpu_mask(wl: Workload):
    return frt.mask(wl.mask.kind, wl.mask.block, wl.mask.window)


def build_rings(case: Case, extra_tokens: int = 0):
    """Fill a GPU ring (through frt_kv_append) and an oracle ring with the case's prior tokens."""
    wl = case.wl
    max_tok = int(case.prior_lengths.max()) + wl.n + extra_tokens + 1
    rope = gpu_rope(wl, max_tok)
    ring = frt.Ring(wl.B, wl.Hkv, wl.d, wl.C)
    oring = oracle.new_ring(wl.B, wl.Hkv, wl.C, wl.d)
    for k, v in case.prior_steps:
        frt.kv_append(ring, rope, to_dev(k), to_dev(v))
        oring = oracle.kv_append(oring, k, v, wl.rope)
    for b, (k, v) in enumerate(case.prior_fills):
        if k.shape[1] == 0:
            continue
        n = k.shape[1]
        # appends of at most C tokens each
        for s in range(0, n, wl.C):
            e = min(n, s + wl.C)
            frt.kv_append(ring.view_stream(b), rope, to_dev(k[:, s:e]), to_dev(v[:, s:e]))
            oring = oracle.kv_append(oring, k[:, s:e], v[:, s:e], wl.rope, streams=[b])
    return ring, oring, rope


def ring_bytes_equal(ring: "frt.Ring", oring) -> bool:
    k = from_dev(ring.k)
    v = from_dev(ring.v_tokens())
    sl = ring.seq_len.cpu().numpy()
    return (np.array_equal(k, oring.k) and np.array_equal(v, oring.v)
            and np.array_equal(sl, oring.seq_len))


def visible_vmax(oring, case: Case) -> float:
    """max|V| over the V rows the step can see (ring tokens held + own tokens)."""
    vals = [np.abs(oracle.bf16_to_f64(case.v_new)).max()]
    for b in range(case.wl.B):
        L = int(oring.seq_len[b])
        held = min(L, case.wl.C)
        if held:
            slots = oracle.slots_of_tokens(np.arange(L - held, L), case.wl.C)
            vals.append(np.abs(oracle.bf16_to_f64(oring.v[b][:, slots])).max())
    return float(max(vals))


def check_close(got: np.ndarray, ref: np.ndarray, vmax: float, what: str = ""):
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got)), what + ": non-finite output"
    mx, mean = float(err.max()), float(err.mean())
    assert mx <= MAX_ERR_REL_V * vmax, "%s: max|err| %.3g > %.3g" % (what, mx, MAX_ERR_REL_V * vmax)
    assert mean <= MEAN_ERR, "%s: mean|err| %.3g > %.3g" % (what, mean, MEAN_ERR)
    return mx, mean
