"""Benchmark one streaming step of chunk-streamed attention on one MI355X.

A step is the whole hot path for one batch: frt_stream_step (chunk
preparation, attention, and the append of the prepared chunk), or for the
decode workload frt_decode_step (split + combine, the combine also appending
the token). The default workload is the 14B-like video step, the largest
configuration of the video-step target that fits one GPU.
Inputs are seeded synthetic bf16 tensors already resident in HBM; the ring is
pre-filled through the library's own append so the measured steps see a
wrapped ring. With --rings R > 1 the steps rotate over R copies of the ring
(separate buffers, same contents), so that the 256 MB Infinity Cache cannot
serve a step's reads from the previous step; the decode workload does this by
default (R = 3) and also reports the same steps on one ring ("hot").

Prints one JSON line. `value` is attention TFLOP/s per step (algorithmic
flops: 4*d per visible (query, key) pair, no credit for masked or padded
work) or, for decode, HBM GB/s per step (each visible K/V byte once plus
q/out), over K plain steps. `roofline` reports the dominant kernel against
MI355X's published peaks, its duration taken with HIP events on the kernel's
own dispatch over K further steps (mean, and the 10th/50th/90th percentiles
of the launches); the events themselves lengthen a step, so they are kept out
of the throughput region. With --graph, `graph` times the same steps
replayed from one HIP graph (no host launch cost between them).
`cpu_baseline` times the fp64 oracle on a bounded sample of the same step. `clock_power` is the graphics
clock and socket power amd-smi reads while the attention repeats (the part
runs at its power limit under this load, so the clock differs between
parts), and `library` times the vendor libraries and two probes on the same
part: a 1 GiB device copy; for the chunk steps torch's fused attention, a
hipBLASLt GEMM and an MFMA-only probe; for decode a streaming-read probe of
the split pass's bytes. `roofline.measured_peak` puts the dominant kernel
against the probe of its kind at this part's clock. Run without --workload, the line also carries
`other_workloads`: the same steps of every other workload (bf16 and FP8),
each measured briefly without the library, clock and CPU legs.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from workloads import WORKLOADS, make_case, MASK_BLOCK_CAUSAL, MASK_CAUSAL  # noqa: E402

DEFAULT_WORKLOAD = "video_14b"
METRIC = "attention TFLOP/s + % bf16 MFMA peak per streaming step; decode HBM GB/s"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA (published 2.5 PFLOP/s)
PEAK_FP8_TFLOPS = 5033.2    # MI355X dense fp8 MFMA (published 5.0 PFLOP/s)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E (published 8 TB/s)


def visible_spans(wl, L: int):
    """Inclusive visible key-token range [lo, hi] of each query i of a stream
    holding L tokens (empty where hi < lo)."""
    i = np.arange(wl.n, dtype=np.int64)
    p = L + i
    if wl.mask.kind == MASK_BLOCK_CAUSAL:
        bp = p // wl.mask.block
        lo = (bp - wl.mask.window) * wl.mask.block if wl.mask.window else np.zeros_like(p)
        hi = (bp + 1) * wl.mask.block - 1
    else:
        lo = p - wl.mask.window + 1 if wl.mask.window else np.zeros_like(p)
        hi = p
    present_lo = max(0, L - wl.C)
    present_hi = L + wl.n - 1
    lo = np.maximum(lo, present_lo)
    hi = np.minimum(hi, present_hi)
    return lo, hi


def visible_counts(wl, L: int):
    """Number of keys each query i of a stream holding L tokens attends to."""
    lo, hi = visible_spans(wl, L)
    return np.maximum(hi - lo + 1, 0)


def step_work(wl, lengths, kv_elem_bytes: int = 2):
    """(attention flops, minimum HBM bytes) of one step for per-stream lengths;
    ring elements take kv_elem_bytes (2 for bf16, 1 for FP8 codes)."""
    flops = 0
    kv_bytes = 0
    for L in lengths:
        lo, hi = visible_spans(wl, int(L))
        live = hi >= lo
        flops += int((hi - lo + 1)[live].sum()) * 4 * wl.d * wl.Hq
        # distinct keys read by the stream: the union of the queries' ranges,
        # which is one range (the ranges' ends never decrease with i)
        if live.any():
            union = int(hi[live].max() - lo[live].min() + 1)
            kv_bytes += union * wl.Hkv * wl.d * 2 * kv_elem_bytes
    qo_bytes = 2 * wl.B * wl.n * wl.Hq * wl.d * 2
    return flops, kv_bytes + qo_bytes


def _blas_threads() -> int:
    try:
        import threadpoolctl
        return max(i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()) or 1
    except Exception:
        return len(os.sched_getaffinity(0))


def fp8_scales(wl):
    """Per-(stream, KV head) FP8 scales: N(0, 1)*qk_scale keys and N(0, 1)
    values land around code 50, their tails well inside +-448."""
    ks = np.full((wl.B, wl.Hkv), 0.02 * wl.qk_scale, np.float32)
    vs = np.full((wl.B, wl.Hkv), 0.02, np.float32)
    return ks, vs


def cpu_baseline(wl, case, seconds: float, fp8: bool = False):
    """Time the fp64 oracle on a bounded sample of the measured step.

    The sample is the first `rows` query tokens of every stream and head; `rows`
    grows from 64 until one timed call takes at least half of `seconds` (or
    covers the whole chunk). The last call is the one reported. With fp8 the
    oracle is the FP8 step's.
    """
    import oracle
    from oracle import fp8 as ofp8
    if fp8:
        ks, vs = fp8_scales(wl)
        oring = ofp8.RingFP8(wl.B, wl.Hkv, wl.C, wl.d)
        app = lambda r, k, v, streams=None: ofp8.kv_append_fp8(r, k, v, wl.rope, ks, vs,  # noqa
                                                               streams=streams)
    else:
        oring = oracle.new_ring(wl.B, wl.Hkv, wl.C, wl.d)
        app = lambda r, k, v, streams=None: oracle.kv_append(r, k, v, wl.rope,  # noqa
                                                             streams=streams)
    for k, v in case.prior_steps:
        oring = app(oring, k, v)
    for b, (k, v) in enumerate(case.prior_fills):
        for s in range(0, k.shape[1], wl.C):
            e = min(k.shape[1], s + wl.C)
            oring = app(oring, k[:, s:e], v[:, s:e], streams=[b])

    def timed(nrows):
        rows = np.arange(min(wl.n, nrows), dtype=np.int64)
        t0 = time.perf_counter()
        if fp8:
            ofp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask, ks, vs,
                                 rows=rows)
        else:
            oracle.stream_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask,
                               rows=rows)
        return rows, time.perf_counter() - t0

    rows, dt = timed(64)
    while dt < 0.5 * seconds and len(rows) < wl.n:
        grow = max(2.0, seconds / max(dt, 1e-3))
        rows, dt = timed(int(len(rows) * grow))
    reps = 1
    while dt < 0.5 * seconds and reps < 20:  # whole chunk covered: repeat it
        dt += timed(len(rows))[1]
        reps += 1
    flops = 0
    for L in case.prior_lengths:
        flops += int(visible_counts(wl, int(L))[rows].sum()) * 4 * wl.d * wl.Hq
    res = {"value": flops * reps / dt / 1e12, "unit": "TFLOP/s", "cores": _blas_threads(),
           "host_cores": len(os.sched_getaffinity(0)), "kind": "oracle",
           "sample": "first %d of %d query tokens per stream, all %d heads, %d call(s) "
                     "(%.2f GFLOP fp64 each, %.1f s)"
                     % (len(rows), wl.n, wl.Hq, reps, flops / 1e9, dt)}
    if not fp8 and wl.B * wl.n * wl.Hq * wl.C * wl.d <= 1 << 20:
        # the pure-Python loop twin of the oracle, on the whole step of a tiny workload
        from oracle import brute
        model = brute.ListRing(wl.B, wl.Hkv, wl.C, wl.d)
        for k, v in case.prior_steps:
            model.append(k.tolist(), v.tolist(), wl.rope)
        q, kn, vn = case.q.tolist(), case.k_new.tolist(), case.v_new.tolist()
        t0 = time.perf_counter()
        brute.attend(model, q, kn, vn, wl.rope, wl.mask, wl.Hq)
        res["brute_twin_ms"] = 1e3 * (time.perf_counter() - t0)
    return res


def cpu_baseline_decode(wl, case, seconds: float, fp8: bool = False):
    """Time the oracle on the whole decode step, repeated up to about `seconds`
    (with fp8, the FP8 step's oracle on an FP8 ring)."""
    import oracle
    from oracle import fp8 as ofp8
    if fp8:
        ks, vs = fp8_scales(wl)
        oring = ofp8.RingFP8(wl.B, wl.Hkv, wl.C, wl.d)
    else:
        oring = oracle.new_ring(wl.B, wl.Hkv, wl.C, wl.d)
    for b in range(wl.B):
        k, v = case.prior_fills[b]
        if fp8:
            ofp8.kv_append_fp8(oring, k, v, wl.rope, ks, vs, streams=[b])
        else:
            oring = oracle.kv_append(oring, k, v, wl.rope, streams=[b])
    reps, dt = 0, 0.0
    while reps < 200 and (reps == 0 or dt < seconds):
        t0 = time.perf_counter()
        if fp8:
            ofp8.stream_attn_fp8(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask, ks, vs)
        else:
            oracle.decode_attn(oring, case.q, case.k_new, case.v_new, wl.rope, wl.mask)
        dt += time.perf_counter() - t0
        reps += 1
    _, by = step_work(wl, case.prior_lengths, 1 if fp8 else 2)
    return {"value": by * reps / dt / 1e9, "unit": "GB/s", "cores": _blas_threads(),
            "host_cores": len(os.sched_getaffinity(0)), "kind": "oracle",
            "sample": "whole step, all %d streams, %d repetitions (%.1f MB each, %.1f s)"
                      % (wl.B, reps, by / 1e6, dt)}


def clock_power(run, seconds: float = 1.5):
    """Graphics clock and socket power while `run` (a few launches, synchronised)
    repeats for about `seconds`, sampled with amd-smi: the part runs at its
    power limit under this load, so the clock a kernel gets differs from one
    MI355X to another. None where amd-smi is missing or prints nothing usable."""
    import subprocess
    import threading

    samples = []
    stop = threading.Event()

    def sample():
        while not stop.is_set():
            try:
                r = subprocess.run(["amd-smi", "metric", "-p", "-c", "--json"],
                                   capture_output=True, text=True, timeout=10)
                samples.append(json.loads(r.stdout))
            except Exception:
                pass
            stop.wait(0.1)

    th = threading.Thread(target=sample, daemon=True)
    t0 = time.perf_counter()
    th.start()
    while time.perf_counter() - t0 < seconds:
        run()
    stop.set()
    th.join(timeout=15)
    clk, pw = [], []
    for d in samples:
        try:
            g = d["gpu_data"][0] if isinstance(d, dict) else d[0]
            c = [v["clk"]["value"] for k, v in g["clock"].items() if k.startswith("gfx_")
                 and isinstance(v.get("clk"), dict) and isinstance(v["clk"].get("value"), (int, float))]
            if c:
                clk.append(float(np.mean(c)))
            w = g["power"]["socket_power"]["value"]
            if isinstance(w, (int, float)):
                pw.append(float(w))
        except (KeyError, IndexError, TypeError):
            continue
    if not clk and not pw:
        return None
    return {"gfx_mhz": float(np.median(clk)) if clk else None,
            "socket_w": float(np.median(pw)) if pw else None, "samples": len(samples),
            "source": "amd-smi metric -p -c, during %.1f s of further launches" % seconds}


def library_baseline(wl, dev):
    """The vendor libraries on the same part, as context for the roofline
    fraction: a 1 GiB device copy (read plus write) and, for the
    chunk steps, torch's scaled_dot_product_attention (its flash or
    memory-efficient kernel, never the math path) at the step's shape with all
    C + n keys visible and no mask (more flops than the step; its own rate),
    and a hipBLASLt bf16 GEMM. An entry the library rejects is reported as its
    error."""
    import torch
    import torch.nn.functional as F

    def timed(fn, iters):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters * 1e-3

    g = torch.Generator(device=dev).manual_seed(0)
    res = {}
    a = torch.empty(1 << 28, device=dev, dtype=torch.float32)  # 1 GiB
    b = torch.empty_like(a)
    t = timed(lambda: b.copy_(a), 10)
    res["copy_1gib"] = {"us": t * 1e6, "GB/s": 2 * a.numel() * 4 / t / 1e9,
                        "note": "read + write bytes"}
    del a, b
    if wl.n == 1:
        return res
    nk = wl.C + wl.n
    q = torch.randn(wl.B, wl.Hq, wl.n, wl.d, device=dev, dtype=torch.bfloat16, generator=g)
    k = torch.randn(wl.B, wl.Hq, nk, wl.d, device=dev, dtype=torch.bfloat16, generator=g)
    v = torch.randn(wl.B, wl.Hq, nk, wl.d, device=dev, dtype=torch.bfloat16, generator=g)
    fl = 4.0 * wl.B * wl.Hq * wl.n * nk * wl.d
    backends = [torch.nn.attention.SDPBackend.FLASH_ATTENTION,
                torch.nn.attention.SDPBackend.EFFICIENT_ATTENTION]
    try:
        with torch.nn.attention.sdpa_kernel(backends):
            t = timed(lambda: F.scaled_dot_product_attention(q, k, v), 5)
        res["sdpa"] = {"us": t * 1e6, "TFLOP/s": fl / t / 1e12,
                       "shape": "q %s, k/v %s (K/V heads expanded to the query heads), "
                                "no mask" % (list(q.shape), list(k.shape))}
    except RuntimeError as e:
        res["sdpa"] = {"error": str(e)[:200]}
    del q, k, v
    n = 8192
    a = torch.randn(n, n, device=dev, dtype=torch.bfloat16, generator=g)
    b = torch.randn(n, n, device=dev, dtype=torch.bfloat16, generator=g)
    t = timed(lambda: a @ b, 10)
    res["gemm_bf16_8192"] = {"us": t * 1e6, "TFLOP/s": 2.0 * n ** 3 / t / 1e12}
    del a, b
    torch.cuda.synchronize()
    return res


def mfma_loop(dev, fp8: bool, no_clock: bool = False):
    """The MFMA-only probe (libfrt_probe.so): random operands, 4 chains per
    wave, one block of 8 waves per CU. Returns its TFLOP/s and launch time (and
    the clock and power while it repeats), or the reason it could not run."""
    import ctypes
    import torch
    from paper_2607_18171_amd.build import PROBE_LIB
    if not os.path.exists(PROBE_LIB):
        return {"error": "%s not built" % PROBE_LIB}
    lib = ctypes.CDLL(PROBE_LIB)
    fn = lib.frt_probe_mfma_fp8 if fp8 else lib.frt_probe_mfma_bf16
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    g = torch.Generator(device=dev).manual_seed(0)
    nfrag = 2 * 4 * 64  # fragments: 16 bytes (bf16) or 32 bytes (FP8) each
    if fp8:
        frags = (torch.randn(nfrag * 32, device=dev, generator=g) * 4).to(torch.float8_e4m3fn)
    else:
        frags = torch.randn(nfrag * 8, device=dev, generator=g).to(torch.bfloat16)
    blocks, iters = 256, 4096
    out = torch.empty(blocks * 512, device=dev, dtype=torch.float32)
    stream = torch.cuda.current_stream()

    def run():
        rc = fn(frags.data_ptr(), out.data_ptr(), blocks, iters, stream.cuda_stream)
        if rc != 0:
            raise RuntimeError("frt_probe_mfma: HIP error %d" % rc)

    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    reps = 10
    e0.record(stream)
    for _ in range(reps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) / reps * 1e-3
    flops = blocks * 8 * 4 * iters * 32 * 32 * (64 if fp8 else 16) * 2

    def burst():
        for _ in range(10):
            run()
        torch.cuda.synchronize()

    cp = None if no_clock else clock_power(burst, 1.0)
    # the same loop on all-zero operands: no switching in the multipliers
    frags.zero_()
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    tz = e0.elapsed_time(e1) / reps * 1e-3
    return {"us": t * 1e6, "TFLOP/s": flops / t / 1e12, "clock_power": cp,
            "zero_operands_TFLOP/s": flops / tz / 1e12,
            "config": "%d blocks x 8 waves, 4 chains of %d MFMAs (32x32x%d %s) on random "
                      "operands, no memory or vector work"
                      % (blocks, iters, 64 if fp8 else 16, "e4m3" if fp8 else "bf16")}


def stream_read(dev, nbytes: int):
    """The streaming-read probe (libfrt_probe.so) on `nbytes`, the dominant
    kernel's algorithmic bytes per launch: plain 16-byte loads over three
    buffers of that size taken in turn (the same rotation as the cold decode
    rings, so the Infinity Cache cannot serve a repeat), at a few grid sizes
    and loads-in-flight counts; the best is the read rate this part reaches
    for that many bytes in one launch."""
    import ctypes
    import torch
    from paper_2607_18171_amd.build import PROBE_LIB
    if not os.path.exists(PROBE_LIB):
        return {"error": "%s not built" % PROBE_LIB}
    lib = ctypes.CDLL(PROBE_LIB)
    fn = lib.frt_probe_read
    fn.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                   ctypes.c_void_p]
    fn.restype = ctypes.c_int
    n = (nbytes + 15) // 16 * 16
    g = torch.Generator(device=dev).manual_seed(0)
    bufs = [torch.randint(0, 1 << 62, (n // 8,), device=dev, dtype=torch.int64, generator=g)
            for _ in range(3)]
    # grid-stride grids, and grids in which every thread issues all of its
    # loads at once (one pass, blocks = words / (256 * unroll))
    configs = [(blocks, unroll) for blocks in (2048, 4096, 8192, 16384) for unroll in (8, 16)]
    configs += [(-(-n // (16 * 256 * unroll)), unroll) for unroll in (2, 4, 8)]
    sink = torch.zeros(max(b for b, _ in configs), device=dev, dtype=torch.int32)
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    table = {}
    for blocks, unroll in configs:
        def run(i):
            rc = fn(bufs[i % 3].data_ptr(), n, sink.data_ptr(), blocks, unroll, stream.cuda_stream)
            if rc != 0:
                raise RuntimeError("frt_probe_read: HIP error %d" % rc)
        for i in range(6):
            run(i)
        torch.cuda.synchronize()
        reps = 30
        e0.record(stream)
        for i in range(reps):
            run(i)
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / reps * 1e-3
        table["%dx%d" % (blocks, unroll)] = n / t / 1e9
    best = max(table, key=table.get)
    del bufs
    torch.cuda.synchronize()
    return {"GB/s": table[best], "us": n / table[best] / 1e3, "bytes": n,
            "config": "%s blocks x loads in flight per thread, 256 threads a block, three "
                      "buffers in turn" % best,
            "by_config_GB/s": {k: round(v, 1) for k, v in table.items()}}


# Default warm-up length: after an idle spell the part needs 15-20 ms of load
# to reach its steady clock (a 1.3B-like step measured 823 -> 745 -> 727 ->
# 701 -> 682 -> 672 us in consecutive 5-step windows from a cold start).
WARMUP_MS = 200

# HBM traffic per launch of the dominant kernel, from rocprofv3 FETCH_SIZE and
# WRITE_SIZE passes scaled by a plain-copy calibration; used only while the
# library's machine code for the kernel is the code the counters were taken on.
TRAFFIC_FILES = {("chunk_attn", "video_14b"): "profiles/chunk_attn_video_14b.txt",
                 ("chunk_attn", "video_1p3b"): "profiles/chunk_attn_video_1p3b.txt",
                 ("decode_split", "decode"): "profiles/decode_split_decode.txt",
                 ("chunk_attn_fp8", "video_1p3b"): "profiles/chunk_attn_fp8_video_1p3b.txt",
                 ("decode_split_fp8", "decode"): "profiles/decode_split_fp8_decode.txt"}
# The kernels' symbols (head_dim 128, the instantiation every bench workload
# runs) in the library's gfx950 code object.
KERNEL_SYMBOLS = {"chunk_attn": "17chunk_attn_kernelILi128ELi8E",
                  "decode_split": "19decode_split_kernelILi128E",
                  "chunk_attn_fp8": "21chunk_attn_fp8_kernelILi128ELi8E",
                  "decode_split_fp8": "23decode_split_fp8_kernelILi128E"}


def _elf_symbol_bytes(elf: bytes, part: str):
    """Name and bytes of every sized symbol whose name contains `part` in an
    ELF64 image (the kernel's code and its kernel descriptor)."""
    import struct
    shoff = struct.unpack_from("<Q", elf, 0x28)[0]
    shentsize, shnum = struct.unpack_from("<HH", elf, 0x3A)
    secs = [struct.unpack_from("<IIQQQQIIQQ", elf, shoff + k * shentsize) for k in range(shnum)]
    out = b""
    for sec in secs:
        if sec[1] != 2:  # SHT_SYMTAB
            continue
        strtab = secs[sec[6]]
        for k in range(sec[5] // 24):
            name_off, _, _, shndx, value, size = struct.unpack_from("<IBBHQQ", elf,
                                                                    sec[4] + 24 * k)
            start = strtab[4] + name_off
            name = elf[start:elf.index(b"\0", start)]
            if size and part.encode() in name and shndx < shnum:
                host = secs[shndx]
                fo = host[4] + (value - host[3])
                out += name + elf[fo:fo + size]
    return out or None


def kernel_code_sha256(kernel: str, lib_path: str):
    """sha256 of a kernel's gfx950 machine code and descriptor in the built
    library (its offload bundles), or None if it is not found."""
    import hashlib
    import struct
    data = open(lib_path, "rb").read()
    magic = b"__CLANG_OFFLOAD_BUNDLE__"
    pos = data.find(magic)
    while pos >= 0:
        n = struct.unpack_from("<Q", data, pos + len(magic))[0]
        off = pos + len(magic) + 8
        for _ in range(n):
            eo, es, tl = struct.unpack_from("<QQQ", data, off)
            triple = data[off + 24:off + 24 + tl]
            off += 24 + tl
            if b"gfx950" in triple and es:
                code = _elf_symbol_bytes(data[pos + eo:pos + eo + es], KERNEL_SYMBOLS[kernel])
                if code is not None:
                    return hashlib.sha256(code).hexdigest()
        pos = data.find(magic, pos + 1)
    return None


def recorded_traffic(kernel: str, workload: str, lib_path: str):
    """HBM bytes per launch from the committed profile summary, while the
    library's machine code for the kernel is the one the counters were taken
    on; None otherwise."""
    path = TRAFFIC_FILES.get((kernel, workload))
    if path is None or not os.path.exists(os.path.join(ROOT, path)):
        return None
    fields = {}
    for line in open(os.path.join(ROOT, path)):
        if " = " in line:
            k, v = line.split(" = ", 1)
            fields[k.strip()] = v.strip()
    code = kernel_code_sha256(kernel, lib_path)
    if code is None or fields.get("kernel_code_sha256") != code:
        return None
    return int(fields["traffic_bytes_per_launch"])


def measure(args) -> dict:
    """Measure one workload as `args` describes it; returns the JSON line's
    fields."""
    import torch
    import paper_2607_18171_amd as frt

    wl = WORKLOADS[args.workload]
    case = make_case(wl, args.seed)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    def to_dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(
            torch.bfloat16).to(dev)

    # at most this many warm-up steps (the rotary table covers every position)
    max_warm = args.warmup if args.warmup >= 0 else (4000 if wl.n == 1 else 400)
    # warm-up, plain, one-ring, instrumented and graph-replayed passes
    total_steps = max_warm + 3 + 4 * args.steps
    max_tokens = int(case.prior_lengths.max()) + (total_steps + 1) * wl.n + 1
    rope = frt.Rope.for_tokens(wl.rope.mode, wl.rope.axis_dims, wl.rope.frame_hw, max_tokens,
                               wl.rope.base)
    if args.fp8:
        ks, vs = fp8_scales(wl)
        ring = frt.RingFp8(wl.B, wl.Hkv, wl.d, wl.C, torch.from_numpy(ks), torch.from_numpy(vs))
        append = frt.kv_append_fp8
    else:
        ring = frt.Ring(wl.B, wl.Hkv, wl.d, wl.C)
        append = frt.kv_append
    for k, v in case.prior_steps:
        append(ring, rope, to_dev(k), to_dev(v))
    for b, (k, v) in enumerate(case.prior_fills):
        for s in range(0, k.shape[1], wl.C):
            e = min(k.shape[1], s + wl.C)
            append(ring.view_stream(b), rope, to_dev(k[:, s:e]), to_dev(v[:, s:e]))
    decode = wl.n == 1
    nrings = args.rings if args.rings > 0 else (3 if decode else 1)
    rings = [ring]
    for _ in range(nrings - 1):  # same contents, separate buffers
        if args.fp8:
            copy = frt.RingFp8(wl.B, wl.Hkv, wl.d, wl.C, torch.from_numpy(ks),
                               torch.from_numpy(vs))
            copy.k.copy_(ring.k)
            copy.v.copy_(ring.v)
            copy.seq_len.copy_(ring.seq_len)
        else:
            copy = frt.Ring(wl.B, wl.Hkv, wl.d, wl.C, k=ring.k.clone(), v=ring.v.clone(),
                            seq_len=ring.seq_len.clone())
        rings.append(copy)
    q, kn, vn = to_dev(case.q), to_dev(case.k_new), to_dev(case.v_new)
    out = torch.empty_like(q)
    msk = frt.mask(wl.mask.kind, wl.mask.block, wl.mask.window)
    if decode and args.fp8:
        ws = torch.empty(frt.decode_fp8_workspace_bytes(ring, wl.Hq), dtype=torch.uint8,
                         device=dev)
    elif decode:
        ws = torch.empty(frt.decode_workspace_bytes(ring, wl.Hq), dtype=torch.uint8, device=dev)
    elif args.fp8:
        ws = torch.empty(frt.stream_attn_fp8_workspace_bytes(ring, wl.n, wl.Hq),
                         dtype=torch.uint8, device=dev)
    else:
        ws = torch.empty(frt.stream_attn_workspace_bytes(ring, wl.n, wl.Hq), dtype=torch.uint8,
                         device=dev)
    torch.cuda.synchronize()

    def step(r=0):
        rg = rings[r]
        if decode and args.fp8:
            frt.decode_step_fp8(rg, rope, msk, q, kn, vn, out, ws)
        elif decode:  # attention and the one-token append in one call
            frt.decode_step(rg, rope, msk, q, kn, vn, out, ws)
        elif args.fp8:
            frt.stream_step_fp8(rg, rope, msk, q, kn, vn, out, ws)
        else:
            frt.stream_step(rg, rope, msk, q, kn, vn, out, ws)

    warmup = 0
    if args.warmup >= 0:
        for _ in range(args.warmup):
            step()
        warmup = args.warmup
    else:
        # Time-based: steps until WARMUP_MS of them have run, then 3 more. A
        # decode step appends one token per stream, so its warm-up runs the
        # attention alone and the stream lengths stay those of the workload;
        # the chunk steps see a window of the ring that is already full.
        def warm(r):
            if decode and args.fp8:
                frt.decode_attn_fp8(rings[r], rope, msk, q, kn, vn, out, ws)
            elif decode:
                frt.decode_attn(rings[r], rope, msk, q, kn, vn, out, ws)
            else:
                step(r)
        t0 = time.perf_counter()
        while warmup + 8 <= max_warm and time.perf_counter() - t0 < WARMUP_MS * 1e-3:
            for i in range(8):
                warm((warmup + i) % nrings)
            warmup += 8
            torch.cuda.synchronize()
        for i in range(3):
            step(i % nrings)
        warmup += 3
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()

    def timed_steps(nr):
        """K steps rotating over the first nr rings, between two events on the
        launch stream; returns (ms per step, algorithmic flops per step,
        algorithmic bytes per step)."""
        lengths = [rg.seq_len.cpu().numpy().copy() for rg in rings[:nr]]
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for s in range(args.steps):
            step(s % nr)
        ev1.record(stream)
        torch.cuda.synchronize()
        # algorithmic work (a ring's lengths advance by n each time it is used)
        flops = bytes_ = 0
        for s in range(args.steps):
            f, by = step_work(wl, lengths[s % nr], 1 if args.fp8 else 2)
            lengths[s % nr] = lengths[s % nr] + wl.n
            flops += f
            bytes_ += by
        return ev0.elapsed_time(ev1) / args.steps, flops / args.steps, bytes_ / args.steps

    # Throughput: K plain steps. Per-kernel durations: K more steps with the
    # library's per-launch events, which add a few microseconds around every
    # launch (a third of a decode step), so they stay out of the first region.
    ms_step, flops_step, bytes_step = timed_steps(nrings)
    hot = None
    if nrings > 1:  # the same steps on one ring, whose reads the Infinity Cache may serve
        hms, hflops, hbytes = timed_steps(1)
        hot = {"ms_per_step": hms,
               "value": (hbytes / (hms * 1e-3) / 1e9) if decode else
                        (hflops / (hms * 1e-3) / 1e12)}
    frt.timing_reset()
    frt.timing_enable(True)
    _, kflops_step, kbytes_step = timed_steps(nrings)
    frt.timing_enable(False)

    graph = None
    if args.graph:
        # The same steps replayed from one HIP graph that holds a step per ring:
        # no host launch cost between steps (what a serving loop that captures
        # its step sees). Not the headline figure.
        lengths = [rg.seq_len.cpu().numpy().copy() for rg in rings]
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for r in range(nrings):
                step(r)
        reps = max(1, args.steps // nrings)
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(reps):
            g.replay()
        ev1.record(stream)
        torch.cuda.synchronize()
        gms = ev0.elapsed_time(ev1) / (reps * nrings)
        gf = gb = 0
        for _ in range(reps):
            for r in range(nrings):
                f, by = step_work(wl, lengths[r], 1 if args.fp8 else 2)
                lengths[r] = lengths[r] + wl.n
                gf += f
                gb += by
        gf /= reps * nrings
        gb /= reps * nrings
        graph = {"ms_per_step": gms,
                 "value": (gb / (gms * 1e-3) / 1e9) if decode else (gf / (gms * 1e-3) / 1e12),
                 "steps": reps * nrings}
        del g

    kernels = {}
    samples = {}
    for name in ("chunk_prep", "chunk_attn", "chunk_append", "decode_split", "decode_combine",
                 "rope_append", "seq_advance"):
        c, ms = frt.timing_query(name)
        if c:
            kernels[name] = {"launches": c, "avg_us": 1000.0 * ms / c}
            samples[name] = np.array(frt.timing_samples(name)) * 1000.0

    def pct(name):
        p10, p50, p90 = np.percentile(samples[name], [10, 50, 90])
        return {"p10_us": float(p10), "p50_us": float(p50), "p90_us": float(p90),
                "avg_us": kernels[name]["avg_us"]}

    if decode:
        value = bytes_step / (ms_step * 1e-3) / 1e9
        unit = "GB/s"
        dom = kernels["decode_split"]
        achieved = kbytes_step / (dom["avg_us"] * 1e-6) / 1e9
        kname = "decode_split_fp8" if args.fp8 else "decode_split"
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS,
                "traffic": recorded_traffic(kname, wl.name, frt.LIB_PATH), "kernel": kname,
                "step_frac": value / PEAK_HBM_GBS, "launch_us": pct("decode_split")}
    else:
        value = flops_step / (ms_step * 1e-3) / 1e12
        unit = "TFLOP/s"
        dom = kernels["chunk_attn"]
        achieved = kflops_step / (dom["avg_us"] * 1e-6) / 1e12
        peak = PEAK_FP8_TFLOPS if args.fp8 else PEAK_BF16_TFLOPS  # the contraction's own dtype
        kname = "chunk_attn_fp8" if args.fp8 else "chunk_attn"
        roof = {"bound": "mfma", "achieved": achieved, "peak": peak,
                "unit": "TFLOP/s", "frac": achieved / peak,
                "traffic": recorded_traffic(kname, wl.name, frt.LIB_PATH), "kernel": kname,
                "step_frac": value / peak, "launch_us": pct("chunk_attn")}

    cp = None
    if not args.no_clock_power:
        def few():  # attention without the append: the streams keep their lengths
            for i in range(4):
                rg = rings[i % nrings]
                if decode and args.fp8:
                    frt.decode_attn_fp8(rg, rope, msk, q, kn, vn, out, ws)
                elif decode:
                    frt.decode_attn(rg, rope, msk, q, kn, vn, out, ws)
                elif args.fp8:
                    frt.stream_attn_step_fp8(rg, rope, msk, q, kn, vn, out, ws)
                else:
                    frt.stream_attn_step(rg, rope, msk, q, kn, vn, out, ws)
            torch.cuda.synchronize()
        cp = clock_power(few)
    lib = None if args.no_library else library_baseline(wl, dev)
    # the measured ceiling beside the published one, at this part's clock:
    # the MFMA-only probe for the chunk steps, the streaming-read probe of the
    # split pass's bytes for decode
    if not args.no_library:
        if decode:
            lib["stream_read"] = stream_read(dev, int(kbytes_step))
            if "GB/s" in lib["stream_read"]:
                mp = lib["stream_read"]["GB/s"]
                roof["measured_peak"] = {"value": mp, "unit": "GB/s",
                                         "frac": roof["achieved"] / mp,
                                         "source": "library.stream_read"}
        else:
            lib["mfma_loop"] = mfma_loop(dev, args.fp8, args.no_clock_power)
            if "TFLOP/s" in lib["mfma_loop"]:
                mp = lib["mfma_loop"]["TFLOP/s"]
                roof["measured_peak"] = {"value": mp, "unit": "TFLOP/s",
                                         "frac": roof["achieved"] / mp,
                                         "source": "library.mfma_loop"}

    cpu = None
    if args.cpu_seconds > 0 and not decode:
        cpu = cpu_baseline(wl, case, args.cpu_seconds, fp8=args.fp8)
    elif args.cpu_seconds > 0:
        cpu = cpu_baseline_decode(wl, case, args.cpu_seconds, fp8=args.fp8)

    line = {
        "metric": METRIC, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
        "warmup": warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp8" if args.fp8 else "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "streams": wl.B, "q_heads": wl.Hq, "kv_heads": wl.Hkv,
                   "head_dim": wl.d, "chunk_tokens": wl.n, "ring_slots": wl.C,
                   "mask": "block_causal" if wl.mask.kind == MASK_BLOCK_CAUSAL else "causal",
                   "window": wl.mask.window, "seed": args.seed,
                   "step_gflop": flops_step / 1e9, "step_min_mb": bytes_step / 1e6,
                   "rings": nrings, "parallelism": "single_gpu"},
        "kernels_us": {k: round(v["avg_us"], 2) for k, v in kernels.items()},
        "hot": hot,
        "graph": graph,
        "roofline": roof,
        "clock_power": cp,
        "library": lib,
        "cpu_baseline": cpu,
    }
    return line


# Measured after the default workload, each briefly (no library, clock or
# CPU legs), so that one bench line holds every configuration:
# (workload, FP8 ring)
OTHER_WORKLOADS = (("video_1p3b", False), ("prefill_swa", False), ("decode", False),
                   ("video_1p3b", True), ("decode", True))


def summary(line: dict) -> dict:
    """The compact record of one workload's measurement."""
    r = line["roofline"]
    return {"workload": line["config"]["workload"], "dtype": line["dtype"],
            "ms_per_step": line["ms_per_step"], "value": line["value"],
            "unit": line["unit"], "rings": line["config"]["rings"],
            "kernel": r["kernel"], "kernel_us": r["launch_us"]["avg_us"],
            "achieved": r["achieved"], "peak": r["peak"], "frac": r["frac"],
            "step_frac": r["step_frac"], "kernels_us": line["kernels_us"],
            "hot": line["hot"]}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=-1,
                    help="untimed warm-up steps (default: %d ms of steps, then 3 more; "
                         "after an idle spell the part takes 15-20 ms to reach its steady "
                         "clock)" % WARMUP_MS)
    ap.add_argument("--workload", default=None, choices=sorted(WORKLOADS),
                    help="default %s; with no --workload the line also carries a brief "
                         "measurement of every other workload (other_workloads)"
                         % DEFAULT_WORKLOAD)
    ap.add_argument("--rings", type=int, default=0,
                    help="ring copies the steps rotate over (default: 3 for decode, whose "
                         "ring would otherwise stay in the Infinity Cache; 1 otherwise)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target length of the oracle's timed CPU sample (0 = skip)")
    ap.add_argument("--fp8", action="store_true",
                    help="the FP8 (e4m3fn) ring (head_dim 128): frt_stream_step_fp8, or "
                         "frt_decode_step_fp8 for the decode workload")
    ap.add_argument("--no-library", action="store_true",
                    help="skip the vendor-library and probe comparison (a device copy; torch "
                         "SDPA, hipBLASLt GEMM and the MFMA probe, or the streaming-read probe "
                         "for decode)")
    ap.add_argument("--no-others", action="store_true",
                    help="skip the brief measurement of the other workloads that a run "
                         "without --workload adds")
    ap.add_argument("--graph", action="store_true",
                    help="also time the same steps replayed from a HIP graph")
    ap.add_argument("--no-clock-power", action="store_true",
                    help="skip sampling the clock and socket power with amd-smi")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-sized device buffer 3 times (known HBM traffic for "
                         "scaling FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args(argv)
    if args.copy_calibration:
        import torch
        a = torch.ones(args.copy_calibration << 18, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": a.numel() * 4}))
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the step runs on one MI355X and nothing in this "
              "library crosses GPUs (requested --gpus %d)" % args.gpus, file=sys.stderr)
        return 2

    explicit = args.workload is not None
    if not explicit:
        args.workload = DEFAULT_WORKLOAD
    if args.fp8 and WORKLOADS[args.workload].d != 128:
        print("--fp8 covers the workloads with head_dim 128", file=sys.stderr)
        return 2
    line = measure(args)
    if not explicit and not args.no_others and not args.fp8:
        others = []
        for name, fp8 in OTHER_WORKLOADS:
            sub = argparse.Namespace(**vars(args))
            sub.workload, sub.fp8, sub.rings = name, fp8, 0
            sub.cpu_seconds, sub.no_library, sub.no_clock_power, sub.graph = 0, True, True, False
            others.append(summary(measure(sub)))
        line["other_workloads"] = others
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
