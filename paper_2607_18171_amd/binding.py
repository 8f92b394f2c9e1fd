"""ctypes binding of libfrt.so: argument marshalling only.

Every computation of the step runs in the library's HIP kernels; this module
only turns torch tensors into pointers, sizes and a hipStream_t, and turns a
non-zero frt_status into FrtError. PyTorch provides device memory and
streams. If libfrt.so is missing the import of the library fails loudly:
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libfrt.so")

FRT_OK = 0
STATUS_NAMES = {0: "FRT_OK", 1: "FRT_ERR_NULL", 2: "FRT_ERR_SHAPE", 3: "FRT_ERR_UNSUPPORTED",
                4: "FRT_ERR_CAPACITY", 5: "FRT_ERR_ALIGN", 6: "FRT_ERR_WORKSPACE",
                7: "FRT_ERR_HIP"}
ROPE_NONE, ROPE_1D, ROPE_3D = 0, 1, 2
MASK_BLOCK_CAUSAL, MASK_CAUSAL = 1, 2

# every symbol include/frt.h declares
EXPORTS = (
    "frt_rope_table_bytes", "frt_rope_table_fill", "frt_kv_append",
    "frt_stream_attn_workspace_bytes", "frt_stream_attn_step", "frt_stream_step",
    "frt_decode_max_splits",
    "frt_decode_workspace_bytes", "frt_decode_attn", "frt_decode_step", "frt_decode_step_noalloc",
    "frt_kv_append_fp8",
    "frt_stream_attn_fp8_workspace_bytes", "frt_stream_attn_step_fp8", "frt_stream_step_fp8",
    "frt_decode_fp8_workspace_bytes", "frt_decode_attn_fp8", "frt_decode_step_fp8",
    "frt_status_str",
    "frt_last_error",
    "frt_timing_enable", "frt_timing_query", "frt_timing_samples", "frt_timing_reset",
)


class FrtError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), message))
        self.status = status


class CRing(ctypes.Structure):
    _fields_ = [("num_streams", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("k_ring", ctypes.c_void_p), ("v_ring", ctypes.c_void_p),
                ("seq_len", ctypes.c_void_p)]


class CRope(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("axis_dims", ctypes.c_int32 * 3),
                ("frame_hw", ctypes.c_int32 * 2), ("max_pos", ctypes.c_int32 * 3),
                ("base", ctypes.c_double), ("table", ctypes.c_void_p)]


class CMask(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("block", ctypes.c_int32), ("window", ctypes.c_int32)]


class CFp8Scales(ctypes.Structure):
    _fields_ = [("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libfrt.so and declare its signatures (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError("libfrt.so not built at %s (run python -m paper_2607_18171_amd.build)"
                          % path)
    # torch first: libfrt then binds to the HIP runtime torch already loaded,
    # so both share one runtime, one device context and the same streams.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I32 = ctypes.c_int32
    SZ = ctypes.c_size_t
    RP, OP, MP = ctypes.POINTER(CRing), ctypes.POINTER(CRope), ctypes.POINTER(CMask)
    SP = ctypes.POINTER(CFp8Scales)
    sig = {
        "frt_rope_table_bytes": (SZ, [OP]),
        "frt_rope_table_fill": (I32, [OP, P, SZ]),
        "frt_kv_append": (I32, [RP, OP, P, P, I32, P]),
        "frt_stream_attn_workspace_bytes": (SZ, [RP, I32, I32]),
        "frt_stream_attn_step": (I32, [RP, OP, MP, P, P, P, I32, I32, ctypes.c_float, P, SZ, P,
                                       P, P]),
        "frt_stream_step": (I32, [RP, OP, MP, P, P, P, I32, I32, ctypes.c_float, P, SZ, P,
                                  P, P]),
        "frt_decode_max_splits": (I32, [RP]),
        "frt_decode_workspace_bytes": (SZ, [RP, I32]),
        "frt_decode_attn": (I32, [RP, OP, MP, P, P, P, I32, ctypes.c_float, P, SZ, P, P, P]),
        "frt_decode_step": (I32, [RP, OP, MP, P, P, P, I32, ctypes.c_float, P, SZ, P, P, P]),
        "frt_decode_step_noalloc": (I32, [RP, OP, MP, P, P, P, I32, ctypes.c_float, P, P, P]),
        "frt_kv_append_fp8": (I32, [RP, SP, OP, P, P, I32, P]),
        "frt_stream_attn_fp8_workspace_bytes": (SZ, [RP, I32, I32]),
        "frt_stream_attn_step_fp8": (I32, [RP, SP, OP, MP, P, P, P, I32, I32, ctypes.c_float, P,
                                           SZ, P, P, P]),
        "frt_stream_step_fp8": (I32, [RP, SP, OP, MP, P, P, P, I32, I32, ctypes.c_float, P,
                                      SZ, P, P, P]),
        "frt_decode_fp8_workspace_bytes": (SZ, [RP, I32]),
        "frt_decode_attn_fp8": (I32, [RP, SP, OP, MP, P, P, P, I32, ctypes.c_float, P, SZ, P, P,
                                      P]),
        "frt_decode_step_fp8": (I32, [RP, SP, OP, MP, P, P, P, I32, ctypes.c_float, P, SZ, P, P,
                                      P]),
        "frt_status_str": (ctypes.c_char_p, [I32]),
        "frt_last_error": (ctypes.c_char_p, []),
        "frt_timing_enable": (I32, [I32]),
        "frt_timing_query": (I32, [ctypes.c_char_p, ctypes.POINTER(I32),
                                   ctypes.POINTER(ctypes.c_double)]),
        "frt_timing_samples": (I32, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_float), I32,
                                     ctypes.POINTER(I32)]),
        "frt_timing_reset": (None, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != FRT_OK:
        raise FrtError(status, load_library().frt_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


# ------------------------------------------------------------------ state --
V_BLOCK = 32  # slots per V ring block


def v_offsets(capacity: int, head_dim: int, slots=None):
    """Element offset of (slot, dim) inside one head's V ring storage, as an
    int64 tensor [len(slots)][head_dim] (every slot when None): blocks of
    V_BLOCK slots, each stored row by row of the head dimension (a partial
    last block has rows of capacity % V_BLOCK slots)."""
    import torch
    if slots is None:
        slots = torch.arange(capacity, dtype=torch.int64)
    s = torch.as_tensor(slots, dtype=torch.int64).reshape(-1, 1)
    d = torch.arange(head_dim, dtype=torch.int64)[None, :]
    nfull = capacity // V_BLOCK
    w = torch.where(s // V_BLOCK < nfull, V_BLOCK, capacity - V_BLOCK * nfull)
    return V_BLOCK * head_dim * (s // V_BLOCK) + w * d + s % V_BLOCK


class Ring:
    """A ring-buffer KV cache in device memory (torch tensors), zero-filled.

    k: bf16 [B][Hkv][C][d]; v: bf16 [B][Hkv][C*d] in blocks of V_BLOCK slots
    (element of slot s, dim d: v_offsets(C, d)[s, d]); seq_len: int64 [B].
    """

    def __init__(self, num_streams: int, num_kv_heads: int, head_dim: int, capacity: int,
                 device="cuda", k=None, v=None, seq_len=None):
        import torch
        self.B, self.Hkv, self.d, self.C = num_streams, num_kv_heads, head_dim, capacity
        self.k = k if k is not None else torch.zeros(
            (num_streams, num_kv_heads, capacity, head_dim), dtype=torch.bfloat16, device=device)
        self.v = v if v is not None else torch.zeros(
            (num_streams, num_kv_heads, capacity * head_dim), dtype=torch.bfloat16, device=device)
        self.seq_len = seq_len if seq_len is not None else torch.zeros(
            num_streams, dtype=torch.int64, device=device)

    def c(self) -> CRing:
        return CRing(self.B, self.Hkv, self.d, self.C, _ptr(self.k), _ptr(self.v),
                     _ptr(self.seq_len))

    def v_index(self, slots=None):
        """Flat element indices into a head's V storage for `slots` (all
        slots when None), shaped [len(slots)][d], on the ring's device."""
        return v_offsets(self.C, self.d, slots).to(self.v.device)

    def v_tokens(self):
        """V as bf16 [B][Hkv][C][d] (slot-major copy of the block layout)."""
        idx = self.v_index()
        return self.v[:, :, idx.reshape(-1)].reshape(self.B, self.Hkv, self.C, self.d)

    def view_stream(self, b: int) -> "Ring":
        """A one-stream view sharing memory with stream b."""
        return Ring(1, self.Hkv, self.d, self.C, k=self.k[b:b + 1], v=self.v[b:b + 1],
                    seq_len=self.seq_len[b:b + 1])


class Rope:
    """Rotary description plus its device table (built by frt_rope_table_fill)."""

    def __init__(self, mode: int, axis_dims: Sequence[int] = (0, 0, 0),
                 frame_hw: Sequence[int] = (0, 0), max_pos: Sequence[int] = (0, 0, 0),
                 base: float = 10000.0, device="cuda"):
        import torch
        self.mode = mode
        self.axis_dims = tuple(int(x) for x in axis_dims)
        self.frame_hw = tuple(int(x) for x in frame_hw)
        self.max_pos = tuple(int(x) for x in max_pos)
        self.base = float(base)
        self.table = None
        if mode != ROPE_NONE:
            c = self.c()
            nbytes = load_library().frt_rope_table_bytes(ctypes.byref(c))
            host = torch.empty(nbytes // 4, dtype=torch.float32)
            _check(load_library().frt_rope_table_fill(ctypes.byref(c), host.data_ptr(), nbytes))
            self.host_table = host
            self.table = host.to(device)

    @staticmethod
    def for_tokens(mode: int, axis_dims, frame_hw=(0, 0), max_tokens: int = 1,
                   base: float = 10000.0, device="cuda") -> "Rope":
        """A table large enough for token positions 0..max_tokens-1."""
        if mode == ROPE_3D:
            fh, fw = frame_hw
            max_pos = ((max_tokens + fh * fw - 1) // (fh * fw), fh, fw)
        elif mode == ROPE_1D:
            max_pos = (max_tokens, 0, 0)
        else:
            max_pos = (0, 0, 0)
        return Rope(mode, axis_dims, frame_hw, max_pos, base, device)

    def c(self) -> CRope:
        return CRope(self.mode, (ctypes.c_int32 * 3)(*self.axis_dims),
                     (ctypes.c_int32 * 2)(*self.frame_hw), (ctypes.c_int32 * 3)(*self.max_pos),
                     self.base, _ptr(self.table))


def mask(kind: int, block: int = 0, window: int = 0) -> CMask:
    return CMask(kind, block, window)


# -------------------------------------------------------------- entry points --
def kv_append(ring: Ring, rope: Rope, k_new, v_new, stream=None) -> None:
    """frt_kv_append: k_new, v_new bf16 [B][n][Hkv][d] on the device."""
    n = k_new.shape[1]
    cr, co = ring.c(), rope.c()
    _check(load_library().frt_kv_append(ctypes.byref(cr), ctypes.byref(co), _ptr(k_new),
                                        _ptr(v_new), n, _stream(stream)))


def stream_attn_workspace_bytes(ring: Ring, n_new: int, num_q_heads: int) -> int:
    cr = ring.c()
    return load_library().frt_stream_attn_workspace_bytes(ctypes.byref(cr), n_new, num_q_heads)


def stream_attn_step(ring: Ring, rope: Rope, msk: CMask, q, k_new, v_new, out, workspace,
                     lse=None, softmax_scale: float = 0.0, stream=None) -> None:
    """frt_stream_attn_step: q/out bf16 [B][n][Hq][d]; workspace a uint8 device tensor."""
    n, hq = q.shape[1], q.shape[2]
    cr, co = ring.c(), rope.c()
    _check(load_library().frt_stream_attn_step(
        ctypes.byref(cr), ctypes.byref(co), ctypes.byref(msk), _ptr(q), _ptr(k_new), _ptr(v_new),
        n, hq, softmax_scale, _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(out), _ptr(lse), _stream(stream)))


def stream_step(ring: Ring, rope: Rope, msk: CMask, q, k_new, v_new, out, workspace,
                lse=None, softmax_scale: float = 0.0, stream=None) -> None:
    """frt_stream_step: stream_attn_step then kv_append, fused."""
    n, hq = q.shape[1], q.shape[2]
    cr, co = ring.c(), rope.c()
    _check(load_library().frt_stream_step(
        ctypes.byref(cr), ctypes.byref(co), ctypes.byref(msk), _ptr(q), _ptr(k_new), _ptr(v_new),
        n, hq, softmax_scale, _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(out), _ptr(lse), _stream(stream)))


def decode_workspace_bytes(ring: Ring, num_q_heads: int) -> int:
    cr = ring.c()
    return load_library().frt_decode_workspace_bytes(ctypes.byref(cr), num_q_heads)


def decode_max_splits(ring: Ring) -> int:
    cr = ring.c()
    return load_library().frt_decode_max_splits(ctypes.byref(cr))


def decode_attn(ring: Ring, rope: Rope, msk: CMask, q, k_new, v_new, out, workspace, lse=None,
                softmax_scale: float = 0.0, stream=None) -> None:
    """frt_decode_attn: one token per stream; q/out bf16 [B][1][Hq][d]."""
    hq = q.shape[2]
    cr, co = ring.c(), rope.c()
    _check(load_library().frt_decode_attn(
        ctypes.byref(cr), ctypes.byref(co), ctypes.byref(msk), _ptr(q), _ptr(k_new), _ptr(v_new),
        hq, softmax_scale, _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(out), _ptr(lse), _stream(stream)))


def decode_step(ring: Ring, rope: Rope, msk: CMask, q, k_new, v_new, out, workspace, lse=None,
                softmax_scale: float = 0.0, stream=None) -> None:
    """frt_decode_step: decode_attn then the one-token kv_append, fused."""
    hq = q.shape[2]
    cr, co = ring.c(), rope.c()
    _check(load_library().frt_decode_step(
        ctypes.byref(cr), ctypes.byref(co), ctypes.byref(msk), _ptr(q), _ptr(k_new), _ptr(v_new),
        hq, softmax_scale, _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(out), _ptr(lse), _stream(stream)))


def decode_step_noalloc(ring: Ring, rope: Rope, msk: CMask, q, k_new, v_new, out, lse=None,
                        softmax_scale: float = 0.0, stream=None) -> None:
    """frt_decode_step_noalloc: decode_step with the library's fixed device scratch
    instead of a workspace (no allocation)."""
    hq = q.shape[2]
    cr, co = ring.c(), rope.c()
    _check(load_library().frt_decode_step_noalloc(
        ctypes.byref(cr), ctypes.byref(co), ctypes.byref(msk), _ptr(q), _ptr(k_new), _ptr(v_new),
        hq, softmax_scale, _ptr(out), _ptr(lse), _stream(stream)))


# ------------------------------------------------------------------ FP8 --
class RingFp8(Ring):
    """An FP8 (e4m3fn) ring: k uint8 [B][Hkv][C][d], v uint8 [B][Hkv][C*d] in
    32-slot blocks, and fp32 [B][Hkv] dequantisation scales k_scale / v_scale."""

    def __init__(self, num_streams: int, num_kv_heads: int, head_dim: int, capacity: int,
                 k_scale, v_scale, device="cuda"):
        import torch
        k = torch.zeros((num_streams, num_kv_heads, capacity, head_dim), dtype=torch.uint8,
                        device=device)
        v = torch.zeros((num_streams, num_kv_heads, capacity * head_dim), dtype=torch.uint8,
                        device=device)
        super().__init__(num_streams, num_kv_heads, head_dim, capacity, device=device, k=k, v=v)
        self.k_scale = k_scale.to(device=device, dtype=torch.float32).contiguous()
        self.v_scale = v_scale.to(device=device, dtype=torch.float32).contiguous()

    def scales(self) -> CFp8Scales:
        return CFp8Scales(_ptr(self.k_scale), _ptr(self.v_scale))

    def view_stream(self, b: int) -> "RingFp8":
        """A one-stream view sharing memory (and scales) with stream b."""
        view = RingFp8.__new__(RingFp8)
        Ring.__init__(view, 1, self.Hkv, self.d, self.C, k=self.k[b:b + 1], v=self.v[b:b + 1],
                      seq_len=self.seq_len[b:b + 1])
        view.k_scale, view.v_scale = self.k_scale[b:b + 1], self.v_scale[b:b + 1]
        return view


def kv_append_fp8(ring: RingFp8, rope: Rope, k_new, v_new, stream=None) -> None:
    """frt_kv_append_fp8: k_new/v_new bf16 [B][n][Hkv][d]."""
    cr, co, cs = ring.c(), rope.c(), ring.scales()
    _check(load_library().frt_kv_append_fp8(ctypes.byref(cr), ctypes.byref(cs), ctypes.byref(co),
                                            _ptr(k_new), _ptr(v_new), k_new.shape[1],
                                            _stream(stream)))


def stream_attn_fp8_workspace_bytes(ring: Ring, n_new: int, num_q_heads: int) -> int:
    cr = ring.c()
    return int(load_library().frt_stream_attn_fp8_workspace_bytes(ctypes.byref(cr), n_new,
                                                                  num_q_heads))


def stream_attn_step_fp8(ring: RingFp8, rope: Rope, msk: CMask, q, k_new, v_new, out, workspace,
                         lse=None, softmax_scale: float = 0.0, stream=None) -> None:
    """frt_stream_attn_step_fp8: q/out bf16 [B][n][Hq][d]."""
    n, hq = q.shape[1], q.shape[2]
    cr, co, cs = ring.c(), rope.c(), ring.scales()
    _check(load_library().frt_stream_attn_step_fp8(
        ctypes.byref(cr), ctypes.byref(cs), ctypes.byref(co), ctypes.byref(msk), _ptr(q),
        _ptr(k_new), _ptr(v_new), n, hq, softmax_scale, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(out), _ptr(lse), _stream(stream)))


def stream_step_fp8(ring: RingFp8, rope: Rope, msk: CMask, q, k_new, v_new, out, workspace,
                    lse=None, softmax_scale: float = 0.0, stream=None) -> None:
    """frt_stream_step_fp8: stream_attn_step_fp8 then kv_append_fp8, fused."""
    n, hq = q.shape[1], q.shape[2]
    cr, co, cs = ring.c(), rope.c(), ring.scales()
    _check(load_library().frt_stream_step_fp8(
        ctypes.byref(cr), ctypes.byref(cs), ctypes.byref(co), ctypes.byref(msk), _ptr(q),
        _ptr(k_new), _ptr(v_new), n, hq, softmax_scale, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(out), _ptr(lse), _stream(stream)))


def decode_fp8_workspace_bytes(ring: RingFp8, num_q_heads: int) -> int:
    cr = ring.c()
    return int(load_library().frt_decode_fp8_workspace_bytes(ctypes.byref(cr), num_q_heads))


def _decode_fp8(fn, ring, rope, msk, q, k_new, v_new, out, workspace, lse, softmax_scale,
                stream):
    hq = q.shape[2]
    cr, co, cs = ring.c(), rope.c(), ring.scales()
    _check(fn(ctypes.byref(cr), ctypes.byref(cs), ctypes.byref(co), ctypes.byref(msk), _ptr(q),
              _ptr(k_new), _ptr(v_new), hq, softmax_scale, _ptr(workspace),
              workspace.numel() * workspace.element_size(), _ptr(out), _ptr(lse),
              _stream(stream)))


def decode_attn_fp8(ring: RingFp8, rope: Rope, msk: CMask, q, k_new, v_new, out, workspace,
                    lse=None, softmax_scale: float = 0.0, stream=None) -> None:
    """frt_decode_attn_fp8: q/out bf16 [B][1][Hq][d], k_new/v_new bf16 [B][1][Hkv][d]."""
    _decode_fp8(load_library().frt_decode_attn_fp8, ring, rope, msk, q, k_new, v_new, out,
                workspace, lse, softmax_scale, stream)


def decode_step_fp8(ring: RingFp8, rope: Rope, msk: CMask, q, k_new, v_new, out, workspace,
                    lse=None, softmax_scale: float = 0.0, stream=None) -> None:
    """frt_decode_step_fp8: decode_attn_fp8 then the one-token kv_append_fp8, fused."""
    _decode_fp8(load_library().frt_decode_step_fp8, ring, rope, msk, q, k_new, v_new, out,
                workspace, lse, softmax_scale, stream)


def timing_enable(on: bool = True) -> None:
    _check(load_library().frt_timing_enable(1 if on else 0))


def timing_query(kernel: str):
    """(count, total_ms) of the recorded launches of `kernel` (waits for them)."""
    c = ctypes.c_int32(0)
    ms = ctypes.c_double(0.0)
    _check(load_library().frt_timing_query(kernel.encode(), ctypes.byref(c), ctypes.byref(ms)))
    return c.value, ms.value


def timing_samples(kernel: str):
    """Durations (ms) of the recorded launches of `kernel`, in launch order."""
    c = ctypes.c_int32(0)
    _check(load_library().frt_timing_samples(kernel.encode(), None, 0, ctypes.byref(c)))
    buf = (ctypes.c_float * max(c.value, 1))()
    _check(load_library().frt_timing_samples(kernel.encode(), buf, c.value, ctypes.byref(c)))
    return [float(buf[i]) for i in range(c.value)]


def timing_reset() -> None:
    load_library().frt_timing_reset()
