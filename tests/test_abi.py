"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before launching anything (CPU only: no kernel runs)."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import oracle
import paper_2607_18171_amd as frt
from paper_2607_18171_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Invalid-argument calls use fake (never dereferenced) device addresses: they
# must fail host validation. They are not run where a GPU is visible.
no_gpu = pytest.mark.skipif(torch.cuda.is_available(), reason="fake pointers: CPU-only check")

FAKE = 0x10000000


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "frt.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(frt_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = frt.load_library()
    names = declared_symbols()
    assert len(names) == 24
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(B.EXPORTS) == names


def test_status_strings():
    lib = frt.load_library()
    for code in range(8):
        assert lib.frt_status_str(code)


def ring(B_=1, H=2, d=128, C=64, k=FAKE, v=FAKE + 4096, s=FAKE + 8192):
    return B.CRing(B_, H, d, C, k, v, s)


def rope(mode=B.ROPE_1D, dims=(128, 0, 0), maxpos=(100, 0, 0), table=FAKE + 12288):
    return B.CRope(mode, (ctypes.c_int32 * 3)(*dims), (ctypes.c_int32 * 2)(0, 0),
                   (ctypes.c_int32 * 3)(*maxpos), 10000.0, table)


def call_append(r, o, k=FAKE, v=FAKE, n=16):
    return frt.load_library().frt_kv_append(ctypes.byref(r), ctypes.byref(o), k, v, n, None)


def call_step(r, o, m, n=16, hq=2, ws=FAKE, wsb=1 << 30, out=FAKE, q=FAKE):
    return frt.load_library().frt_stream_attn_step(
        ctypes.byref(r), ctypes.byref(o), ctypes.byref(m), q, FAKE, FAKE, n, hq, 0.0, ws, wsb,
        out, None, None)


@no_gpu
@pytest.mark.parametrize("r,code", [
    (ring(d=96), 3), (ring(d=0), 2), (ring(C=60), 5), (ring(C=0), 2), (ring(k=0), 1),
    (ring(B_=0), 2), (ring(k=FAKE + 2), 5), (ring(s=0), 1),
    (ring(C=8388608), 2),  # 2^31 bytes of K per head at head_dim 128: one block past the limit
])
def test_append_rejects_bad_ring(r, code):
    assert call_append(r, rope()) == code
    assert frt.load_library().frt_last_error()


@no_gpu
def test_append_rejects_bad_sizes_and_rope():
    assert call_append(ring(), rope(), n=65) == 4                      # n > capacity
    assert call_append(ring(), rope(), n=-1) == 2
    assert call_append(ring(), rope(), n=0) == 0                       # no-op
    assert call_append(ring(), rope(), k=0) == 1
    assert call_append(ring(), rope(dims=(130, 0, 0))) == 2            # wider than head_dim
    assert call_append(ring(), rope(dims=(7, 0, 0))) == 2              # odd
    assert call_append(ring(), rope(table=0)) == 1
    assert call_append(ring(), rope(maxpos=(0, 0, 0))) == 2
    bad3d = B.CRope(B.ROPE_3D, (ctypes.c_int32 * 3)(44, 42, 42), (ctypes.c_int32 * 2)(0, 52),
                    (ctypes.c_int32 * 3)(4, 30, 52), 10000.0, FAKE)
    assert call_append(ring(), bad3d) == 2                             # frame height 0


@no_gpu
def test_step_rejects_bad_arguments():
    m = B.CMask(B.MASK_BLOCK_CAUSAL, 16, 3)
    assert call_step(ring(), rope(), m, hq=3) == 2                     # Hq % Hkv
    assert call_step(ring(), rope(), B.CMask(B.MASK_BLOCK_CAUSAL, 16, 5)) == 4  # 5*16 > 64
    assert call_step(ring(), rope(), B.CMask(B.MASK_CAUSAL, 0, 66)) == 4       # 65 > 64
    assert call_step(ring(), rope(), B.CMask(3, 1, 0)) == 2
    assert call_step(ring(), rope(), B.CMask(B.MASK_BLOCK_CAUSAL, 0, 0)) == 2
    assert call_step(ring(), rope(), m, n=65) == 4
    assert call_step(ring(), rope(), m, ws=0) == 6
    assert call_step(ring(), rope(), m, wsb=100) == 6
    assert call_step(ring(), rope(), m, out=0) == 1
    assert call_step(ring(), rope(), m, q=FAKE + 8) == 5
    assert call_step(ring(), rope(), m, n=0) == 0


@no_gpu
def test_decode_rejects_bad_arguments():
    lib = frt.load_library()
    r = ring(H=1)
    m = B.CMask(B.MASK_CAUSAL, 0, 0)
    o = rope()
    wsb = lib.frt_decode_workspace_bytes(ctypes.byref(r), 8)
    # piece waves: the resident count (2048) plus one per (stream, KV head),
    # rounded up to blocks of 4; the workspace adds one own-token partial per
    # head (a partial: max[8], sum[8], out[8][128] floats)
    waves = lib.frt_decode_max_splits(ctypes.byref(r))
    assert waves == (2048 + 1 + 3) // 4 * 4
    assert wsb == (waves + 1) * (16 + 8 * 128) * 4

    for fn in (lib.frt_decode_attn, lib.frt_decode_step):
        def dec(hq=8, ws=FAKE, n=wsb):
            return fn(ctypes.byref(r), ctypes.byref(o), ctypes.byref(m), FAKE, FAKE, FAKE, hq, 0.0,
                      ws, n, FAKE, None, None)
        assert dec(hq=17) == 3
        assert dec(ws=0) == 6
        assert dec(n=wsb - 4) == 6


def test_workspace_sizes():
    lib = frt.load_library()
    r = ring(B_=1, H=12, d=128, C=18720)
    got = lib.frt_stream_attn_workspace_bytes(ctypes.byref(r), 4680, 12)
    n_pad = 4736
    # rotated queries, own keys, own values (each a multiple of 256 bytes here),
    # then one int64 per stream, rounded up to 256 bytes
    expect = 4680 * 12 * 128 * 2 + 2 * (12 * n_pad * 128 * 2) + 256
    assert got == expect


def test_rope_table_fill_matches_oracle_bitwise():
    """Host-side table: fp32(cos/sin(pos * base^(-2i/D))) equals the oracle's table."""
    lib = frt.load_library()
    for mode, dims, hw, maxpos in [(B.ROPE_1D, (128, 0, 0), (0, 0), (9000, 0, 0)),
                                   (B.ROPE_1D, (64, 0, 0), (0, 0), (300, 0, 0)),
                                   (B.ROPE_3D, (44, 42, 42), (30, 52), (31, 30, 52))]:
        c = B.CRope(mode, (ctypes.c_int32 * 3)(*dims), (ctypes.c_int32 * 2)(*hw),
                    (ctypes.c_int32 * 3)(*maxpos), 10000.0, None)
        nbytes = lib.frt_rope_table_bytes(ctypes.byref(c))
        buf = np.zeros(nbytes // 4, np.float32)
        assert lib.frt_rope_table_fill(ctypes.byref(c), buf.ctypes.data, nbytes) == 0
        off = 0
        naxes = 1 if mode == B.ROPE_1D else 3
        for a in range(naxes):
            D, npos = dims[a], maxpos[a]
            cs, sn = oracle.rope_cos_sin(D, 10000.0, np.arange(npos))
            blk = buf[off:off + npos * (D // 2) * 2].reshape(npos, D // 2, 2)
            assert np.array_equal(blk[..., 0], cs) and np.array_equal(blk[..., 1], sn)
            off += npos * (D // 2) * 2
        assert off == buf.size
        assert lib.frt_rope_table_fill(ctypes.byref(c), buf.ctypes.data, nbytes - 4) == 2


def test_kernel_code_hash_finds_the_measured_kernels():
    """bench.py keys recorded HBM traffic on the dominant kernels' machine code:
    each must be found in the built library's gfx950 code objects."""
    import bench
    lib = frt.binding.LIB_PATH
    if not os.path.exists(lib):
        pytest.skip("library not built")
    hashes = {k: bench.kernel_code_sha256(k, lib) for k in bench.KERNEL_SYMBOLS}
    assert all(h is not None and len(h) == 64 for h in hashes.values()), hashes
    assert len(set(hashes.values())) == len(hashes)
