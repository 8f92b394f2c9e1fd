"""The measurement probes that bench.py times beside the kernels
(libfrt_probe.so, no part of the attention library): the library loads,
exports its three entry points, and rejects bad arguments before launching
anything (CPU); on the GPU the streaming read runs and leaves its sink alone."""
import ctypes
import os

import pytest
import torch

from paper_2607_18171_amd.build import PROBE_LIB

HIP_INVALID_VALUE = 1
FAKE = 0x10000000

no_gpu = pytest.mark.skipif(torch.cuda.is_available(), reason="fake pointers: CPU-only check")


def _lib():
    if not os.path.exists(PROBE_LIB):
        pytest.fail("%s is not built (run __graft_entry__.build())" % PROBE_LIB)
    lib = ctypes.CDLL(PROBE_LIB)
    lib.frt_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                   ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    lib.frt_probe_read.restype = ctypes.c_int
    for f in (lib.frt_probe_mfma_bf16, lib.frt_probe_mfma_fp8):
        f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                      ctypes.c_void_p]
        f.restype = ctypes.c_int
    return lib


def test_probe_exports():
    lib = _lib()
    for name in ("frt_probe_mfma_bf16", "frt_probe_mfma_fp8", "frt_probe_read"):
        assert hasattr(lib, name), name


@no_gpu
@pytest.mark.parametrize("args", [
    (None, 4096, FAKE, 8, 8),       # no source
    (FAKE, 4096, None, 8, 8),       # no sink
    (FAKE, 0, FAKE, 8, 8),          # nothing to read
    (FAKE, 4100, FAKE, 8, 8),       # not whole 16-byte words
    (FAKE, 4096, FAKE, 0, 8),       # empty grid
    (FAKE, 4096, FAKE, 8, 3),       # unsupported loads per thread
])
def test_probe_read_rejects_bad_arguments(args):
    assert _lib().frt_probe_read(*args, None) == HIP_INVALID_VALUE


@no_gpu
@pytest.mark.parametrize("args", [(None, FAKE, 4, 8), (FAKE, None, 4, 8), (FAKE, FAKE, 0, 8),
                                  (FAKE, FAKE, 4, 6)])
def test_probe_mfma_rejects_bad_arguments(args):
    lib = _lib()
    assert lib.frt_probe_mfma_bf16(*args, None) == HIP_INVALID_VALUE
    assert lib.frt_probe_mfma_fp8(*args, None) == HIP_INVALID_VALUE


@pytest.mark.gpu
@pytest.mark.parametrize("blocks,unroll", [(1, 2), (7, 4), (64, 8), (300, 16)])
def test_probe_read_runs(blocks, unroll):
    """Grid-stride and one-pass shapes over a buffer that is not a multiple of
    any of them: the call succeeds and, on random data, writes nothing."""
    lib = _lib()
    g = torch.Generator(device="cuda").manual_seed(1)
    src = torch.randint(0, 1 << 62, ((3 << 20) // 8 + 6,), device="cuda", dtype=torch.int64,
                        generator=g)
    sink = torch.zeros(blocks, device="cuda", dtype=torch.int32)
    rc = lib.frt_probe_read(src.data_ptr(), src.numel() * 8, sink.data_ptr(), blocks, unroll,
                            torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert rc == 0
    assert int(sink.abs().sum()) == 0
