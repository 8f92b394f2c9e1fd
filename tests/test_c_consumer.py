"""The C ABI from plain C: tests/c/frt_consumer.c compiles with gcc as C99
against include/frt.h alone (-Wall -Wextra -Werror -pedantic), links
libfrt.so, and runs the host-side calls that need no GPU (status strings,
sizes, the rotary table, argument validation)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_18171_amd")


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


# The invalid-argument calls pass fake (never dereferenced) device addresses;
# like the ctypes ABI tests they run only where no GPU is visible.
@pytest.mark.skipif(shutil.which("gcc") is None, reason="no C compiler")
@pytest.mark.skipif(_gpu_visible(), reason="fake pointers: CPU-only check")
def test_c99_consumer_compiles_links_and_runs(tmp_path):
    if not os.path.exists(os.path.join(PKG, "libfrt.so")):
        pytest.fail("libfrt.so is not built (run __graft_entry__.build())")
    exe = str(tmp_path / "frt_consumer")
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "frt_consumer.c"),
                    "-L", PKG, "-lfrt", "-Wl,-rpath," + PKG, "-o", exe],
                   check=True, capture_output=True, text=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "ok: 0 failure(s)" in res.stdout
