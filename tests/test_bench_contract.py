"""bench.py's command-line contract: one GPU only, FP8 only at head_dim 128
(CPU, before any device is touched); and on the GPU, the one JSON line a
short decode run prints, with the fields its readers rely on."""
import contextlib
import io
import json

import pytest

import bench


def _run(argv):
    out, err = io.StringIO(), io.StringIO()
    with contextlib.redirect_stdout(out), contextlib.redirect_stderr(err):
        rc = bench.main(argv)
    return rc, out.getvalue(), err.getvalue()


@pytest.mark.parametrize("n", [0, 2, 8])
def test_more_than_one_gpu_is_refused(n):
    rc, out, err = _run(["--gpus", str(n)])
    assert rc == 2 and out == ""
    assert "one GPU" in err and "--gpus %d" % n in err


def test_world_size_above_one_is_refused(monkeypatch):
    monkeypatch.setenv("WORLD_SIZE", "2")
    rc, out, err = _run([])
    assert rc == 2 and out == "" and "one GPU" in err


def test_fp8_needs_head_dim_128():
    rc, out, err = _run(["--workload", "tiny", "--fp8"])
    assert rc == 2 and out == "" and "head_dim 128" in err


def test_summary_keeps_the_compact_fields():
    line = {"config": {"workload": "decode", "rings": 3}, "dtype": "bf16", "ms_per_step": 0.066,
            "value": 4500.0, "unit": "GB/s", "kernels_us": {"decode_split": 58.0},
            "hot": None,
            "roofline": {"kernel": "decode_split", "launch_us": {"avg_us": 58.0},
                         "achieved": 5100.0, "peak": 8000.0, "frac": 0.6375,
                         "step_frac": 0.5625}}
    s = bench.summary(line)
    assert s["workload"] == "decode" and s["kernel_us"] == 58.0 and s["frac"] == 0.6375
    assert set(s) == {"workload", "dtype", "ms_per_step", "value", "unit", "rings", "kernel",
                      "kernel_us", "achieved", "peak", "frac", "step_frac", "kernels_us", "hot"}


@pytest.mark.gpu
def test_decode_line_fields():
    rc, out, _ = _run(["--workload", "decode", "--steps", "3", "--warmup", "2",
                       "--cpu-seconds", "0", "--no-library", "--no-clock-power"])
    assert rc == 0
    lines = [l for l in out.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 2
    assert d["unit"] == "GB/s" and d["dtype"] == "bf16" and d["higher_is_better"] is True
    assert d["config"]["workload"] == "decode" and d["config"]["rings"] == 3
    assert d["vs_baseline"] is None and d["cpu_baseline"] is None
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == bench.PEAK_HBM_GBS
    assert 0 < r["frac"] < 1 and abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-9
    assert 0 < d["value"] <= r["achieved"] * 1.001  # the whole step is slower than its split pass
    assert abs(d["ms_per_step"] * 1e-3 * d["value"] * 1e9 / 1e6
               - d["config"]["step_min_mb"]) < 1e-3 * d["config"]["step_min_mb"]
