"""bench.py's output contract, on a short run of the benchmark workload: one
JSON line on stdout with the metric, the whole-job value, the timing fields,
the roofline of the dominant kernel (bound, achieved / peak = frac), the
reduction figures, the overlap of Sec. 4.1 and a consistent configuration;
--gpus above 1 exits with a message; the attention and linear modes print one
line each.  (Runs bench.py as a child process; its timings are not checked.)"""
import json
import math
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args, timeout=240):
    print("bench.py", *args, flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                       capture_output=True, text=True, timeout=timeout, cwd=ROOT)
    return r


def _line(r):
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    return json.loads(lines[0])


def test_bench_default_line():
    d = _line(_run("--steps", "3", "--warmup", "1", "--no-cpu-baseline"))
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "reduce", "overlap", "kernels"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["unit"] == "TFLOP/s" and d["higher_is_better"] is True and d["dtype"] == "bf16"
    cfg = d["config"]
    assert cfg["workload"] == "wide_h20480_col_8x1" and cfg["mesh"] == [8, 1]
    assert cfg["tokens"] == 4096 and cfg["h"] == 20480 and cfg["chunks"] == 8
    # value is the step's algorithmic FLOP over the measured time
    assert math.isclose(d["value"], cfg["gflop_per_step"] / d["ms_per_step"], rel_tol=2e-3)
    rf = d["roofline"]
    assert rf["bound"] == "mfma" and rf["unit"] == "TFLOP/s" and rf["peak"] == 2500.0
    assert math.isclose(rf["frac"], rf["achieved"] / rf["peak"], rel_tol=1e-3)
    assert 0 < rf["frac"] < 1
    assert rf["flops_per_launch"] > 0 and rf["avg_launch_us"] > 0
    red = d["reduce"]
    assert red["unit"] == "GB/s" and 0 < red["frac"] < 1 and red["alone"]["frac"] < 1
    ov = d["overlap"]
    assert ov["serial_ms"] > 0 and ov["reduce_ms"] > 0
    assert math.isclose(ov["hidden"], (ov["serial_ms"] - ov["pipelined_ms"]) / ov["reduce_ms"],
                        rel_tol=1e-2, abs_tol=1e-3)


def test_bench_refuses_several_gpus():
    r = _run("--gpus", "2")
    assert r.returncode != 0
    assert "one GPU" in r.stderr


def test_bench_attention_and_linear_lines():
    a = _line(_run("--attention", "--steps", "2", "--warmup", "1", "--no-cpu-baseline"))
    assert a["unit"] == "TFLOP/s" and a["value"] > 0
    assert {k["name"] for k in a["kernels"]} == {"attention_fwd", "attention_bwd"}
    lin = _line(_run("--linear", "--steps", "2", "--warmup", "1"))
    assert set(lin["variants"]) == {"chunked_f32", "chunked_f32_serial", "unchunked_f32",
                                    "chunked_bf16_partials", "fused_epilogue"}
    assert lin["value"] == lin["variants"]["chunked_f32"]["ms"]
