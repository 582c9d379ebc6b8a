"""bench.py's output line on the GPU: one JSON object with the fields its
readers rely on (the metric and its unit, the step counts and timing, the
workload, the roofline of the timed kernel and the CPU baseline), for a short
run of the default workload and of the backward mode."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print(f"[bench] {' '.join(args)}", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                       timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    return json.loads(lines[0])


def _check_common(d, steps, warmup):
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
              "scaling", "vs_baseline", "dtype", "data", "config", "roofline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == steps and d["warmup"] == warmup
    assert d["unit"] == "GB/s" and d["higher_is_better"] is True and d["scaling"] == "weak"
    assert d["value"] > 0 and d["ms_per_step"] > 0
    assert isinstance(d["config"].get("workload"), str) and d["config"]["workload"]
    r = d["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in r, k
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-3
    assert r["traffic"] is None or r["traffic"] > 0


def test_default_workload_line():
    # the default workload is c5 (64 int8 row-wise tables, the largest that
    # fits one GPU), with its uniform-index control
    d = _bench("--steps", "20", "--warmup", "3", "--cpu-budget", "1", "--cold-reps", "3", "--uniform-steps", "5")
    _check_common(d, 20, 3)
    assert d["config"]["workload"].startswith("c5")
    assert d["dtype"] == "u8->f32" and d["accumulate"] == "f32"
    assert abs(d["algorithmic_pct_of_peak"] - 100 * d["value"] / 8000.0) < 0.01
    u = d["uniform_control"]
    assert u["index_law"] == "uniform" and u["steps"] == 5 and u["kernel_ms_avg"] > 0
    assert abs(u["frac"] - u["achieved"] / 8000.0) < 1e-3
    assert 0 < u["frac"] <= 1.0  # no reuse: every row comes from HBM
    cb = d["cpu_baseline"]
    for k in ("value", "unit", "cores", "kind", "sample"):
        assert k in cb, k
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1 and cb["unit"] == d["unit"]
    assert isinstance(cb.get("cpu_model"), str) and cb["cpu_model"]
    if cb["cores"] > 1:  # the same sample on one host thread
        one = cb["one_thread"]
        assert one["value"] > 0 and one["lookups_per_s"] > 0 and one["unit"] == d["unit"]


def test_backward_mode_line():
    d = _bench("--mode", "backward", "--config", "c2", "--steps", "5", "--warmup", "2", "--cpu-budget", "0",
               "--cold-reps", "0")
    _check_common(d, 5, 2)
    assert "bwd" in d["metric"] and d["dtype"] == "f32"
    assert d["uniform_control"] is None
