"""bench.py's output line on the GPU (a short run in a child process): one JSON
object with the fields of the measurement contract, a consistent roofline and
valid outputs."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.gpu


def test_bench_line_fields():
    print("case bench.py --steps 5 --warmup 2", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "5", "--warmup", "2",
                        "--no-cpu-baseline", "--no-pipeline", "--no-graph"],
                       capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
              "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "settle"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 5 and d["warmup"] == 2
    assert d["unit"] == "positions/s" and d["higher_is_better"] is True and d["scaling"] == "weak"
    assert d["dtype"] == "int8" and "synthetic" in d["data"] and d["vs_baseline"] is None
    assert d["config"]["workload"] == "net20x128_int8_b1024" and d["config"]["batch"] == 1024
    assert d["value"] > 0 and abs(d["value"] * d["ms_per_step"] * 1e-3 - 1024) < 1e-6 * 1024
    rf = d["roofline"]
    assert rf["bound"] == "mfma" and rf["unit"] == "TFLOP/s" and 0.0 < rf["frac"] < 1.0
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-9
    assert rf["traffic"] is None or rf["traffic"] > 0
    assert rf["mfma_busy"] is None or 0.0 < rf["mfma_busy"] < 1.0
    assert d["outputs_valid"] is True
    assert d["settle"]["seconds"] > 0 and d["settle"]["calls"] > 0
    print(f"  {d['ms_per_step'] * 1e3:.1f} us per batch, frac {rf['frac']:.3f}", flush=True)
