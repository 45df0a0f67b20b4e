"""bench.py's command-line contract on the CPU: more than one GPU is refused with
a message and exit status 2 before anything touches a device; the counter table
names only known workloads, tilings and batches; the roofline peak and FLOP
count are those the documentation derives."""

import os
import subprocess
import sys

import pytest

import azgen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "8"})])
def test_more_than_one_gpu_is_refused(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       env={**os.environ, **env}, timeout=120)
    assert r.returncode == 2, (r.returncode, r.stderr[-500:])
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_counter_table_keys_and_values():
    for (name, tiling, batch), (sha, fetch, write, busy) in bench.COUNTERS.items():
        assert name in azgen.WORKLOADS
        assert tiling in (0, 1, 2, 3) and batch >= 1
        assert len(sha) == 64 and fetch > 0 and write > 0 and 0.0 <= busy <= 1.0


def test_roofline_flop_and_peak_of_the_headline():
    w = azgen.WORKLOADS["net20x128_int8_b1024"]
    flop, peak = bench.roofline_peak(w.shape, w.dtype)
    assert flop == 759_152_896            # 2 x MACs of the layer list, per position
    assert 4.9e15 < peak < 5.0e15         # int8 tower at 5.0 P, stem and heads at bf16 2.5 P, value FC fp32
