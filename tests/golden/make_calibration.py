"""Writes the stored quantisation scales of the seeded 20x128 network
(weights seed 1004, residual scale 1/sqrt(20), bf16-valued) used by bench.py.

Scales: absmax over 512 seeded calibration positions (seed 3004) of every
activation tensor h0, t0, ..., h20 on the oracle's float64 network, and per
output channel absmax of every residual-conv weight; divided by 127 (int8) or
448 (fp8 e4m3).  Only the oracle computes them.

    python tests/golden/make_calibration.py
"""

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import azgen  # noqa: E402
from oracle import az_oracle as O  # noqa: E402

WORKLOAD = "net20x128_int8_b1024"
OUT = os.path.join(HERE, "calib_net20x128_seed1004.npz")


def main():
    w = azgen.WORKLOADS[WORKLOAD]
    blob = azgen.workload_weights(w)
    amax = O.calibrate_absmax(w.shape, blob, azgen.make_calibration_planes(w))
    out = {"absmax": amax}
    for fmt in ("int8", "fp8"):
        out[f"w_scales_{fmt}"] = O.weight_scales(w.shape, blob, fmt)
        out[f"act_scales_{fmt}"] = O.act_scales_from_absmax(amax, fmt)
    np.savez(OUT, **out)
    print(f"wrote {OUT}")


if __name__ == "__main__":
    main()
