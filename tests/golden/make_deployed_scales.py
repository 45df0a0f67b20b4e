"""Writes the stored int8 scales of the seeded deployed network (14 blocks of
160 channels, weights seed 1006, residual scale 1/sqrt(14) and conditioned
heads, bf16-valued) used by bench.py.

Scales: per output channel absmax of every residual-conv weight divided by 127
(computed by the oracle), and the fixed activation scale 6/127 of every tensor
between layers: with the ReLU6 cap every activation lies in [0, 6], so the
capped network needs no activation calibration (Section 4.3, "Quantization as
an architectural constraint").

    python tests/golden/make_deployed_scales.py
"""

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import azgen  # noqa: E402
from oracle import deployed as OD  # noqa: E402

WORKLOAD = "deployed14x160_int8_b1024"
OUT = os.path.join(HERE, "scales_deployed14x160_seed1006.npz")


def main():
    w = azgen.WORKLOADS[WORKLOAD]
    blob = azgen.workload_weights(w)
    ws = OD.weight_scales(w.shape, blob, "int8")
    acs = np.full(2 * w.shape.blocks + 1, 6.0 / 127.0, dtype=np.float32)
    np.savez(OUT, w_scales_int8=ws, act_scales_int8=acs)
    print(f"wrote {OUT}")


if __name__ == "__main__":
    main()
