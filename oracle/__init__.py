"""CPU oracle for batched policy/value evaluation (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  It shares no code with the GPU library.
"""
from .az_oracle import *  # noqa: F401,F403
from .az_oracle import (forward, forward_quant, conv3x3, softmax_legal, value_head,  # noqa: F401
                        unpack, calibrate_absmax, weight_scales, act_scales_from_absmax,
                        e4m3_round, e4m3_decode, quant_int8, to_bf16)
