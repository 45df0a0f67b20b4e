"""Seeded synthetic workloads for batched policy/value evaluation of search leaves.

This module is shared by the tests, the benchmark and the oracle's callers.  It
draws inputs and weights and lays them out in the canonical blob order; it holds
none of the method's arithmetic (no convolution, activation, softmax, value head
or quantisation).

What the inputs stand in for.  The paper evaluates real self-play leaf
positions encoded as side-to-move planes (Appendix D, Table D.1, planes 0-11 are
the twelve piece-location masks), with legal-move masks from a chess rules
engine, on trained weights.  None of those exist here, so:

* planes 0-11: a one-hot piece encoding.  A position holds n pieces,
  n ~ U{lo..hi}, on n distinct squares drawn uniformly without replacement; each
  occupied square gets one of the 12 piece planes uniformly.  No chess legality
  is imposed.
* planes 12..in_planes-1: each plane is independently all-zero or all-one with
  probability 1/2 (the constant flag planes of Table D.1, rows 12-15).
* legal mask: k ~ U{20..40} distinct legal indices of the 73*64 = 4672 move-plane
  cells, one byte per cell, 1 = legal.
* weights: N(0, 2/fan_in) (fan_in = C_in*3*3 for 3x3 convs, C_in for 1x1 convs,
  in_features for linear layers); biases N(0, 0.1^2) stand in for folded
  batch-norm shifts.  Optionally each residual block's second convolution and
  its bias are multiplied by alpha = 1/sqrt(blocks), the residual-branch scale
  that Section 4.3 ("Quantization as an architectural constraint") folds into
  the second convolution at export.  For the reduced-precision workloads every
  weight is then rounded to the nearest bfloat16 (ties to even), so that the
  oracle and the GPU library see the same bf16-valued network.

Random generator: numpy PCG64.  Seeds: weights 1000+k, inputs 2000+k,
calibration positions 3000+k, where k is the workload's index (1..5).
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, Tuple

import numpy as np

N_SQUARES = 64
N_PIECE_PLANES = 12


@dataclasses.dataclass(frozen=True)
class NetShape:
    """Layer list of the residual policy/value network (canonical blob order)."""

    in_planes: int
    blocks: int
    filters: int
    policy_planes: int
    value_hidden: int
    value_conv_relu: int = 0
    act_cap: float = 0.0

    @property
    def n_moves(self) -> int:
        return self.policy_planes * N_SQUARES

    def layer_sizes(self):
        """(name, shape) for every array of the blob, in blob order."""
        C, F, P, H = self.in_planes, self.filters, self.policy_planes, self.value_hidden
        out = [("stem.w", (F, C, 3, 3)), ("stem.b", (F,))]
        for j in range(self.blocks):
            out += [(f"block{j}.w1", (F, F, 3, 3)), (f"block{j}.b1", (F,)),
                    (f"block{j}.w2", (F, F, 3, 3)), (f"block{j}.b2", (F,))]
        out += [("policy.w", (P, F)), ("policy.b", (P,)),
                ("value.w", (1, F)), ("value.b", (1,)),
                ("fc1.w", (H, N_SQUARES)), ("fc1.b", (H,)),
                ("fc2.w", (1, H)), ("fc2.b", (1,))]
        return out

    def weight_count(self) -> int:
        return int(sum(int(np.prod(s)) for _, s in self.layer_sizes()))

    def n_quant_convs(self) -> int:
        return 2 * self.blocks

    def n_act_scales(self) -> int:
        return 2 * self.blocks + 1


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int            # k in the seed scheme
    shape: NetShape
    dtype: str            # "f32" | "bf16" | "int8" | "fp8"
    batch: int
    pieces: Tuple[int, int]
    alpha_fold: bool
    legal: Tuple[int, int] = (20, 40)

    @property
    def weight_seed(self) -> int:
        return 1000 + self.index

    @property
    def input_seed(self) -> int:
        return 2000 + self.index

    @property
    def calib_seed(self) -> int:
        return 3000 + self.index


def _shape(blocks, filters, hidden):
    return NetShape(in_planes=20, blocks=blocks, filters=filters, policy_planes=73,
                    value_hidden=hidden)


WORKLOADS: Dict[str, Workload] = {
    w.name: w for w in [
        Workload("tiny_2x32_f32_b16", 1, _shape(2, 32, 64), "f32", 16, (16, 32), False),
        Workload("net20x128_bf16_b32", 2, _shape(20, 128, 128), "bf16", 32, (16, 32), True),
        Workload("net20x128_bf16_b256", 3, _shape(20, 128, 128), "bf16", 256, (2, 32), True),
        Workload("net20x128_int8_b1024", 4, _shape(20, 128, 128), "int8", 1024, (16, 32), True),
        Workload("net20x128_fp8_b1024", 4, _shape(20, 128, 128), "fp8", 1024, (16, 32), True),
        Workload("net20x128_bf16_b1024", 4, _shape(20, 128, 128), "bf16", 1024, (16, 32), True),
        Workload("net24x256_bf16_b1024", 5, _shape(24, 256, 128), "bf16", 1024, (16, 32), True),
    ]
}


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (ties to even), returned as float32.  Input handling
    only: it makes weights exactly representable in the GPU's storage format."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    bits = (bits + 0x7FFF + ((bits >> 16) & 1)) & 0xFFFF0000
    return bits.astype(np.uint32).view(np.float32).reshape(x.shape)


def make_weights(shape: NetShape, seed: int, alpha_fold: bool, bf16: bool) -> np.ndarray:
    """Flat float32 weight blob in canonical order (see NetShape.layer_sizes)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    alpha = 1.0 / math.sqrt(shape.blocks) if alpha_fold else 1.0
    parts = []
    for name, shp in shape.layer_sizes():
        if len(shp) == 1:                       # biases
            a = rng.standard_normal(shp) * 0.1
        elif len(shp) == 4:
            a = rng.standard_normal(shp) * math.sqrt(2.0 / (shp[1] * 9))
        else:
            a = rng.standard_normal(shp) * math.sqrt(2.0 / shp[1])
        if ".w2" in name or ".b2" in name:
            a = a * alpha
        parts.append(a.astype(np.float32).ravel())
    blob = np.concatenate(parts)
    if bf16:
        blob = round_to_bf16(blob)
    assert blob.size == shape.weight_count()
    return blob


def make_planes(n: int, in_planes: int, pieces: Tuple[int, int], rng) -> np.ndarray:
    planes = np.zeros((n, in_planes, 8, 8), dtype=np.float32)
    lo, hi = pieces
    for i in range(n):
        k = int(rng.integers(lo, hi + 1))
        sq = rng.choice(N_SQUARES, size=k, replace=False)
        pc = rng.integers(0, N_PIECE_PLANES, size=k)
        planes[i, pc, sq // 8, sq % 8] = 1.0
        n_const = in_planes - N_PIECE_PLANES
        if n_const > 0:
            bits = rng.integers(0, 2, size=n_const).astype(np.float32)
            planes[i, N_PIECE_PLANES:, :, :] = bits[:, None, None]
    return planes


def make_legal(n: int, n_moves: int, legal: Tuple[int, int], rng) -> np.ndarray:
    mask = np.zeros((n, n_moves), dtype=np.uint8)
    lo, hi = legal
    for i in range(n):
        k = int(rng.integers(lo, hi + 1))
        mask[i, rng.choice(n_moves, size=k, replace=False)] = 1
    return mask


def make_inputs(w: Workload, n: int | None = None, seed: int | None = None):
    """(planes [n,C,8,8] f32, legal [n,P*64] u8) for a workload."""
    n = w.batch if n is None else n
    rng = np.random.Generator(np.random.PCG64(w.input_seed if seed is None else seed))
    planes = make_planes(n, w.shape.in_planes, w.pieces, rng)
    legal = make_legal(n, w.shape.n_moves, w.legal, rng)
    return planes, legal


def make_calibration_planes(w: Workload, n: int = 512) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(w.calib_seed))
    return make_planes(n, w.shape.in_planes, w.pieces, rng)


def workload_weights(w: Workload, alpha_fold: bool | None = None) -> np.ndarray:
    fold = w.alpha_fold if alpha_fold is None else alpha_fold
    return make_weights(w.shape, w.weight_seed, fold, bf16=(w.dtype != "f32"))
