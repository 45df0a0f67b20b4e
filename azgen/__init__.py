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
* the same flag conditions the deployed network's heads: the token embedding
  (weights and bias) is multiplied by 1/4 and the WDL output layer by 1/8.
  Drawn literally, the seeded from-to logits have a spread of about 13 (a
  one-hot policy) and the value saturates at 1; conditioned, the logits have a
  spread of about 1 and the values are spread over (-1, 1), as a trained
  network's are.

* the deployed network's 52 planes follow the structure of Table D.1 (see
  make_planes_52), and its legal mask covers the 1,880 from-to actions.

Random generator: numpy PCG64.  Seeds: weights 1000+k, inputs 2000+k,
calibration positions 3000+k, where k is the workload's index (1..6).
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, Tuple

import numpy as np

N_SQUARES = 64
N_PIECE_PLANES = 12


N_FROMTO_ACTIONS = 1880   # 1,792 ray / knight origin-destination pairs + 88 promotions

# conditioning of the deployed network's seeded heads (see the module notes)
HEAD_EMBED_SCALE = 0.25
WDL_OUT_SCALE = 0.125


@dataclasses.dataclass(frozen=True)
class NetShape:
    """Layer list of the residual policy/value network (canonical blob order).

    The deployed network of the paper adds three options: global-pooling blocks
    (pool_every = 2: blocks 1, 3, 5, ... split their first convolution into
    filters - filters/4 regular and filters/4 pooled output channels, project the
    pooled channels' board means and maxima back as biases on the regular ones,
    and run the second convolution on the regular channels), the from-to policy
    head (policy_head = "fromto": token, query and key projections of width
    token_dim and four promotion offsets, 1,880 actions) and the WDL value head
    (value_head = "wdl": value_channels 1x1 channels, a hidden layer of
    value_hidden units, three outputs)."""

    in_planes: int
    blocks: int
    filters: int
    policy_planes: int
    value_hidden: int
    value_conv_relu: int = 0
    act_cap: float = 0.0
    pool_every: int = 0
    policy_head: str = "planes"
    token_dim: int = 128
    value_head: str = "tanh"
    value_channels: int = 1

    @property
    def n_moves(self) -> int:
        if self.policy_head == "fromto":
            return N_FROMTO_ACTIONS
        return self.policy_planes * N_SQUARES

    @property
    def pool_channels(self) -> int:
        return self.filters // 4 if self.pool_every else 0

    def is_pool_block(self, j: int) -> bool:
        return bool(self.pool_every) and j % self.pool_every == self.pool_every - 1

    def layer_sizes(self):
        """(name, shape) for every array of the blob, in blob order."""
        C, F, P, H = self.in_planes, self.filters, self.policy_planes, self.value_hidden
        out = [("stem.w", (F, C, 3, 3)), ("stem.b", (F,))]
        for j in range(self.blocks):
            if self.is_pool_block(j):
                g = self.pool_channels
                out += [(f"block{j}.w1", (F, F, 3, 3)), (f"block{j}.b1", (F,)),
                        (f"block{j}.pool", (F - g, 2 * g)),
                        (f"block{j}.w2", (F, F - g, 3, 3)), (f"block{j}.b2", (F,))]
            else:
                out += [(f"block{j}.w1", (F, F, 3, 3)), (f"block{j}.b1", (F,)),
                        (f"block{j}.w2", (F, F, 3, 3)), (f"block{j}.b2", (F,))]
        if self.policy_head == "fromto":
            D = self.token_dim
            out += [("embed.w", (D, F)), ("embed.b", (D,)), ("query.w", (D, D)), ("query.b", (D,)),
                    ("key.w", (D, D)), ("key.b", (D,)), ("promo.w", (4, D))]
        else:
            out += [("policy.w", (P, F)), ("policy.b", (P,))]
        if self.value_head == "wdl":
            V = self.value_channels
            out += [("value.w", (V, F)), ("value.b", (V,)),
                    ("fc1.w", (H, V * N_SQUARES)), ("fc1.b", (H,)),
                    ("fc2.w", (3, H)), ("fc2.b", (3,))]
        else:
            out += [("value.w", (1, F)), ("value.b", (1,)),
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


# The paper's deployed network (Section 3.5, Appendix D): 52 input planes, 14
# blocks of 160 channels with ReLU6 and global pooling in every second block,
# from-to policy head with 128-wide tokens, WDL head with two 1x1 channels
# (followed by ReLU) and 48 hidden units.
DEPLOYED_14X160 = NetShape(in_planes=52, blocks=14, filters=160, policy_planes=0, value_hidden=48,
                           value_conv_relu=1, act_cap=6.0, pool_every=2, policy_head="fromto",
                           token_dim=128, value_head="wdl", value_channels=2)


WORKLOADS: Dict[str, Workload] = {
    w.name: w for w in [
        Workload("tiny_2x32_f32_b16", 1, _shape(2, 32, 64), "f32", 16, (16, 32), False),
        Workload("net20x128_bf16_b32", 2, _shape(20, 128, 128), "bf16", 32, (16, 32), True),
        Workload("net20x128_bf16_b256", 3, _shape(20, 128, 128), "bf16", 256, (2, 32), True),
        Workload("net20x128_int8_b1024", 4, _shape(20, 128, 128), "int8", 1024, (16, 32), True),
        Workload("net20x128_fp8_b1024", 4, _shape(20, 128, 128), "fp8", 1024, (16, 32), True),
        Workload("net20x128_bf16_b1024", 4, _shape(20, 128, 128), "bf16", 1024, (16, 32), True),
        Workload("net24x256_bf16_b1024", 5, _shape(24, 256, 128), "bf16", 1024, (16, 32), True),
        Workload("deployed14x160_int8_b1024", 6, DEPLOYED_14X160, "int8", 1024, (16, 32), True),
        Workload("deployed14x160_bf16_b1024", 6, DEPLOYED_14X160, "bf16", 1024, (16, 32), True),
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
        if alpha_fold and name.startswith("embed."):
            a = a * HEAD_EMBED_SCALE
        if alpha_fold and shape.value_head == "wdl" and name.startswith("fc2."):
            a = a * WDL_OUT_SCALE
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


def make_planes_52(n: int, pieces: Tuple[int, int], rng) -> np.ndarray:
    """Inputs with the structure of the paper's 52-plane encoding (Appendix D,
    Table D.1), drawn at random with no chess legality: planes 0-11 one-hot
    pieces as in make_planes; 12-15 castling flags (constant 0/1); 16-17 own /
    opponent occupancy of the drawn pieces; 18 up to two checker squares among
    the opponent's pieces; 19 an en-passant square on row 5 with probability 1/4;
    20-21 repetition flags (21 only with 20); 22-37 origin/destination masks of
    the m ~ U{0..8} most recent moves, older entries zero; 38 the fixed
    checkerboard with row 0, column 0 set; 39 a constant flag; 40-45 own minus
    opponent piece counts per type; 46 a halfmove clock ~ U{0..100}; 47-51 own
    pawn, knight, bishop, rook and queen counts.  Planes 40-51 hold unnormalised
    integers, as in the paper."""
    planes = np.zeros((n, 52, 8, 8), dtype=np.float32)
    lo, hi = pieces
    rows, cols = np.indices((8, 8))
    board = ((rows + cols) % 2 == 0).astype(np.float32)
    for i in range(n):
        k = int(rng.integers(lo, hi + 1))
        sq = rng.choice(N_SQUARES, size=k, replace=False)
        pc = rng.integers(0, N_PIECE_PLANES, size=k)
        pl = planes[i]
        pl[pc, sq // 8, sq % 8] = 1.0
        pl[12:16] = rng.integers(0, 2, size=4).astype(np.float32)[:, None, None]
        pl[16] = pl[0:6].max(axis=0)
        pl[17] = pl[6:12].max(axis=0)
        opp = np.flatnonzero(pl[17].ravel())
        n_chk = min(int(rng.integers(0, 3)), opp.size)
        for s in rng.choice(opp, size=n_chk, replace=False):
            pl[18, s // 8, s % 8] = 1.0
        if rng.integers(0, 4) == 0:
            pl[19, 5, int(rng.integers(0, 8))] = 1.0
        rep1 = int(rng.integers(0, 2))
        pl[20] = rep1
        pl[21] = rep1 * int(rng.integers(0, 2))
        for mv in range(int(rng.integers(0, 9))):
            o, d = rng.choice(N_SQUARES, size=2, replace=False)
            pl[22 + 2 * mv, o // 8, o % 8] = 1.0
            pl[23 + 2 * mv, d // 8, d % 8] = 1.0
        pl[38] = board
        pl[39] = int(rng.integers(0, 2))
        own = pl[0:6].sum(axis=(1, 2))
        their = pl[6:12].sum(axis=(1, 2))
        pl[40:46] = (own - their)[:, None, None]
        pl[46] = int(rng.integers(0, 101))
        pl[47:52] = own[:5, None, None]
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
    planes = _planes(n, w.shape.in_planes, w.pieces, rng)
    legal = make_legal(n, w.shape.n_moves, w.legal, rng)
    return planes, legal


def _planes(n, in_planes, pieces, rng):
    if in_planes == 52:
        return make_planes_52(n, pieces, rng)
    return make_planes(n, in_planes, pieces, rng)


def make_calibration_planes(w: Workload, n: int = 512) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(w.calib_seed))
    return _planes(n, w.shape.in_planes, w.pieces, rng)


def workload_weights(w: Workload, alpha_fold: bool | None = None) -> np.ndarray:
    fold = w.alpha_fold if alpha_fold is None else alpha_fold
    return make_weights(w.shape, w.weight_seed, fold, bf16=(w.dtype != "f32"))
