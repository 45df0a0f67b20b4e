"""Plain CPU oracle for the paper's deployed policy/value network.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module; the GPU library never does.

What it computes.  The network the paper serves (Section 3.5 "Chess
representation and outputs", Section 4.3 "Convolution, attention, and global
context", "Value and training-only heads", "Three policy representations",
Appendix D "Network input and output contract"), on top of the residual tower of
az_oracle:

  stem, blocks   as in az_oracle (capped activation, residual scale folded into
                 the second convolution), except that every second block (blocks
                 1, 3, 5, ...) is a global-pooling block:
                   z  = conv3x3(h) + b1                     (F output channels)
                   p  = act(z[Fr:F])                       (the last F/4 channels)
                   g  = [mean over squares of p, max over squares of p]   (2 F/4)
                   c  = Wg g                               (Fr = F - F/4 biases)
                   t  = act(z[0:Fr] + c)                   (the regular channels)
                   h' = act(h + conv3x3(t) + b2)           (second conv reads Fr channels)
  from-to head   tok[s] = relu(We h[:, s] + be)            (128-wide token per square)
                 Q[s] = Wq tok[s] + bq,  K[s] = Wk tok[s] + bk
                 S[f, t] = Q[f] . K[t] / sqrt(128)          (origin f, destination t)
                 O[c, k] = Wp[k] . K[56 + c]               (promotion offsets, last-row
                                                            destination c, piece k)
                 logit(pair f->t) = S[f, t];  logit(promotion f->t, k) = S[f, t] + O[t-56, k]
                 P = softmax of the 1,880 logits over the legal actions
  WDL head       u = relu(Wv h + bv)                        (2 channels x 64 squares)
                 y = relu(W1 u + b1)                        (48 units; u flattened channel-major)
                 (W, D, L) = softmax(W2 y + b2),  V = W - L

The action order (action_table) and every other point the paper leaves open are
the readings listed with this implementation's design notes: pooled channels are
the last quarter of the first convolution's outputs, the token projection is
followed by ReLU, promotion offsets are read from the destination square's key
and are not scaled, pairs are ordered by (origin, destination) and promotions by
(origin, destination, piece Q R B N).

Modes.
  forward(...)        float64 definition (parity reference for the bf16 path).
  forward_quant(...)  the int8 network, the plain definition in float64:
                      residual convolutions on int8 codes as in
                      az_oracle.forward_quant; the pooling step in floating
                      point (Section 4.3: context operations stay in floating
                      point inside the INT8 trunk): the pooled channels'
                      activations, their means and maxima and the projection c
                      in float64, c added to the regular channels before their
                      activation and requantisation; heads in floating point.
"""

from __future__ import annotations

import math

import numpy as np

from .az_oracle import N_SQUARES, act, conv3x3, quantize_weights, requant, softmax_legal, to_bf16

N_PAIRS = 1792
N_PROMOS = 88
N_ACTIONS = N_PAIRS + N_PROMOS


# --------------------------------------------------------------------------- #
# Action encoding (Section 3.5; Appendix D)
# --------------------------------------------------------------------------- #
def action_table():
    """[1880, 3] int array of (origin, destination, promotion piece or -1).

    Squares are row * 8 + column in the side-to-move frame (row 0 the player's
    home rank).  Pairs: every origin-destination pair on a common row, column or
    diagonal, or a knight's jump apart, in ascending (origin, destination) order.
    Promotions: origin on row 6, destination on row 7 at most one column away,
    four pieces each (0 queen, 1 rook, 2 bishop, 3 knight), in ascending
    (origin, destination, piece) order."""
    rows = []
    for f in range(64):
        fr, fc = divmod(f, 8)
        for t in range(64):
            if t == f:
                continue
            tr, tc = divmod(t, 8)
            dr, dc = abs(tr - fr), abs(tc - fc)
            if dr == 0 or dc == 0 or dr == dc or (dr, dc) in ((1, 2), (2, 1)):
                rows.append((f, t, -1))
    for fc in range(8):
        for tc in range(max(fc - 1, 0), min(fc + 1, 7) + 1):
            for k in range(4):
                rows.append((48 + fc, 56 + tc, k))
    return np.array(rows, dtype=np.int64)


# --------------------------------------------------------------------------- #
# Weight blob (canonical order)
# --------------------------------------------------------------------------- #
def is_pool_block(spec, j):
    e = getattr(spec, "pool_every", 0)
    return bool(e) and j % e == e - 1


def unpack(spec, blob):
    """Named float64 arrays of a canonical blob:
    stem W[F][C][3][3], b[F]; per block W1[F][F][3][3], b1[F], (pooling blocks:
    Wg[Fr][2 F/4]), W2[F][K][3][3] (K = Fr in pooling blocks, else F), b2[F];
    from-to head We[D][F], be[D], Wq[D][D], bq[D], Wk[D][D], bk[D], Wp[4][D] (or
    the move-plane head W[P][F], b[P]); WDL head Wv[V][F], bv[V], W1[H][V*64],
    b1[H], W2[3][H], b2[3] (or the scalar head of az_oracle)."""
    C, F, P, H = spec.in_planes, spec.filters, spec.policy_planes, spec.value_hidden
    g = F // 4 if getattr(spec, "pool_every", 0) else 0
    Fr = F - g
    blob = np.asarray(blob, dtype=np.float64).ravel()
    sizes = [("stem.w", (F, C, 3, 3)), ("stem.b", (F,))]
    for j in range(spec.blocks):
        pool = is_pool_block(spec, j)
        sizes += [(f"w1.{j}", (F, F, 3, 3)), (f"b1.{j}", (F,))]
        if pool:
            sizes += [(f"pool.{j}", (Fr, 2 * g))]
        sizes += [(f"w2.{j}", (F, Fr if pool else F, 3, 3)), (f"b2.{j}", (F,))]
    if getattr(spec, "policy_head", "planes") == "fromto":
        D = spec.token_dim
        sizes += [("embed.w", (D, F)), ("embed.b", (D,)), ("query.w", (D, D)), ("query.b", (D,)),
                  ("key.w", (D, D)), ("key.b", (D,)), ("promo.w", (4, D))]
    else:
        sizes += [("policy.w", (P, F)), ("policy.b", (P,))]
    if getattr(spec, "value_head", "tanh") == "wdl":
        V = spec.value_channels
        sizes += [("value.w", (V, F)), ("value.b", (V,)), ("fc1.w", (H, V * N_SQUARES)), ("fc1.b", (H,)),
                  ("fc2.w", (3, H)), ("fc2.b", (3,))]
    else:
        sizes += [("value.w", (1, F)), ("value.b", (1,)), ("fc1.w", (H, N_SQUARES)), ("fc1.b", (H,)),
                  ("fc2.w", (1, H)), ("fc2.b", (1,))]
    out, off = {}, 0
    for name, shp in sizes:
        n = int(np.prod(shp))
        out[name] = blob[off:off + n].reshape(shp)
        off += n
    if off != blob.size:
        raise ValueError(f"blob has {blob.size} values, layer list needs {off}")
    return out


# --------------------------------------------------------------------------- #
# Global pooling (Section 4.3 "Convolution, attention, and global context")
# --------------------------------------------------------------------------- #
def pool_features(p):
    """[B, 2 g] board means then board maxima of p [B, g, 8, 8], float64."""
    ps = np.asarray(p, dtype=np.float64).reshape(p.shape[0], p.shape[1], N_SQUARES)
    return np.concatenate([ps.sum(axis=2) / N_SQUARES, ps.max(axis=2)], axis=1)


# --------------------------------------------------------------------------- #
# Float network
# --------------------------------------------------------------------------- #
def tower(spec, W, x, record=None):
    """Stem and blocks in float64; record receives h0, t0, h1, t1, ..., h_N
    (t of a pooling block: its Fr regular channels)."""
    cap = spec.act_cap
    F = spec.filters
    h = act(conv3x3(x, W["stem.w"], W["stem.b"]), cap)
    if record is not None:
        record.append(h)
    for j in range(spec.blocks):
        z = conv3x3(h, W[f"w1.{j}"], W[f"b1.{j}"])
        if is_pool_block(spec, j):
            Fr = F - F // 4
            c = pool_features(act(z[:, Fr:], cap)) @ W[f"pool.{j}"].T
            t = act(z[:, :Fr] + c[:, :, None, None], cap)
        else:
            t = act(z, cap)
        if record is not None:
            record.append(t)
        h = act(h + conv3x3(t, W[f"w2.{j}"], W[f"b2.{j}"]), cap)
        if record is not None:
            record.append(h)
    return h


def fromto_logits(spec, W, h):
    """[B, 1880] action logits of the from-to head."""
    B, F = h.shape[:2]
    D = spec.token_dim
    hs = np.asarray(h, dtype=np.float64).reshape(B, F, N_SQUARES).transpose(0, 2, 1)   # [B, 64, F]
    tok = np.maximum(hs @ W["embed.w"].T + W["embed.b"], 0.0)                         # [B, 64, D]
    Q = tok @ W["query.w"].T + W["query.b"]
    K = tok @ W["key.w"].T + W["key.b"]
    S = Q @ K.transpose(0, 2, 1) / math.sqrt(D)                                        # [B, f, t]
    O = K[:, 56:64, :] @ W["promo.w"].T                                                # [B, 8, 4]
    tab = action_table()
    z = S[:, tab[:, 0], tab[:, 1]]
    pr = tab[:, 2] >= 0
    z[:, pr] += O[:, tab[pr, 1] - 56, tab[pr, 2]]
    return z


def wdl_head(spec, W, h):
    """(WDL [B, 3], V [B]) of the WDL value head."""
    B, F = h.shape[:2]
    hs = np.asarray(h, dtype=np.float64).reshape(B, F, N_SQUARES)
    u = np.einsum("cf,bfs->bcs", W["value.w"], hs) + W["value.b"][None, :, None]
    if spec.value_conv_relu:
        u = np.maximum(u, 0.0)
    y = np.maximum(u.reshape(B, -1) @ W["fc1.w"].T + W["fc1.b"], 0.0)
    z = y @ W["fc2.w"].T + W["fc2.b"]
    e = np.exp(z - z.max(axis=1, keepdims=True))
    wdl = e / e.sum(axis=1, keepdims=True)
    return wdl, wdl[:, 0] - wdl[:, 2]


def heads(spec, W, h, legal):
    """(P [B, 1880], V [B], WDL [B, 3])."""
    P = softmax_legal(fromto_logits(spec, W, h), legal)
    wdl, V = wdl_head(spec, W, h)
    return P, V, wdl


def forward(spec, blob, planes, legal):
    """Policy over the 1,880 actions, scalar value W - L and (W, D, L), float64."""
    W = unpack(spec, blob)
    h = tower(spec, W, np.asarray(planes, dtype=np.float64))
    return heads(spec, W, h, legal)


def calibrate_absmax(spec, blob, planes, chunk=64):
    """Per-tensor absolute maxima of h0, t0, h1, ..., h_N over a calibration set."""
    W = unpack(spec, blob)
    amax = np.zeros(2 * spec.blocks + 1)
    for s in range(0, planes.shape[0], chunk):
        rec = []
        tower(spec, W, np.asarray(planes[s:s + chunk], dtype=np.float64), record=rec)
        amax = np.maximum(amax, [np.abs(a).max() for a in rec])
    return amax


# --------------------------------------------------------------------------- #
# int8 network
# --------------------------------------------------------------------------- #
def weight_scales(spec, blob, fmt="int8"):
    """Per-output-channel absmax scales of the 2 N residual convolutions (F rows
    each), float32."""
    from .az_oracle import qmax
    W = unpack(spec, blob)
    out = []
    for j in range(spec.blocks):
        for key in (f"w1.{j}", f"w2.{j}"):
            a = np.abs(W[key]).reshape(spec.filters, -1).max(axis=1) / qmax(fmt)
            out.append(np.where(a > 0, a, 1.0))
    return np.concatenate(out).astype(np.float32)


def pool_bias(acc, m_in, b, cap, Wg):
    """Pooled-context biases of one pooling block of the int8 network: the pooled
    channels' activations p = act(acc * m_in + b) (m_in = a_in * s_w per channel,
    acc the exact sum of code products), their board means and maxima and the
    projection c = Wg [mean, max], all float64 (Section 4.3: the context
    operations stay in floating point inside the INT8 trunk).
    acc: [B, g, 8, 8]; returns [B, Fr]."""
    bc = lambda v: np.asarray(v, dtype=np.float64)[None, :, None, None]  # noqa: E731
    p = act(np.asarray(acc, dtype=np.float64) * bc(m_in) + bc(b), cap)
    return pool_features(p) @ np.asarray(Wg, dtype=np.float64).T


def forward_quant(spec, blob, w_scales, act_scales, planes, legal, record=None):
    """int8 deployed network, the plain definition in float64.  Codes, scales and
    requantisation as in az_oracle.forward_quant; in a pooling block the first
    convolution's output y = acc * a[n] * s_w[f] + b1[f] splits into
        pooled channels   p = act(y[Fr:])  (floating point, never quantised),
                          c = pool_bias(...) = Wg [mean p, max p]
        regular channels  q = sat(rne(act(y[:Fr] + c) / a[n+1]))
    and the second convolution reads the Fr regular channels only."""
    fmt = "int8"
    F, nb = spec.filters, spec.blocks
    Fr = F - F // 4
    W = unpack(spec, blob)
    sw = np.asarray(w_scales, dtype=np.float32).astype(np.float64).reshape(2 * nb, F)
    a = np.asarray(act_scales, dtype=np.float32).astype(np.float64)
    cap = spec.act_cap
    bc = lambda v: v[None, :, None, None]  # noqa: E731

    x = to_bf16(np.asarray(planes, dtype=np.float64))
    q = requant(conv3x3(x, W["stem.w"], W["stem.b"]), a[0], cap, fmt)
    if record is not None:
        record.append(q)
    for j in range(nb):
        q_in = q
        pool = is_pool_block(spec, j)
        # first convolution
        n = 2 * j
        acc = conv3x3(q, quantize_weights(W[f"w1.{j}"], sw[n], fmt))
        y = acc * a[n] * bc(sw[n]) + bc(W[f"b1.{j}"])
        if pool:
            c = pool_bias(acc[:, Fr:], a[n] * sw[n][Fr:], W[f"b1.{j}"][Fr:], cap, W[f"pool.{j}"])
            q = requant(y[:, :Fr] + c[:, :, None, None], a[n + 1], cap, fmt)
        else:
            q = requant(y, a[n + 1], cap, fmt)
        if record is not None:
            record.append(q)
        # second convolution (+ residual)
        n = 2 * j + 1
        acc = conv3x3(q, quantize_weights(W[f"w2.{j}"], sw[n], fmt))
        y = acc * a[n] * bc(sw[n]) + bc(W[f"b2.{j}"]) + q_in * a[n - 1]
        q = requant(y, a[n + 1], cap, fmt)
        if record is not None:
            record.append(q)
    h = q * a[2 * nb]
    return heads(spec, W, h, legal)
