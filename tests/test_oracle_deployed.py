"""Pins of the deployed-network oracle (global pooling, from-to policy head, WDL
value head) against facts it does not compute itself:

* parameter counts the paper prints (the from-to head's 50,048 parameters on a
  128-channel trunk; the 97,020 parameters a 32-channel value reduction adds over
  the 2-channel one; the 6.32 million parameters of the final model);
* textbook counts of the action encoding and an independent ray-walking
  enumeration of it;
* loop nests written from the definitions of pooling and of the from-to logits;
* torch's conv2d / linear / matmul / softmax in float64 on the CPU for the whole
  network;
* closed forms (zero heads, zero pooling projection) and convergence of the
  int8 network to the float one as its grid becomes fine.
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as TF

import azgen
from oracle import az_oracle as O
from oracle import deployed as OD


def _rng(seed=0):
    return np.random.Generator(np.random.PCG64(seed))


def _spec(**kw):
    base = dict(in_planes=52, blocks=2, filters=16, policy_planes=0, value_hidden=12, value_conv_relu=1,
                act_cap=6.0, pool_every=2, policy_head="fromto", token_dim=8, value_head="wdl",
                value_channels=2)
    base.update(kw)
    return azgen.NetShape(**base)


def _inputs(spec, n, seed):
    rng = _rng(seed)
    planes = azgen.make_planes_52(n, (4, 20), rng) if spec.in_planes == 52 else \
        rng.standard_normal((n, spec.in_planes, 8, 8))
    legal = (rng.random((n, spec.n_moves)) < 0.05).astype(np.uint8)
    legal[:, 0] = 1
    return planes, legal


# --------------------------------------------------------------------------- #
# Action encoding
# --------------------------------------------------------------------------- #
def _walk_pairs():
    """Origin-destination pairs by walking the eight rays to the board edge and
    the eight knight jumps from every square."""
    out = set()
    rays = [(1, 0), (-1, 0), (0, 1), (0, -1), (1, 1), (1, -1), (-1, 1), (-1, -1)]
    jumps = [(1, 2), (2, 1), (-1, 2), (-2, 1), (1, -2), (2, -1), (-1, -2), (-2, -1)]
    for r in range(8):
        for c in range(8):
            for dr, dc in rays:
                rr, cc = r + dr, c + dc
                while 0 <= rr < 8 and 0 <= cc < 8:
                    out.add((r * 8 + c, rr * 8 + cc))
                    rr, cc = rr + dr, cc + dc
            for dr, dc in jumps:
                rr, cc = r + dr, c + dc
                if 0 <= rr < 8 and 0 <= cc < 8:
                    out.add((r * 8 + c, rr * 8 + cc))
    return out


def test_action_table_counts_order_and_enumeration():
    tab = OD.action_table()
    assert tab.shape == (1880, 3) and OD.N_ACTIONS == 1880
    pairs, promos = tab[tab[:, 2] < 0], tab[tab[:, 2] >= 0]
    assert len(pairs) == 1792 and len(promos) == 88              # Section 3.5, Appendix D
    assert np.all(tab[:1792, 2] < 0) and np.all(tab[1792:, 2] >= 0)
    assert {(int(f), int(t)) for f, t, _ in pairs} == _walk_pairs()
    # a queen on an empty board has 1,456 moves in total, a knight 336
    knight = [(f, t) for f, t, _ in pairs
              if sorted((abs(f // 8 - t // 8), abs(f % 8 - t % 8))) == [1, 2]]
    assert len(knight) == 336 and len(pairs) - len(knight) == 1456
    # corner a1 (square 0): 21 ray + 2 knight destinations; d4 (row 3, col 3): 27 + 8
    assert int(np.sum(pairs[:, 0] == 0)) == 23 and int(np.sum(pairs[:, 0] == 27)) == 35
    # promotions: 22 pawn steps from the seventh to the eighth row, four pieces each
    steps = {(int(f), int(t)) for f, t, _ in promos}
    assert len(steps) == 22
    for f, t in steps:
        assert f // 8 == 6 and t // 8 == 7 and abs(f % 8 - t % 8) <= 1
    assert all(sorted(promos[(promos[:, 0] == f) & (promos[:, 1] == t), 2].tolist()) == [0, 1, 2, 3]
               for f, t in steps)
    keys = [tuple(r) for r in tab[:1792, :2]] + [tuple(r) for r in tab[1792:]]
    assert keys[:1792] == sorted(keys[:1792]) and keys[1792:] == sorted(keys[1792:])
    assert len(set(map(tuple, tab))) == 1880


# --------------------------------------------------------------------------- #
# Parameter counts printed in the paper
# --------------------------------------------------------------------------- #
def _sizes(spec):
    W = OD.unpack(spec, np.zeros(spec.weight_count()))
    return {k: v.size for k, v in W.items()}


def test_fromto_head_has_50048_parameters_on_a_128_channel_trunk():
    # Section 4.3 "Three policy representations": 50,048 head parameters
    s = _sizes(_spec(filters=128, token_dim=128))
    assert sum(s[k] for k in ("embed.w", "embed.b", "query.w", "query.b", "key.w", "key.b", "promo.w")) == 50048


def test_value_reduction_of_32_channels_adds_97020_parameters():
    # Section 4.3 "Value and training-only heads": a 32-channel reduction adds 97,020
    # parameters over the retained 2-channel one (160-channel trunk, 48 hidden
    # units).  The training model normalises the reduction (gamma and beta per
    # channel) where the folded blob has one bias per channel: one more per channel.
    def head(v):
        s = _sizes(_spec(filters=160, value_channels=v, value_hidden=48))
        return sum(s[k] for k in ("value.w", "value.b", "fc1.w", "fc1.b", "fc2.w", "fc2.b")) + v
    assert head(32) - head(2) == 97020


def test_final_model_has_6_32_million_parameters():
    # Table "Final training run": 6.32 million.  Training form of the deployed
    # blob: every convolution normalised (one extra parameter per output channel),
    # plus the two training-only heads (a second from-to head for the next searched
    # policy and a value-shaped head with one output for the remaining length).
    # A plain 14-block tower without the split pooling blocks would have 6.66 M.
    spec = azgen.DEPLOYED_14X160
    s = _sizes(spec)
    folded = sum(s.values())
    bn = spec.filters * (1 + 2 * spec.blocks) + spec.value_channels
    ft = sum(s[k] for k in ("embed.w", "embed.b", "query.w", "query.b", "key.w", "key.b", "promo.w"))
    length = s["value.w"] + 2 * spec.value_channels + s["fc1.w"] + s["fc1.b"] + spec.value_hidden + 1
    total = folded + bn + ft + length
    assert total == 6320876 and round(total / 1e4) / 100 == 6.32
    assert folded == azgen.DEPLOYED_14X160.weight_count() == 6255525


# --------------------------------------------------------------------------- #
# Loop nests from the definitions
# --------------------------------------------------------------------------- #
def _act(v, cap):
    return min(max(v, 0.0), cap) if cap > 0 else max(v, 0.0)


def _conv_loops(x, w, b):
    B, C = x.shape[:2]
    F = w.shape[0]
    y = np.zeros((B, F, 8, 8))
    for n in range(B):
        for f in range(F):
            for r in range(8):
                for c in range(8):
                    s = b[f]
                    for i in range(C):
                        for dy in range(3):
                            for dx in range(3):
                                rr, cc = r + dy - 1, c + dx - 1
                                if 0 <= rr < 8 and 0 <= cc < 8:
                                    s += w[f, i, dy, dx] * x[n, i, rr, cc]
                    y[n, f, r, c] = s
    return y


def test_pooling_block_matches_loops():
    spec = _spec(in_planes=5, filters=8, blocks=2)
    blob = azgen.make_weights(spec, 3, alpha_fold=True, bf16=False)
    W = OD.unpack(spec, blob)
    x = _rng(4).standard_normal((2, 5, 8, 8))
    cap = spec.act_cap
    h = np.vectorize(lambda v: _act(v, cap))(_conv_loops(x, W["stem.w"], W["stem.b"]))
    # block 0: plain
    t = np.vectorize(lambda v: _act(v, cap))(_conv_loops(h, W["w1.0"], W["b1.0"]))
    h = np.vectorize(lambda v: _act(v, cap))(h + _conv_loops(t, W["w2.0"], W["b2.0"]))
    # block 1: pooling; pooled channels 6, 7; regular 0..5
    z = _conv_loops(h, W["w1.1"], W["b1.1"])
    t = np.zeros((2, 6, 8, 8))
    for n in range(2):
        feats = []
        for ch in (6, 7):
            vals = [_act(z[n, ch, r, c], cap) for r in range(8) for c in range(8)]
            feats.append(sum(vals) / 64.0)
        for ch in (6, 7):
            feats.append(max(_act(z[n, ch, r, c], cap) for r in range(8) for c in range(8)))
        for f in range(6):
            bias = sum(W["pool.1"][f, k] * feats[k] for k in range(4))
            for r in range(8):
                for c in range(8):
                    t[n, f, r, c] = _act(z[n, f, r, c] + bias, cap)
    h = np.vectorize(lambda v: _act(v, cap))(h + _conv_loops(t, W["w2.1"], W["b2.1"]))
    np.testing.assert_allclose(OD.tower(spec, W, x), h, rtol=0, atol=1e-12)


def test_fromto_logits_match_loops():
    spec = _spec(in_planes=5, filters=6, blocks=1, token_dim=4)
    blob = azgen.make_weights(spec, 8, alpha_fold=False, bf16=False)
    W = OD.unpack(spec, blob)
    h = _rng(5).random((1, 6, 8, 8)) * 3.0
    z = OD.fromto_logits(spec, W, h)[0]
    tok = np.zeros((64, 4))
    for s in range(64):
        for d in range(4):
            tok[s, d] = max(W["embed.b"][d] + sum(W["embed.w"][d, f] * h[0, f, s // 8, s % 8] for f in range(6)), 0.0)
    Q = np.array([[W["query.b"][d] + sum(W["query.w"][d, e] * tok[s, e] for e in range(4)) for d in range(4)]
                  for s in range(64)])
    K = np.array([[W["key.b"][d] + sum(W["key.w"][d, e] * tok[s, e] for e in range(4)) for d in range(4)]
                  for s in range(64)])
    for a, (f, t, k) in enumerate(OD.action_table()):
        want = sum(Q[f, d] * K[t, d] for d in range(4)) / 2.0     # sqrt(token_dim) = 2
        if k >= 0:
            want += sum(W["promo.w"][k, d] * K[t, d] for d in range(4))
        assert abs(z[a] - want) < 1e-12, a


# --------------------------------------------------------------------------- #
# Whole network against torch (float64, CPU)
# --------------------------------------------------------------------------- #
def _torch_deployed(spec, blob, planes, legal):
    W = {k: torch.from_numpy(np.array(v)) for k, v in OD.unpack(spec, blob).items()}
    x = torch.from_numpy(np.asarray(planes, dtype=np.float64))
    cap = spec.act_cap
    F = spec.filters
    Fr = F - F // 4

    def a(t):
        return torch.clamp(torch.relu(t), max=cap)

    h = a(TF.conv2d(x, W["stem.w"], W["stem.b"], padding=1))
    for j in range(spec.blocks):
        z = TF.conv2d(h, W[f"w1.{j}"], W[f"b1.{j}"], padding=1)
        if j % 2 == 1:
            p = a(z[:, Fr:])
            g = torch.cat([TF.adaptive_avg_pool2d(p, 1).flatten(1), TF.adaptive_max_pool2d(p, 1).flatten(1)], 1)
            t = a(z[:, :Fr] + TF.linear(g, W[f"pool.{j}"])[:, :, None, None])
        else:
            t = a(z)
        h = a(h + TF.conv2d(t, W[f"w2.{j}"], W[f"b2.{j}"], padding=1))
    tok = torch.relu(TF.conv2d(h, W["embed.w"][:, :, None, None], W["embed.b"]).flatten(2).transpose(1, 2))
    Q = TF.linear(tok, W["query.w"], W["query.b"])
    K = TF.linear(tok, W["key.w"], W["key.b"])
    S = torch.matmul(Q, K.transpose(1, 2).contiguous()) / math.sqrt(spec.token_dim)
    promo = TF.linear(K[:, 56:, :], W["promo.w"])                  # [B, 8, 4]
    logits = []
    for f, t, k in OD.action_table():                             # gather written per action
        v = S[:, f, t]
        if k >= 0:
            v = v + promo[:, t - 56, k]
        logits.append(v)
    z = torch.stack(logits, 1)
    m = torch.from_numpy(np.asarray(legal) != 0)
    P = torch.nan_to_num(torch.softmax(z.masked_fill(~m, -math.inf), 1), nan=0.0)
    u = torch.relu(TF.conv2d(h, W["value.w"][:, :, None, None], W["value.b"])).flatten(1)
    y = torch.relu(TF.linear(u, W["fc1.w"], W["fc1.b"]))
    wdl = torch.softmax(TF.linear(y, W["fc2.w"], W["fc2.b"]), 1)
    return P.numpy(), (wdl[:, 0] - wdl[:, 2]).numpy(), wdl.numpy()


@pytest.mark.parametrize("filters,blocks", [(16, 2), (12, 4)])
def test_deployed_forward_matches_torch(filters, blocks):
    spec = _spec(filters=filters, blocks=blocks)
    blob = azgen.make_weights(spec, 11 + blocks, alpha_fold=True, bf16=False)
    planes, legal = _inputs(spec, 5, 12)
    legal[3] = 0                                                   # a row without legal actions
    P, V, WDL = OD.forward(spec, blob, planes, legal)
    Pt, Vt, WDLt = _torch_deployed(spec, blob, planes, legal)
    np.testing.assert_allclose(P, Pt, rtol=0, atol=1e-12)
    np.testing.assert_allclose(V, Vt, rtol=0, atol=1e-12)
    np.testing.assert_allclose(WDL, WDLt, rtol=0, atol=1e-12)
    assert np.all(P[3] == 0.0)


# --------------------------------------------------------------------------- #
# Closed forms and invariants
# --------------------------------------------------------------------------- #
def _zeroed(spec, blob, prefixes):
    blob = np.array(blob, dtype=np.float64)
    off = 0
    for name, shp in spec.layer_sizes():
        n = int(np.prod(shp))
        if any(name.startswith(p) for p in prefixes):
            blob[off:off + n] = 0.0
        off += n
    return blob


def test_zero_heads_give_uniform_policy_and_even_wdl():
    spec = _spec()
    blob = azgen.make_weights(spec, 21, alpha_fold=True, bf16=False)
    blob = _zeroed(spec, blob, ("embed.", "query.", "key.", "promo.", "fc2."))
    planes, legal = _inputs(spec, 4, 22)
    P, V, WDL = OD.forward(spec, blob, planes, legal)
    for i in range(4):
        m = legal[i] != 0
        np.testing.assert_allclose(P[i, m], 1.0 / m.sum(), rtol=0, atol=1e-15)
        assert np.all(P[i, ~m] == 0.0)
    np.testing.assert_allclose(WDL, 1.0 / 3.0, rtol=0, atol=1e-15)
    assert np.all(V == 0.0)


def test_zero_pooling_projection_is_a_plain_block_on_the_regular_channels():
    # with Wg = 0 a pooling block is an ordinary block whose first convolution
    # keeps its first F - F/4 outputs: the pooled channels are the last quarter
    spec = _spec(in_planes=7, filters=16, blocks=2)
    blob = _zeroed(spec, azgen.make_weights(spec, 31, alpha_fold=True, bf16=False), ("block1.pool",))
    W = OD.unpack(spec, blob)
    x = _rng(32).standard_normal((3, 7, 8, 8))
    cap = spec.act_cap
    h = O.act(O.conv3x3(x, W["stem.w"], W["stem.b"]), cap)
    t = O.act(O.conv3x3(h, W["w1.0"], W["b1.0"]), cap)
    h = O.act(h + O.conv3x3(t, W["w2.0"], W["b2.0"]), cap)
    t = O.act(O.conv3x3(h, W["w1.1"][:12], W["b1.1"][:12]), cap)
    h = O.act(h + O.conv3x3(t, W["w2.1"], W["b2.1"]), cap)
    np.testing.assert_allclose(OD.tower(spec, W, x), h, rtol=0, atol=1e-13)


def test_wdl_and_policy_invariants():
    spec = _spec()
    blob = azgen.make_weights(spec, 41, alpha_fold=True, bf16=False)
    planes, legal = _inputs(spec, 6, 42)
    P, V, WDL = OD.forward(spec, blob, planes, legal)
    np.testing.assert_allclose(WDL.sum(1), 1.0, rtol=0, atol=1e-14)
    assert np.all(WDL > 0) and np.all(np.abs(V) <= 1.0)
    np.testing.assert_allclose(V, WDL[:, 0] - WDL[:, 2], rtol=0, atol=0)
    np.testing.assert_allclose(P.sum(1), 1.0, rtol=0, atol=1e-13)
    assert np.all(P[legal == 0] == 0.0)
    # positions are independent: permuting the batch permutes the outputs
    perm = np.array([5, 3, 1, 0, 2, 4])
    Pp, Vp, Wp = OD.forward(spec, blob, planes[perm], legal[perm])
    np.testing.assert_array_equal(Pp, P[perm])
    np.testing.assert_array_equal(Vp, V[perm])


# --------------------------------------------------------------------------- #
# int8 network
# --------------------------------------------------------------------------- #
def test_quant_deployed_converges_to_float_and_codes_are_exact():
    spec = _spec(filters=16, blocks=2)
    blob = azgen.make_weights(spec, 51, alpha_fold=True, bf16=True)
    planes, legal = _inputs(spec, 6, 52)
    P, V, WDL = OD.forward(spec, blob, planes, legal)
    ws = OD.weight_scales(spec, blob)
    acts = np.full(2 * spec.blocks + 1, 6.0 / 127.0, dtype=np.float32)
    rec = []
    Pq, Vq, Wq = OD.forward_quant(spec, blob, ws, acts, planes, legal, record=rec)
    assert len(rec) == 2 * spec.blocks + 1
    assert rec[2].shape[1] == 16 and rec[3].shape[1] == 12       # pooling block's t: regular channels
    for q in rec:
        assert np.all(q == np.rint(q)) and np.all(q >= 0) and np.all(q <= 127)
    assert np.abs(Pq - P).max() < 0.1 and np.abs(Vq - V).max() < 0.1
    # int8 definition with a 128x finer grid and far saturation: rounding only
    old = O.INT8_MAX
    try:
        O.INT8_MAX = 127.0 * 256
        Pf, Vf, Wf = OD.forward_quant(spec, blob, ws / np.float32(128.0),
                                      (acts / np.float32(128.0)).astype(np.float32), planes, legal)
    finally:
        O.INT8_MAX = old
    assert np.abs(Pf - P).max() < 2e-3 and np.abs(Vf - V).max() < 2e-3 and np.abs(Wf - WDL).max() < 2e-3


def test_quant_pool_bias_is_the_float_pooling_of_dequantised_values():
    # pool_bias on exact integer accumulators is the pooling of act(acc * m + b):
    # board means and maxima, projected (written here with explicit loops)
    rng = _rng(61)
    acc = rng.integers(-3000, 3000, size=(3, 4, 8, 8)).astype(np.float32)
    m = np.float32(1.0 / 512.0) * (1 + rng.random(4)).astype(np.float32)
    b = rng.standard_normal(4).astype(np.float32)
    Wg = rng.standard_normal((5, 8))
    c = OD.pool_bias(acc, m, b, 6.0, Wg)
    for n in range(3):
        feats = []
        for ch in range(4):
            vals = [min(max(float(acc[n, ch, r, q]) * float(m[ch]) + float(b[ch]), 0.0), 6.0)
                    for r in range(8) for q in range(8)]
            feats.append((sum(vals) / 64.0, max(vals)))
        g = [f[0] for f in feats] + [f[1] for f in feats]
        for o in range(5):
            want = sum(Wg[o, i] * g[i] for i in range(8))
            assert abs(c[n, o] - want) <= 1e-12 * (1 + abs(want))
