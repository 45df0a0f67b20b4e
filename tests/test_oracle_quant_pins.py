"""Pins of the oracle's quantised networks against exact rational arithmetic.

The int8 / fp8 networks are defined by their quantisation (Section 5.3
"Inference runtimes and precision": explicit quantise / dequantise operations
around INT8 trunk convolutions, the start block and heads at higher precision;
Section 4.3 "Quantization as an architectural constraint" for the block and the
capped activation; Section 4.3 "Convolution, attention, and global context" for
the pooling that stays in floating point).  Here that definition is written a
second time, per element, as loop nests over Python Fractions: every product,
sum, rescale and division is exact and every rounding is taken on an exact
rational value (round half to even; e4m3 by its grid).  The oracle works in
float64, so its codes must equal these exactly, except at an exact tie, which
the rational version reports and the check then allows either way.

A plausible slip in the oracle (the residual or bias dropped, a scale taken from
the wrong tensor, per-input instead of per-output weight scales, the activation
before the residual add, saturation or the cap missed, truncation instead of
rounding, the pooled context added after the activation, the mean or maximum of
the wrong channels) changes codes on these nets and fails.
"""

from fractions import Fraction as Fr

import numpy as np
import pytest
import torch
import torch.nn.functional as TF

import azgen
from oracle import az_oracle as O
from oracle import deployed as OD


# --------------------------------------------------------------------------- #
# exact quantisers
# --------------------------------------------------------------------------- #
class Tie(Exception):
    pass


TIES = []


def _rne(x: Fr) -> int:
    if (x - x.__floor__()) == Fr(1, 2):
        TIES.append(x)
    return round(x)          # Fraction.__round__: half to even


def _e4m3(x: Fr) -> Fr:
    """Nearest e4m3fn value of an exact rational, ties to even, saturating."""
    if x == 0:
        return Fr(0)
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fr(2) ** e > a:
        e -= 1
    e = max(e, -6)
    step = Fr(2) ** (e - 3)
    r = min(_rne(a / step) * step, Fr(448))
    return r if x > 0 else -r


def _code(x: Fr, fmt) -> Fr:
    if fmt == "int8":
        return Fr(max(-127, min(127, _rne(x))))
    return _e4m3(x)


def _act(y: Fr, cap) -> Fr:
    y = max(y, Fr(0))
    return min(y, Fr(float(cap))) if cap else y


def _conv(xq, wq, bias=None):
    """xq[b][c][64] (Fractions or ints), wq[f][c][3][3] -> [b][f][64], exact."""
    B, C, F = len(xq), len(xq[0]), len(wq)
    out = [[[Fr(0)] * 64 for _ in range(F)] for _ in range(B)]
    for b in range(B):
        for f in range(F):
            for r in range(8):
                for col in range(8):
                    s = Fr(0) if bias is None else bias[f]
                    for c in range(C):
                        for dy in range(3):
                            for dx in range(3):
                                rr, cc = r + dy - 1, col + dx - 1
                                if 0 <= rr < 8 and 0 <= cc < 8:
                                    v = xq[b][c][rr * 8 + cc]
                                    if v:
                                        s += wq[f][c][dy][dx] * v
                    out[b][f][r * 8 + col] = s
    return out


def _frac(a):
    return [_frac(x) for x in a] if isinstance(a, (list, np.ndarray)) and np.ndim(a) > 0 else Fr(float(a))


def _rational_tower(spec, W, planes, ws, acs, fmt, pool_every=0):
    """Codes h0, t0, h1, ..., h_N of the quantised network in exact arithmetic."""
    F, nb, cap = spec.filters, spec.blocks, spec.act_cap
    a = [Fr(float(v)) for v in np.asarray(acs, np.float32)]
    sw = np.asarray(ws, np.float32).reshape(2 * nb, F)
    x = [[[Fr(float(v)) for v in O.to_bf16(planes[b, c]).ravel()] for c in range(planes.shape[1])]
         for b in range(planes.shape[0])]
    y = _conv(x, _frac(W["stem.w"]), _frac(W["stem.b"]))
    q = [[[_code(_act(v, cap) / a[0], fmt) for v in row] for row in bd] for bd in y]
    rec = [q]
    g = F // 4 if pool_every else 0
    Fr_ = F - g
    for j in range(nb):
        q_in = q
        pool = pool_every and j % pool_every == pool_every - 1
        for second in (0, 1):
            n = 2 * j + second
            key = f"w{1 + second}.{j}"
            Wn = W[key]
            s_w = [Fr(float(v)) for v in sw[n]]
            wq = [[[[_code(Fr(float(Wn[f, c, dy, dx])) / s_w[f], fmt) for dx in range(3)] for dy in range(3)]
                   for c in range(Wn.shape[1])] for f in range(F)]
            acc = _conv(q, wq)
            bvec = [Fr(float(v)) for v in W[f"b{1 + second}.{j}"]]
            yv = [[[acc[b][f][s] * a[n] * s_w[f] + bvec[f] for s in range(64)] for f in range(F)]
                  for b in range(len(acc))]
            if second:
                yv = [[[yv[b][f][s] + q_in[b][f][s] * a[n - 1] for s in range(64)] for f in range(F)]
                      for b in range(len(yv))]
            if pool and not second:
                Wg = W[f"pool.{j}"]
                out = []
                for b in range(len(yv)):
                    p = [[_act(v, cap) for v in yv[b][f]] for f in range(Fr_, F)]
                    feats = [sum(r) / 64 for r in p] + [max(r) for r in p]
                    c = [sum(Fr(float(Wg[o, i])) * feats[i] for i in range(2 * g)) for o in range(Fr_)]
                    out.append([[_code(_act(yv[b][f][s] + c[f], cap) / a[n + 1], fmt) for s in range(64)]
                                for f in range(Fr_)])
                q = out
            else:
                q = [[[_code(_act(v, cap) / a[n + 1], fmt) for v in row] for row in bd] for bd in yv]
            rec.append(q)
    return rec


def _as_array(q):
    return np.array([[[float(v) for v in row] for row in bd] for bd in q])


def _tiny_spec(cap):
    return azgen.NetShape(in_planes=3, blocks=2, filters=4, policy_planes=2, value_hidden=8, act_cap=cap)


def _tiny_inputs(spec, n, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    planes = (rng.random((n, spec.in_planes, 8, 8)) < 0.35).astype(np.float32)
    planes[:, -1] = 1.0                                     # a constant plane, as in the workloads
    legal = np.zeros((n, spec.n_moves), dtype=np.uint8)
    for i in range(n):
        legal[i, rng.choice(spec.n_moves, size=10, replace=False)] = 1
    return planes, legal


def _heads_torch(spec, W, h, legal):
    """Move-plane policy and tanh value heads with torch float64 library routines."""
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))  # noqa: E731
    H = t(h)
    B = H.shape[0]
    z = TF.conv2d(H, t(W["policy.w"])[:, :, None, None], t(W["policy.b"])).reshape(B, -1)
    m = torch.from_numpy(legal != 0)
    z = torch.where(m, z, torch.tensor(-torch.inf, dtype=torch.float64))
    P = torch.where(m, torch.softmax(z, dim=1), torch.zeros_like(z))
    u = TF.conv2d(H, t(W["value.w"])[:, :, None, None], t(W["value.b"])).reshape(B, 64)
    if spec.value_conv_relu:
        u = torch.relu(u)
    g = torch.relu(TF.linear(u, t(W["fc1.w"]), t(W["fc1.b"])))
    V = torch.tanh(TF.linear(g, t(W["fc2.w"]), t(W["fc2.b"])))[:, 0]
    return P.numpy(), V.numpy()


@pytest.mark.parametrize("fmt,cap,act_mul", [("int8", 0.0, 1.0), ("int8", 6.0, 0.5), ("fp8", 0.0, 1.0),
                                              ("fp8", 6.0, 0.25)])
def test_quantised_network_codes_match_exact_rational_loops(fmt, cap, act_mul):
    # act_mul < 1 shrinks the activation scales below absmax calibration so that
    # codes saturate (int8 at 127, e4m3 at 448) as well as round
    spec = _tiny_spec(cap)
    blob = azgen.make_weights(spec, 91, alpha_fold=True, bf16=True)
    W = O.unpack(spec, blob)
    planes, legal = _tiny_inputs(spec, 2, 92)
    calib, _ = _tiny_inputs(spec, 16, 93)
    ws = O.weight_scales(spec, blob, fmt)
    acs = (O.act_scales_from_absmax(O.calibrate_absmax(spec, blob, calib), fmt) * np.float32(act_mul)).astype(np.float32)
    rec = []
    P, V = O.forward_quant(spec, blob, ws, acs, fmt, planes, legal, record=rec)
    TIES.clear()
    exact = _rational_tower(spec, W, planes, ws, acs, fmt)
    assert len(rec) == len(exact) == 2 * spec.blocks + 1
    for k, (qo, qe) in enumerate(zip(rec, exact)):
        qe = _as_array(qe)
        assert qo.shape == qe.reshape(qo.shape).shape
        diff = qo.reshape(qe.shape) != qe
        if TIES:
            assert diff.sum() <= len(TIES), (k, int(diff.sum()), len(TIES))
        else:
            assert not diff.any(), (k, int(diff.sum()))
    assert max(float(np.abs(q).max()) for q in rec) == O.qmax(fmt) or act_mul == 1.0
    # the heads on the exact codes' dequantised tower output, by torch
    h = _as_array(exact[-1]).reshape(rec[-1].shape) * float(acs[-1])
    Pt, Vt = _heads_torch(spec, W, h, legal)
    np.testing.assert_allclose(P, Pt, rtol=0, atol=1e-12)
    np.testing.assert_allclose(V, Vt, rtol=0, atol=1e-12)


def test_quantised_saturates_and_caps_where_the_definition_says():
    # act_mul 0.5 with the ReLU6 cap: some t / h codes sit at the cap's code and
    # some at 127; and no code of a post-activation tensor is negative
    spec = _tiny_spec(6.0)
    blob = azgen.make_weights(spec, 91, alpha_fold=True, bf16=True)
    planes, legal = _tiny_inputs(spec, 2, 92)
    ws = O.weight_scales(spec, blob, "int8")
    acs = np.full(spec.n_act_scales(), np.float32(6.0 / 127.0 * 0.5), np.float32)
    rec = []
    O.forward_quant(spec, blob, ws, acs, "int8", planes, legal, record=rec)
    top = [float(q.max()) for q in rec]
    assert max(top) == 127.0 and min(float(q.min()) for q in rec) == 0.0


def test_deployed_int8_codes_match_exact_rational_loops():
    # a pooling block (block 1 of 2): pooled channels activated from the exact
    # dequantised sums, mean and maximum over the board, projected, added to the
    # regular channels before their activation and rounding
    spec = azgen.NetShape(in_planes=4, blocks=2, filters=8, policy_planes=0, value_hidden=6, value_conv_relu=1,
                          act_cap=6.0, pool_every=2, policy_head="fromto", token_dim=8, value_head="wdl",
                          value_channels=2)
    blob = azgen.make_weights(spec, 95, alpha_fold=True, bf16=True)
    W = OD.unpack(spec, blob)
    rng = np.random.Generator(np.random.PCG64(96))
    planes = (rng.random((2, 4, 8, 8)) < 0.35).astype(np.float32)
    planes[:, 3] = 2.0                                      # an integer count plane
    legal = np.zeros((2, spec.n_moves), dtype=np.uint8)
    legal[:, rng.choice(spec.n_moves, size=30, replace=False)] = 1
    ws = OD.weight_scales(spec, blob)
    acs = np.full(2 * spec.blocks + 1, np.float32(6.0 / 127.0), np.float32)
    rec = []
    OD.forward_quant(spec, blob, ws, acs, planes, legal, record=rec)
    TIES.clear()
    exact = _rational_tower(spec, W, planes, ws, acs, "int8", pool_every=2)
    assert [r.shape[1] for r in rec] == [8, 8, 8, 6, 8]
    for k, (qo, qe) in enumerate(zip(rec, exact)):
        qe = _as_array(qe).reshape(qo.shape)
        diff = qo != qe
        assert diff.sum() <= len(TIES), (k, int(diff.sum()), len(TIES))
