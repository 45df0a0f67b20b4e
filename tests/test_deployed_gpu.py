"""GPU parity of the deployed network (global-pooling blocks, from-to policy
head over 1,880 actions, WDL value head) against the CPU oracle, through the C
ABI on seeded inputs.

int8 (the paper's deployment: int8 trunk with the fixed ReLU6 activation scale
6/127, per-output-channel weight scales, pooling and heads in floating point)
is compared with the oracle's int8 network, the plain float64 definition
(exact integer sums, float64 pooling, rescale and rounding); bf16 with the
float64 network.  The kernels compute the same definition except for the bf16
stem's fp32 sums: on the CPU that flips 1 of the 10.5 M stem codes of the
seeded 1,024-position batch, which moves that position by max|dP| 0.0044 and
|dV| 0.0098, under a third of the tolerance.
Tolerances: int8 max |dP| 3e-2 and |dV| 5e-2, bf16 1e-2 and 2e-2 (the WDL
probabilities are held to the value tolerance).  Both kernel tilings (one wave
per board, four waves per board) are run and must agree bitwise."""

import numpy as np
import pytest

import azgen
from oracle import deployed as OD

from ._harness import TOL, assert_policy_structure

pytestmark = pytest.mark.gpu

DEP = azgen.DEPLOYED_14X160
RELU6_SCALE = 6.0 / 127.0


def _shape(blocks, **kw):
    return azgen.NetShape(**{**DEP.__dict__, "blocks": blocks, **kw})


def _inputs(shape, n, seed, pieces=(16, 32)):
    rng = np.random.Generator(np.random.PCG64(seed))
    planes = azgen.make_planes_52(n, pieces, rng) if shape.in_planes == 52 else \
        azgen.make_planes(n, shape.in_planes, pieces, rng)
    legal = azgen.make_legal(n, shape.n_moves, (20, 40), rng)
    return planes, legal


def _edge_rows(legal):
    """Row 0: no legal action; row 1: one; row 2: every promotion and a few
    pairs; row 3: every action."""
    legal = legal.copy()
    legal[0] = 0
    legal[1] = 0
    legal[1, 1234] = 1
    legal[2] = 0
    legal[2, 1792:] = 1
    legal[2, [0, 17, 999]] = 1
    legal[3] = 1
    return legal


def _scales(shape, blob):
    return OD.weight_scales(shape, blob), np.full(2 * shape.blocks + 1, RELU6_SCALE, np.float32)


def gpu_eval(shape, blob, dtype, planes, legal, ws=None, acs=None, tiling=0):
    import torch

    import paper_2609_37447_amd as az
    B = planes.shape[0]
    net = az.az_net_load(az.spec_from_shape(shape, B), blob, dtype, ws, acs)
    try:
        assert az.az_net_moves(net) == 1880
        az.az_net_set_tiling(net, tiling)
        print(f"case {dtype} blocks={shape.blocks} B={B} tiling={tiling or az.az_net_tiling_for(net, B)}", flush=True)
        dev = torch.device("cuda:0")
        pl = torch.from_numpy(np.ascontiguousarray(planes, dtype=np.float32)).to(dev)
        lg = torch.from_numpy(np.ascontiguousarray(legal, dtype=np.uint8)).to(dev)
        pol = torch.full((B, 1880), float("nan"), device=dev)
        val = torch.full((B,), float("nan"), device=dev)
        wdl = torch.full((B, 3), float("nan"), device=dev)
        az.eval_tensors(net, pl, lg, pol, val, wdl=wdl)
        val2 = torch.full((B,), float("nan"), device=dev)
        pol2 = torch.full((B, 1880), float("nan"), device=dev)
        az.eval_tensors(net, pl, lg, pol2, val2)          # without the WDL output
        torch.cuda.synchronize()
        assert torch.equal(pol, pol2) and torch.equal(val, val2)
    finally:
        az.az_net_free(net)
    f = lambda t: t.cpu().numpy().astype(np.float64)  # noqa: E731
    return f(pol), f(val), f(wdl)


def _check(got, ref, legal, dtype):
    (Pg, Vg, Wg), (Pr, Vr, Wr) = got, ref
    assert_policy_structure(Pg, legal)
    assert np.all(np.abs(Wg.sum(axis=1) - 1.0) <= 1e-5)
    assert np.allclose(Vg, Wg[:, 0] - Wg[:, 2], atol=1e-6)
    tp, tv = TOL[dtype]
    dp, dv, dw = np.abs(Pg - Pr).max(), np.abs(Vg - Vr).max(), np.abs(Wg - Wr).max()
    print(f"{dtype}: max|dP| {dp:.3g}  max|dV| {dv:.3g}  max|dWDL| {dw:.3g}")
    assert dp <= tp and dv <= tv and dw <= tv, (dp, dv, dw)
    return dp, dv


@pytest.mark.parametrize("tiling", [1, 2])
@pytest.mark.parametrize("blocks,B", [(2, 13), (4, 37)])
def test_deployed_int8_matches_quantised_oracle(blocks, B, tiling):
    shape = _shape(blocks)
    blob = azgen.make_weights(shape, 1006, alpha_fold=True, bf16=True)
    planes, legal = _inputs(shape, B, 2006 + blocks)
    legal = _edge_rows(legal)
    ws, acs = _scales(shape, blob)
    got = gpu_eval(shape, blob, "int8", planes, legal, ws, acs, tiling=tiling)
    ref = OD.forward_quant(shape, blob, ws, acs, planes, legal)
    _check(got, ref, legal, "int8")


def test_deployed_int8_literal_heads():
    # literal draw (no residual or head conditioning): a one-hot policy and a
    # saturated value, still equal to the quantised oracle's
    shape = _shape(2)
    blob = azgen.make_weights(shape, 1026, alpha_fold=False, bf16=True)
    planes, legal = _inputs(shape, 10, 2126)
    ws, acs = _scales(shape, blob)
    got = gpu_eval(shape, blob, "int8", planes, legal, ws, acs)
    ref = OD.forward_quant(shape, blob, ws, acs, planes, legal)
    _check(got, ref, legal, "int8")


@pytest.mark.parametrize("tiling", [1, 2])
@pytest.mark.parametrize("blocks,B", [(2, 11), (3, 20)])
def test_deployed_bf16_matches_float_oracle(blocks, B, tiling):
    shape = _shape(blocks)
    blob = azgen.make_weights(shape, 1006, alpha_fold=True, bf16=True)
    planes, legal = _inputs(shape, B, 2106 + blocks)
    legal = _edge_rows(legal)
    got = gpu_eval(shape, blob, "bf16", planes, legal, tiling=tiling)
    ref = OD.forward(shape, blob, planes, legal)
    _check(got, ref, legal, "bf16")


@pytest.mark.parametrize("tiling", [1, 2])
def test_deployed_no_pooling_and_other_shapes(tiling):
    # pooling switched off, 20 input planes, 5 value channels, 100 hidden units,
    # no ReLU after the value convolution, uncapped activation
    shape = _shape(2, in_planes=20, pool_every=0, value_channels=5, value_hidden=100, value_conv_relu=0,
                   act_cap=0.0)
    blob = azgen.make_weights(shape, 1016, alpha_fold=True, bf16=True)
    planes, legal = _inputs(shape, 9, 2116)
    got = gpu_eval(shape, blob, "bf16", planes, legal, tiling=tiling)
    ref = OD.forward(shape, blob, planes, legal)
    _check(got, ref, legal, "bf16")


@pytest.mark.parametrize("tiling", [1, 2])
@pytest.mark.parametrize("pool_every,dtype", [(1, "int8"), (3, "bf16")])
def test_deployed_pooling_period(pool_every, dtype, tiling):
    # global pooling in every block, or in every third (blocks 2 and 5 of six)
    shape = _shape(3 if pool_every == 1 else 6, pool_every=pool_every)
    blob = azgen.make_weights(shape, 1066, alpha_fold=True, bf16=True)
    planes, legal = _inputs(shape, 7, 2266 + pool_every)
    if dtype == "int8":
        ws, acs = _scales(shape, blob)
        got = gpu_eval(shape, blob, "int8", planes, legal, ws, acs, tiling=tiling)
        ref = OD.forward_quant(shape, blob, ws, acs, planes, legal)
    else:
        got = gpu_eval(shape, blob, "bf16", planes, legal, tiling=tiling)
        ref = OD.forward(shape, blob, planes, legal)
    _check(got, ref, legal, dtype)


def _oracle_rows(shape, blob, dtype, planes, legal, ws, acs, chunk=128):
    outs = []
    for s in range(0, planes.shape[0], chunk):
        pl, lg = planes[s:s + chunk], legal[s:s + chunk]
        outs.append(OD.forward_quant(shape, blob, ws, acs, pl, lg) if dtype == "int8"
                    else OD.forward(shape, blob, pl, lg))
        print(f"  oracle rows {s}..{s + pl.shape[0] - 1}", flush=True)
    return tuple(np.concatenate([o[i] for o in outs]) for i in range(3))


def test_deployed_14x160_int8_batch1024_every_row():
    w = azgen.WORKLOADS["deployed14x160_int8_b1024"]
    blob = azgen.workload_weights(w)
    planes, legal = azgen.make_inputs(w)
    ws, acs = _scales(w.shape, blob)
    Pg, Vg, Wg = gpu_eval(w.shape, blob, "int8", planes, legal, ws, acs)
    assert_policy_structure(Pg, legal)
    ref = _oracle_rows(w.shape, blob, "int8", planes, legal, ws, acs)
    _check((Pg, Vg, Wg), ref, legal, "int8")


def test_deployed_14x160_bf16_every_row():
    w = azgen.WORKLOADS["deployed14x160_bf16_b1024"]
    blob = azgen.workload_weights(w)
    planes, legal = azgen.make_inputs(w, n=256)
    Pg, Vg, Wg = gpu_eval(w.shape, blob, "bf16", planes, legal)
    assert_policy_structure(Pg, legal)
    ref = _oracle_rows(w.shape, blob, "bf16", planes, legal, None, None)
    _check((Pg, Vg, Wg), ref, legal, "bf16")


@pytest.mark.parametrize("dtype,B", [("int8", 64), ("int8", 256), ("bf16", 64)])
def test_deployed_14x160_small_batch_every_row(dtype, B):
    # the interactive regime: the default tiling below 257 boards is four waves per board
    w = azgen.WORKLOADS[f"deployed14x160_{dtype}_b1024"]
    blob = azgen.workload_weights(w)
    planes, legal = azgen.make_inputs(w, n=B)
    ws, acs = _scales(w.shape, blob) if dtype == "int8" else (None, None)
    Pg, Vg, Wg = gpu_eval(w.shape, blob, dtype, planes, legal, ws, acs)
    assert_policy_structure(Pg, legal)
    ref = _oracle_rows(w.shape, blob, dtype, planes, legal, ws, acs)
    _check((Pg, Vg, Wg), ref, legal, dtype)


@pytest.mark.parametrize("dtype", ["int8", "bf16"])
def test_deployed_tilings_agree_bitwise(dtype):
    # every tile's K sums run in the same order in both tilings, and the pooling
    # projection and the heads are the same code: identical outputs
    shape = _shape(4)
    blob = azgen.make_weights(shape, 1056, alpha_fold=True, bf16=True)
    planes, legal = _inputs(shape, 21, 2256)
    legal = _edge_rows(legal)
    ws, acs = _scales(shape, blob) if dtype == "int8" else (None, None)
    one = gpu_eval(shape, blob, dtype, planes, legal, ws, acs, tiling=1)
    four = gpu_eval(shape, blob, dtype, planes, legal, ws, acs, tiling=2)
    for a, b in zip(one, four):
        assert np.array_equal(a, b)


def test_deployed_rows_do_not_depend_on_the_batch():
    shape = _shape(2)
    blob = azgen.make_weights(shape, 1006, alpha_fold=True, bf16=True)
    planes, legal = _inputs(shape, 8, 2206)
    ws, acs = _scales(shape, blob)
    full = gpu_eval(shape, blob, "int8", planes, legal, ws, acs)
    one = gpu_eval(shape, blob, "int8", planes[5:6], legal[5:6], ws, acs)
    for a, b in zip(full, one):
        assert np.array_equal(a[5:6], b)


def test_deployed_tiling_choice():
    # the tiling with fewer rounds x time per round on 256 compute units: four
    # waves per board (256 boards a round) against one wave per board (1,024 int8
    # or 768 bf16 boards a round, 2.5x / 2.8x as long)
    import paper_2609_37447_amd as az
    shape = _shape(2)
    blob = azgen.make_weights(shape, 1036, alpha_fold=True, bf16=True)
    ws, acs = _scales(shape, blob)
    want = {"int8": {1: 2, 64: 2, 256: 2, 512: 2, 513: 1, 768: 1, 1024: 1},
            "bf16": {1: 2, 64: 2, 512: 2, 513: 1, 768: 1, 769: 2, 1024: 2}}
    for dtype, cases in want.items():
        net = az.az_net_load(az.spec_from_shape(shape, 1024), blob, dtype,
                             *((ws, acs) if dtype == "int8" else (None, None)))
        try:
            assert {B: az.az_net_tiling_for(net, B) for B in cases} == cases
            for t in (0, 1, 2):
                assert az.az_net_set_tiling(net, t) == az.AZ_OK
            assert az.az_net_tiling_for(net, 64) == 2
            for t in (3, -1):
                assert az.az_net_set_tiling(net, t, raise_on_error=False) == az.AZ_ERR_INVALID_ARG
        finally:
            az.az_net_free(net)


def test_deployed_validate_gate():
    # deployment validation (top-1 legal agreement, legal-policy KL, value error)
    # of the int8 deployed network against its bf16 source over the 1,880 actions:
    # the faithful network passes, one with activation scales x 0.1 does not
    import torch

    import paper_2609_37447_amd as az
    from oracle import az_oracle as O
    shape = _shape(4)
    blob = azgen.make_weights(shape, 1046, alpha_fold=True, bf16=True)
    planes, legal = _inputs(shape, 64, 2246)
    legal = _edge_rows(legal)
    ws, acs = _scales(shape, blob)
    dev = torch.device("cuda:0")
    pl = torch.from_numpy(planes).to(dev)
    lg = torch.from_numpy(legal).to(dev)
    spec = az.spec_from_shape(shape, 64)
    ref = az.az_net_load(spec, blob, "bf16")
    good = az.az_net_load(spec, blob, "int8", ws, acs)
    broken = az.az_net_load(spec, blob, "int8", ws, acs * np.float32(0.1))
    try:
        r_good = az.validate(good, ref, pl, lg)
        r_bad = az.validate(broken, ref, pl, lg)
        print(f"faithful: top1 {r_good['top1']:.3f} KL {r_good['kl']:.4f} |dV| {r_good['dv_max']:.3f}; "
              f"broken: top1 {r_bad['top1']:.3f} KL {r_bad['kl']:.4f} |dV| {r_bad['dv_max']:.3f}")
        assert r_good["passed"] and not r_bad["passed"]
        # per-row metrics against the definition on the same evaluations
        P = {}
        for key, net in (("ref", ref), ("test", good)):
            pol = torch.empty((64, 1880), device=dev)
            val = torch.empty((64,), device=dev)
            az.eval_tensors(net, pl, lg, pol, val)
            P[key] = (pol.cpu().numpy(), val.cpu().numpy())
        torch.cuda.synchronize()
        top1, kl, dv = O.compare_outputs(P["ref"][0], P["ref"][1], P["test"][0], P["test"][1], legal)
        g = r_good["rows"]
        assert np.array_equal(g[:, 0], top1)
        assert np.all(np.abs(g[:, 1] - kl) <= 1e-5 + 1e-4 * np.abs(kl))
        assert np.all(np.abs(g[:, 2] - dv) <= 1e-7)
    finally:
        for n in (ref, good, broken):
            az.az_net_free(n)
