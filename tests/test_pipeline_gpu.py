"""Host submission pipeline: what comes back in a slot's host buffers equals
az_eval_batch on the same inputs, bit for bit, with and without graph replay,
over several slots in flight at once and changing batch sizes (needs gfx950)."""

import numpy as np
import pytest

import azgen
from tests import _harness as H

pytestmark = pytest.mark.gpu

W = azgen.WORKLOADS


def _print(*a):
    print(*a, flush=True)


@pytest.mark.parametrize("use_graphs", [False, True])
@pytest.mark.parametrize("wname,dtype", [("net20x128_int8_b1024", "int8"), ("tiny_2x32_f32_b16", "f32")])
def test_pipeline_matches_eval_batch(wname, dtype, use_graphs):
    import torch

    import paper_2609_37447_amd as az
    w = W[wname]
    blob = azgen.workload_weights(w)
    ws, acs = H.quant_scales(w.name, dtype) if dtype != "f32" else (None, None)
    MB, SLOTS = 48, 3
    _print(f"case pipeline {wname} graphs={use_graphs} max_batch={MB} slots={SLOTS}")
    spec = az.spec_from_shape(w.shape, MB)
    net = az.az_net_load(spec, blob, dtype, ws, acs)
    pipe = None
    try:
        pipe = az.Pipeline(net, spec, MB, SLOTS, use_graphs)
        dev = torch.device("cuda:0")
        # batch sizes per round and slot: full, ragged, one, empty, a repeat of
        # an earlier size (graph reuse) and a change back (recapture)
        rounds = [(48, 17, 1), (17, 48, 0), (48, 17, 5), (1, 1, 48)]
        for r, sizes in enumerate(rounds):
            want = []
            for k, B in enumerate(sizes):
                planes, legal = azgen.make_inputs(w, n=max(B, 1), seed=100 + 10 * r + k)
                pl, lg, po, va = pipe.views[k]
                pl[:B] = planes[:B]
                lg[:B] = legal[:B]
                po[:] = np.nan
                va[:] = np.nan
                P0 = torch.full((max(B, 1), w.shape.n_moves), float("nan"), device=dev)
                V0 = torch.full((max(B, 1),), float("nan"), device=dev)
                if B:
                    az.eval_tensors(net, torch.from_numpy(planes[:B]).to(dev),
                                    torch.from_numpy(legal[:B]).to(dev), P0[:B], V0[:B])
                want.append((P0[:B].cpu().numpy(), V0[:B].cpu().numpy()))
            torch.cuda.synchronize()
            for k, B in enumerate(sizes):
                pipe.submit(k, B)
            for k in reversed(range(SLOTS)):
                pipe.wait(k)
                assert pipe.query(k)
            for k, B in enumerate(sizes):
                _, _, po, va = pipe.views[k]
                assert np.array_equal(po[:B], want[k][0]), f"round {r} slot {k} B={B} policy"
                assert np.array_equal(va[:B], want[k][1]), f"round {r} slot {k} B={B} value"
                assert np.all(np.isnan(po[B:])) and np.all(np.isnan(va[B:])), "rows past B written"
            _print(f"  round {r} sizes {sizes} ok")
        # a slot in flight refuses a second submission until it is waited for
        pipe.submit(0, 48)
        with pytest.raises(az.AzError):
            pipe.submit(0, 48)
        pipe.wait(0)
        with pytest.raises(az.AzError):
            pipe.submit(0, 49)
    finally:
        if pipe is not None:
            pipe.close()
        az.az_net_free(net)
