"""Host submission pipeline: what comes back in a slot's host buffers equals
az_eval_batch on the same inputs, bit for bit, with and without graph replay,
over several slots in flight at once and changing batch sizes (needs gfx950)."""

import ctypes

import numpy as np
import pytest

import azgen
from tests import _harness as H

pytestmark = pytest.mark.gpu

W = azgen.WORKLOADS


def _print(*a):
    print(*a, flush=True)


def _scales(w, dtype):
    if dtype == "f32":
        return None, None
    if w.shape.policy_head == "fromto":   # deployed network: fixed ReLU6 activation scale
        from oracle import deployed as OD
        blob = azgen.workload_weights(w)
        return OD.weight_scales(w.shape, blob), np.full(2 * w.shape.blocks + 1, 6.0 / 127.0, np.float32)
    return H.quant_scales(w.name, dtype)


@pytest.mark.parametrize("use_graphs", [False, True])
@pytest.mark.parametrize("wname,dtype", [("net20x128_int8_b1024", "int8"), ("tiny_2x32_f32_b16", "f32"),
                                         ("deployed14x160_int8_b1024", "int8")])
def test_pipeline_matches_eval_batch(wname, dtype, use_graphs):
    import torch

    import paper_2609_37447_amd as az
    w = W[wname]
    blob = azgen.workload_weights(w)
    ws, acs = _scales(w, dtype)
    MB, SLOTS = 48, 3
    _print(f"case pipeline {wname} graphs={use_graphs} max_batch={MB} slots={SLOTS}")
    spec = az.spec_from_shape(w.shape, MB)
    net = az.az_net_load(spec, blob, dtype, ws, acs)
    pipe = None
    try:
        pipe = az.Pipeline(net, spec, MB, SLOTS, use_graphs)
        assert pipe.views[0][4] is None
        dev = torch.device("cuda:0")
        # batch sizes per round and slot: full, ragged, one, empty, a repeat of
        # an earlier size (graph reuse) and a change back (recapture)
        rounds = [(48, 17, 1), (17, 48, 0), (48, 17, 5), (1, 1, 48)]
        for r, sizes in enumerate(rounds):
            want = []
            for k, B in enumerate(sizes):
                planes, legal = azgen.make_inputs(w, n=max(B, 1), seed=100 + 10 * r + k)
                pl, lg, po, va, _ = pipe.views[k]
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
                _, _, po, va, _ = pipe.views[k]
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


def _compact_definition(P, legal, K):
    """Per row: probabilities of the legal cells in ascending cell order, first K, zero-padded."""
    out = np.zeros((P.shape[0], K), np.float32)
    cnt = np.zeros(P.shape[0], np.int32)
    for r in range(P.shape[0]):
        v = P[r][legal[r] != 0]
        cnt[r] = v.size
        out[r, :min(K, v.size)] = v[:K]
    return out, cnt


@pytest.mark.parametrize("use_graphs", [False, True])
@pytest.mark.parametrize("wname", ["net20x128_int8_b1024", "deployed14x160_int8_b1024"])
def test_pipeline_compact_policy(use_graphs, wname):
    import torch

    import paper_2609_37447_amd as az
    w = W[wname]
    blob = azgen.workload_weights(w)
    ws, acs = _scales(w, "int8")
    MB, K = 300, 48
    _print(f"case pipeline compact {wname} graphs={use_graphs} max_batch={MB} max_legal={K}")
    spec = az.spec_from_shape(w.shape, MB)
    net = az.az_net_load(spec, blob, "int8", ws, acs)
    pipe = None
    try:
        pipe = az.Pipeline(net, spec, MB, 2, use_graphs, max_legal=K)
        dev = torch.device("cuda:0")
        for r, B in enumerate((MB, 257, 1)):
            planes, legal = azgen.make_inputs(w, n=B, seed=300 + r)
            if B > 4:
                legal[0] = 0                          # terminal row: nothing legal
                legal[1] = 0
                legal[1, -K:] = 1                     # exactly max_legal, at the end of the row
                legal[2] = 0
                legal[2, 5] = 1                       # single legal move
                legal[3] = 0
                legal[3, ::97] = 1                    # spread over the row, cut to exactly max_legal
                legal[3, 97 * K:] = 0
            k = r % 2
            pl, lg, po, va, cnt = pipe.views[k]
            pl[:B] = planes
            lg[:B] = legal
            po[:] = np.nan
            cnt[:] = -1
            P0 = torch.empty((B, w.shape.n_moves), device=dev)
            V0 = torch.empty((B,), device=dev)
            az.eval_tensors(net, torch.from_numpy(planes).to(dev), torch.from_numpy(legal).to(dev), P0, V0)
            Pd, Vd = P0.cpu().numpy(), V0.cpu().numpy()
            pipe.submit(k, B)
            pipe.wait(k)
            want, wcnt = _compact_definition(Pd, legal, K)
            assert np.array_equal(cnt[:B], wcnt), f"B={B} counts"
            assert np.array_equal(po[:B], want), f"B={B} compact policy"
            assert np.array_equal(va[:B], Vd), f"B={B} value"
            assert np.all(np.isnan(po[B:])) and np.all(cnt[B:] == -1)
            _print(f"  B={B} ok (legal counts {wcnt.min()}..{wcnt.max()})")
        # a row with more legal cells than max_legal: the wait reports it, the row
        # holds its first K legal probabilities and the true count
        planes, legal = azgen.make_inputs(w, n=8, seed=399)
        legal[5, :K + 9] = 1
        pl, lg, po, va, cnt = pipe.views[0]
        pl[:8] = planes
        lg[:8] = legal
        pipe.submit(0, 8)
        with pytest.raises(az.AzError, match="more than max_legal"):
            pipe.wait(0)
        P0 = torch.empty((8, w.shape.n_moves), device=dev)
        V0 = torch.empty((8,), device=dev)
        az.eval_tensors(net, torch.from_numpy(planes).to(dev), torch.from_numpy(legal).to(dev), P0, V0)
        want, wcnt = _compact_definition(P0.cpu().numpy(), legal, K)
        assert cnt[5] == K + 9 + np.count_nonzero(legal[5, K + 9:])
        assert np.array_equal(cnt[:8], wcnt) and np.array_equal(po[:8], want)
        pipe.submit(0, 8)                             # the slot is usable again
        with pytest.raises(az.AzError):
            pipe.wait(0)
    finally:
        if pipe is not None:
            pipe.close()
        az.az_net_free(net)


def test_pipeline_worker_threads_share_one_pipeline():
    # four threads, two slots each, submitting concurrently into one pipeline
    import threading

    import torch

    import paper_2609_37447_amd as az
    w = W["net20x128_int8_b1024"]
    blob = azgen.workload_weights(w)
    ws, acs = H.quant_scales(w.name, "int8")
    MB, K, WORKERS, ROUNDS = 96, 64, 4, 3
    _print(f"case pipeline threads int8 workers={WORKERS} max_batch={MB} max_legal={K}")
    spec = az.spec_from_shape(w.shape, MB)
    net = az.az_net_load(spec, blob, "int8", ws, acs)
    pipe = None
    try:
        pipe = az.Pipeline(net, spec, MB, 2 * WORKERS, False, max_legal=K)
        dev = torch.device("cuda:0")
        # per slot and round: inputs and the expected compact outputs
        jobs = {}
        for k in range(2 * WORKERS):
            for r in range(ROUNDS):
                B = MB - 7 * k - r
                planes, legal = azgen.make_inputs(w, n=B, seed=500 + 10 * k + r)
                P0 = torch.empty((B, w.shape.n_moves), device=dev)
                V0 = torch.empty((B,), device=dev)
                az.eval_tensors(net, torch.from_numpy(planes).to(dev), torch.from_numpy(legal).to(dev), P0, V0)
                want, wcnt = _compact_definition(P0.cpu().numpy(), legal, K)
                jobs[k, r] = (planes, legal, want, wcnt, V0.cpu().numpy())
        torch.cuda.synchronize()
        errors = []

        def run(mine):
            try:
                for r in range(ROUNDS):
                    for k in mine:
                        planes, legal = jobs[k, r][:2]
                        B = planes.shape[0]
                        pipe.views[k][0][:B] = planes
                        pipe.views[k][1][:B] = legal
                        pipe.submit(k, B)
                    for k in mine:
                        pipe.wait(k)
                        _, _, want, wcnt, V = jobs[k, r]
                        B = want.shape[0]
                        _, _, po, va, cnt = pipe.views[k]
                        assert np.array_equal(cnt[:B], wcnt), f"slot {k} round {r} counts"
                        assert np.array_equal(po[:B], want), f"slot {k} round {r} policy"
                        assert np.array_equal(va[:B], V), f"slot {k} round {r} value"
            except Exception as e:  # re-raised in the main thread
                errors.append(e)

        th = [threading.Thread(target=run, args=([2 * j, 2 * j + 1],)) for j in range(WORKERS)]
        for t in th:
            t.start()
        for t in th:
            t.join()
        if errors:
            raise errors[0]
    finally:
        if pipe is not None:
            pipe.close()
        az.az_net_free(net)


@pytest.mark.parametrize("use_graphs", [False, True])
def test_native_driver_outputs_and_statuses(use_graphs):
    # az_pipeline_drive resubmits each slot's resident inputs from native worker
    # threads; afterwards every slot holds the compact outputs of its own inputs
    import torch

    import paper_2609_37447_amd as az
    w = W["net20x128_int8_b1024"]
    blob = azgen.workload_weights(w)
    ws, acs = H.quant_scales(w.name, "int8")
    MB, K, WORKERS, PER = 64, 64, 3, 2
    _print(f"case native driver int8 graphs={use_graphs} workers={WORKERS}x{PER} max_batch={MB}")
    spec = az.spec_from_shape(w.shape, MB)
    net = az.az_net_load(spec, blob, "int8", ws, acs)
    pipe = None
    try:
        pipe = az.Pipeline(net, spec, MB, WORKERS * PER, use_graphs, max_legal=K)
        dev = torch.device("cuda:0")
        want = []
        for k in range(WORKERS * PER):
            planes, legal = azgen.make_inputs(w, n=MB, seed=900 + k)
            pipe.views[k][0][:] = planes
            pipe.views[k][1][:] = legal
            P0 = torch.empty((MB, w.shape.n_moves), device=dev)
            V0 = torch.empty((MB,), device=dev)
            az.eval_tensors(net, torch.from_numpy(planes).to(dev), torch.from_numpy(legal).to(dev), P0, V0)
            want.append(_compact_definition(P0.cpu().numpy(), legal, K) + (V0.cpu().numpy(),))
        torch.cuda.synchronize()
        sec = pipe.drive(WORKERS, PER, MB, 4, 8)
        assert sec > 0.0
        for k in range(WORKERS * PER):
            _, _, po, va, cnt = pipe.views[k]
            wp, wc, wv = want[k]
            assert np.array_equal(cnt, wc), f"slot {k} counts"
            assert np.array_equal(po, wp), f"slot {k} policy"
            assert np.array_equal(va, wv), f"slot {k} value"
        # bad arguments: nothing is submitted
        L, sec_c = az.lib(), ctypes.c_double()
        bad = [(0, PER, MB, 0, 1), (WORKERS, PER + 1, MB, 0, 1), (WORKERS, PER, MB + 1, 0, 1),
               (WORKERS, PER, 0, 0, 1), (WORKERS, PER, MB, -1, 1), (WORKERS, PER, MB, 0, 0)]
        for a in bad:
            assert L.az_pipeline_drive(pipe.p, *a, ctypes.byref(sec_c)) == az.AZ_ERR_INVALID_ARG, a
        assert L.az_pipeline_drive(pipe.p, WORKERS, PER, MB, 0, 1, None) == az.AZ_ERR_INVALID_ARG
        # a row with more than max_legal legal cells surfaces from a worker thread
        # with its message on the calling thread
        pipe.views[1][1][5, :] = 1
        st = L.az_pipeline_drive(pipe.p, WORKERS, PER, MB, 0, 2, ctypes.byref(sec_c))
        assert st == az.AZ_ERR_INVALID_ARG, st
        assert b"max_legal" in L.az_last_error(), L.az_last_error()
    finally:
        if pipe is not None:
            pipe.close()
        az.az_net_free(net)
