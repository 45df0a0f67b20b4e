"""az_eval_batch_compact_noalloc, the entry point that allocates nothing: its
compact outputs equal the pipeline's compact outputs (az_pipeline_submit, whose
dense policy buffer the library allocates) element for element, on two calls in
a row, the second with a smaller batch; no allocation is made; sizes past the
static array and bad arguments are rejected before the device is touched."""

import ctypes

import numpy as np
import pytest

import azgen
from tests import _harness as H

pytestmark = pytest.mark.gpu


def _print(*a):
    print(*a, flush=True)


def _int8_scales(w):
    if w.shape.policy_head == "fromto":   # deployed network: fixed ReLU6 activation scale
        from oracle import deployed as OD
        blob = azgen.workload_weights(w)
        return OD.weight_scales(w.shape, blob), np.full(2 * w.shape.blocks + 1, 6.0 / 127.0, np.float32)
    return H.quant_scales(w.name, "int8")


@pytest.mark.parametrize("wname,K", [("net20x128_int8_b1024", 256), ("deployed14x160_int8_b1024", 256),
                                     ("net20x128_int8_b1024", 16)])
def test_noalloc_matches_pipeline_compact(wname, K):
    # K = 16: most rows have more legal moves than max_legal and are truncated
    import torch

    import paper_2609_37447_amd as az
    w = azgen.WORKLOADS[wname]
    blob = azgen.workload_weights(w)
    ws, acs = _int8_scales(w)
    MB = 128
    _print(f"case noalloc {wname} max_batch={MB} max_legal={K}")
    spec = az.spec_from_shape(w.shape, MB)
    net = az.az_net_load(spec, blob, "int8", ws, acs)
    pipe = None
    L = az.lib()
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    try:
        pipe = az.Pipeline(net, spec, MB, 1, False, max_legal=K)
        for B, seed in ((MB, 301), (37, 302)):
            planes, legal = azgen.make_inputs(w, n=B, seed=seed)
            # the existing entry point: the pipeline's compact outputs
            pipe.views[0][0][:B] = planes
            pipe.views[0][1][:B] = legal
            pipe.submit(0, B)
            st = L.az_pipeline_wait(pipe.p, 0)
            assert st in (az.AZ_OK, az.AZ_ERR_INVALID_ARG), st  # INVALID_ARG: some row overflowed K
            _, _, po, va, cnt = pipe.views[0]
            want_p, want_v, want_c = po[:B].copy(), va[:B].copy(), cnt[:B].copy()
            # the allocation-free entry point on device buffers
            pl = torch.from_numpy(planes).to(dev)
            lg = torch.from_numpy(legal).to(dev)
            pol = torch.full((B, K), 7.0, device=dev)
            cnt_d = torch.full((B,), -1, dtype=torch.int32, device=dev)
            val = torch.full((B,), 7.0, device=dev)
            torch.cuda.synchronize()
            live = az.az_debug_live_allocations()
            st = L.az_eval_batch_compact_noalloc(net, pl.data_ptr(), lg.data_ptr(), B, K, pol.data_ptr(),
                                                 cnt_d.data_ptr(), val.data_ptr(), stream.cuda_stream)
            assert st == az.AZ_OK, (st, L.az_last_error())
            torch.cuda.synchronize()
            assert az.az_debug_live_allocations() == live
            got_p, got_c, got_v = pol.cpu().numpy(), cnt_d.cpu().numpy(), val.cpu().numpy()
            assert np.array_equal(got_c, want_c), f"B={B} counts"
            assert np.array_equal(got_p, want_p), f"B={B} policy"
            assert np.array_equal(got_v, want_v), f"B={B} value"
            # the counts are the true numbers of legal cells, also past max_legal
            assert np.array_equal(got_c, (legal != 0).sum(axis=1).astype(np.int32))
            if K == 16:
                assert (got_c > K).any()
            _print(f"  B={B}: equal to the pipeline, {int(got_c.max())} legal moves at most")
    finally:
        if pipe is not None:
            pipe.close()
        az.az_net_free(net)


def test_noalloc_rejects_sizes_past_its_array_and_bad_arguments():
    import torch

    import paper_2609_37447_amd as az
    w = azgen.WORKLOADS["net20x128_bf16_b1024"]
    blob = azgen.workload_weights(w)
    net = az.az_net_load(az.spec_from_shape(w.shape, 1024), blob, "bf16")
    L = az.lib()
    E = az.AZ_ERR_INVALID_ARG
    try:
        dev = torch.device("cuda:0")
        pl = torch.zeros((1024, w.shape.in_planes, 8, 8), device=dev)
        lg = torch.zeros((1024, w.shape.n_moves), dtype=torch.uint8, device=dev)
        pol = torch.full((1024, 256), 7.0, device=dev)
        cnt = torch.zeros((1024,), dtype=torch.int32, device=dev)
        val = torch.full((1024,), 7.0, device=dev)
        args = (pl.data_ptr(), lg.data_ptr())
        outs = (pol.data_ptr(), cnt.data_ptr(), val.data_ptr())
        # 667 positions of 4,672 cells exceed the 3,112,960-float array; 666 fit
        assert L.az_eval_batch_compact_noalloc(net, *args, 667, 256, *outs, 0) == E
        assert b"scratch" in L.az_last_error() and b"666 positions" in L.az_last_error()
        assert L.az_eval_batch_compact_noalloc(None, *args, 8, 256, *outs, 0) == E
        assert L.az_eval_batch_compact_noalloc(net, *args, 8, 0, *outs, 0) == E
        assert L.az_eval_batch_compact_noalloc(net, *args, 8, w.shape.n_moves + 1, *outs, 0) == E
        assert L.az_eval_batch_compact_noalloc(net, *args, -1, 256, *outs, 0) == E
        assert L.az_eval_batch_compact_noalloc(net, *args, 1025, 256, *outs, 0) == E
        assert L.az_eval_batch_compact_noalloc(net, *args, 8, 256, None, cnt.data_ptr(), val.data_ptr(), 0) == E
        assert L.az_eval_batch_compact_noalloc(net, *args, 8, 256, pol.data_ptr() + 2, cnt.data_ptr(),
                                               val.data_ptr(), 0) == E
        assert L.az_eval_batch_compact_noalloc(net, *args, 0, 256, *outs, 0) == az.AZ_OK  # B = 0: no-op
        torch.cuda.synchronize()
        assert bool((pol == 7.0).all()) and bool((val == 7.0).all())
        # the largest batch that fits runs
        assert L.az_eval_batch_compact_noalloc(net, *args, 666, 256, *outs, 0) == az.AZ_OK
        torch.cuda.synchronize()
        assert bool((cnt[:666] == 0).all())  # no legal cells in an all-zero mask
    finally:
        az.az_net_free(net)
