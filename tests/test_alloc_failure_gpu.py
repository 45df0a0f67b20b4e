"""Allocation failures: every device or pinned-host allocation az_net_load and
az_pipeline_create make is forced to fail in turn, from the host
(az_debug_fail_allocation); each call must return AZ_ERR_NOMEM with a message,
and the library's count of live allocations must come back to where it was, so
nothing leaks on any failure path.  No kernel runs while a failure is armed.
"""

import numpy as np
import pytest

import azgen

pytestmark = pytest.mark.gpu


def test_weight_allocation_failure_returns_nomem_and_leaks_nothing():
    import paper_2609_37447_amd as az
    w = azgen.WORKLOADS["tiny_2x32_f32_b16"]
    blob = azgen.workload_weights(w)
    spec = az.spec_from_shape(w.shape, 16)
    base = az.az_debug_live_allocations()
    try:
        az.az_debug_fail_allocation(1)
        st, net = az.az_net_load(spec, blob, "f32", raise_on_error=False)
        assert st == az.AZ_ERR_NOMEM and net is None, st
        assert "hipMalloc" in az.az_last_error()
        assert az.az_debug_live_allocations() == base
    finally:
        az.az_debug_fail_allocation(0)
    net = az.az_net_load(spec, blob, "f32")
    assert az.az_debug_live_allocations() == base + 1
    az.az_net_free(net)
    assert az.az_debug_live_allocations() == base


@pytest.mark.parametrize("flags,max_legal", [(0, 0), (2, 64), (3, 64)])
def test_pipeline_allocation_failures_return_nomem_and_leak_nothing(flags, max_legal):
    # flags: 0 dense; 2 compact policy (one more device buffer per slot); 3 compact
    # with graphs (a stream per slot instead of three shared ones)
    import paper_2609_37447_amd as az
    w = azgen.WORKLOADS["net20x128_bf16_b256"]
    blob = azgen.workload_weights(w)
    net = az.az_net_load(az.spec_from_shape(w.shape, 64), blob, "bf16")
    try:
        base = az.az_debug_live_allocations()
        slots = 2
        per_slot = 3 + 3 + (1 if flags & 2 else 0)      # pinned host: planes, legal, outputs; device: same (+ dense)
        n_alloc = slots * per_slot
        for n in range(1, n_alloc + 1):
            az.az_debug_fail_allocation(n)
            try:
                st = az.az_pipeline_create(net, 64, slots, flags, max_legal, raise_on_error=False)
            finally:
                az.az_debug_fail_allocation(0)
            assert st == az.AZ_ERR_NOMEM, (n, st)
            assert az.az_debug_live_allocations() == base, n
        # armed past the last allocation: creation succeeds, every buffer is counted,
        # and freeing the pipeline returns them all
        az.az_debug_fail_allocation(n_alloc + 1)
        try:
            p = az.az_pipeline_create(net, 64, slots, flags, max_legal)
        finally:
            az.az_debug_fail_allocation(0)
        assert az.az_debug_live_allocations() == base + n_alloc
        az.az_pipeline_free(p)
        assert az.az_debug_live_allocations() == base
        # the handle still evaluates after the failed creations
        import torch
        planes, legal = azgen.make_inputs(w, n=8)
        dev = torch.device("cuda:0")
        pol = torch.empty((8, w.shape.n_moves), device=dev)
        val = torch.empty((8,), device=dev)
        az.eval_tensors(net, torch.from_numpy(planes).to(dev), torch.from_numpy(legal).to(dev), pol, val)
        torch.cuda.synchronize()
        assert np.allclose(pol.sum(dim=1).cpu().numpy(), 1.0, atol=1e-5)
    finally:
        az.az_net_free(net)
