"""The C-ABI library loads, exports every symbol include/az.h declares, and turns
argument errors into status codes before touching a device (no GPU needed)."""

import ctypes
import os
import re

import numpy as np
import pytest

import azgen
import paper_2609_37447_amd as az

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "az.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(az_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = az.lib()
    declared = _header_functions()
    assert declared, "no declarations parsed"
    assert set(declared) == set(az.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_weight_count_matches_layer_list():
    for w in azgen.WORKLOADS.values():
        spec = az.spec_from_shape(w.shape, w.batch)
        assert az.az_weight_count(spec) == w.shape.weight_count()
    assert az.az_weight_count(az.make_spec(20, 20, 128, 73, 128, max_batch=1)) == 5944523
    assert az.az_weight_count(az.make_spec(20, 2, 32, 73, 64, max_batch=1)) == 49451
    assert az.az_weight_count(az.make_spec(20, 24, 256, 73, 128, max_batch=1)) == 28397643
    assert az.az_weight_count(az.make_spec(20, 2, 32, 73, 64, max_batch=1, abi_version=7)) == 0
    # the deployed network: 52 planes, 14 x 160 with pooling every second block,
    # from-to head with 128-wide tokens, WDL head with 2 channels and 48 units
    dep = azgen.DEPLOYED_14X160
    assert az.az_weight_count(az.spec_from_shape(dep, 1)) == dep.weight_count() == 6255525


def test_version1_spec_layout_is_accepted():
    # a caller built against the first version passes only the first nine fields
    v1 = az.az_layer_spec_v1(1, 20, 20, 128, 73, 128, 0, 0.0, 1)
    ptr = ctypes.cast(ctypes.pointer(v1), ctypes.POINTER(az.az_layer_spec))
    assert az.lib().az_weight_count(ptr) == 5944523


def test_deployed_spec_validation_before_device():
    dep = azgen.DEPLOYED_14X160
    good = az.spec_from_shape(dep, 4)
    blob = np.zeros(dep.weight_count(), np.float32)
    ws = np.ones(2 * dep.blocks * dep.filters, np.float32)
    acs = np.ones(2 * dep.blocks + 1, np.float32)

    def spec(**kw):
        s = az.spec_from_shape(dep, 4)
        for k, v in kw.items():
            setattr(s, k, v)
        return s

    def st(sp, dtype, ws_=None, acs_=None):
        n = az.az_weight_count(sp)
        return _load_status(sp, np.zeros(max(n, 1), np.float32), dtype, ws_, acs_)

    # well-formed but not built: fp8 / f32, other widths, token width, head combinations
    assert _load_status(good, blob, "fp8", ws, acs) == az.AZ_ERR_UNSUPPORTED
    assert _load_status(good, blob, "f32") == az.AZ_ERR_UNSUPPORTED
    assert st(spec(filters=128), "bf16") == az.AZ_ERR_UNSUPPORTED
    assert st(spec(token_dim=64), "bf16") == az.AZ_ERR_UNSUPPORTED
    assert st(spec(value_channels=33), "bf16") == az.AZ_ERR_UNSUPPORTED
    assert st(spec(in_planes=65), "bf16") == az.AZ_ERR_UNSUPPORTED
    assert st(spec(value_head=az.AZ_VALUE_TANH, value_channels=1), "bf16") == az.AZ_ERR_UNSUPPORTED
    assert st(spec(policy_head=az.AZ_POLICY_PLANES, token_dim=0, policy_planes=73), "bf16") == az.AZ_ERR_UNSUPPORTED
    planes_pool = az.make_spec(20, 2, 128, 73, 128, max_batch=4, pool_every=2)
    assert st(planes_pool, "bf16") == az.AZ_ERR_UNSUPPORTED
    # malformed
    for bad in (spec(policy_planes=73), spec(token_dim=0), spec(value_channels=0), spec(policy_head=2),
                spec(value_head=5), spec(pool_every=-1), spec(filters=162)):
        assert az.az_weight_count(bad) == 0
        assert _load_status(bad, blob, "bf16") == az.AZ_ERR_INVALID_ARG
    # counts
    assert _load_status(good, blob[:-1], "bf16") == az.AZ_ERR_INVALID_ARG
    assert _load_status(good, blob, "int8", ws[:-1], acs) == az.AZ_ERR_INVALID_ARG
    assert _load_status(good, blob, "int8") == az.AZ_ERR_INVALID_ARG
    assert az.az_weight_count(az.make_spec(20, 0, 32, 73, 64, max_batch=1)) == 0


def test_status_strings():
    assert az.az_status_string(0) == "ok"
    for st in (-1, -2, -3, -4):
        assert az.az_status_string(st) and az.az_status_string(st) != "unknown status"
    assert az.az_status_string(5) == "unknown status"


def _load_status(spec, blob, dtype, ws=None, acs=None):
    st, h = az.az_net_load(spec, blob, dtype, ws, acs, raise_on_error=False)
    assert h is None
    return st


def test_load_rejects_bad_arguments_before_device():
    shape = azgen.WORKLOADS["tiny_2x32_f32_b16"].shape
    good = az.spec_from_shape(shape, 16)
    blob = np.zeros(shape.weight_count(), dtype=np.float32)
    # wrong weight count
    assert _load_status(good, blob[:-1], "f32") == az.AZ_ERR_INVALID_ARG
    assert "n_weights" in az.az_last_error()
    # malformed spec
    for bad in (az.make_spec(20, 2, 32, 73, 64, max_batch=0),
                az.make_spec(20, 2, 32, 73, 64, max_batch=4, abi_version=3),
                az.make_spec(20, 2, 32, 73, 64, max_batch=4, abi_version=0),
                az.make_spec(20, 2, 32, 73, 64, value_conv_relu=3, max_batch=4),
                az.make_spec(20, 2, 32, 73, 64, act_cap=-1.0, max_batch=4)):
        assert _load_status(bad, blob, "f32") == az.AZ_ERR_INVALID_ARG
    # unknown dtype
    assert _load_status(good, blob, 9) == az.AZ_ERR_INVALID_ARG
    # unsupported shapes
    assert _load_status(good, blob, "bf16") == az.AZ_ERR_UNSUPPORTED          # F=32 on MFMA
    sp = az.make_spec(40, 2, 32, 73, 64, max_batch=4)
    assert _load_status(sp, np.zeros(az.az_weight_count(sp), np.float32), "f32") == az.AZ_ERR_UNSUPPORTED
    sp = az.make_spec(20, 2, 32, 96, 64, max_batch=4)
    assert _load_status(sp, np.zeros(az.az_weight_count(sp), np.float32), "f32") == az.AZ_ERR_UNSUPPORTED
    sp = az.make_spec(20, 2, 36, 73, 64, max_batch=4)
    assert _load_status(sp, np.zeros(az.az_weight_count(sp), np.float32), "f32") == az.AZ_ERR_UNSUPPORTED
    # scales: missing for quantised dtypes, present for float ones, wrong counts, non-positive
    shp = azgen.WORKLOADS["net20x128_int8_b1024"].shape
    sp = az.spec_from_shape(shp, 8)
    b2 = np.zeros(shp.weight_count(), np.float32)
    ws = np.ones(2 * shp.blocks * shp.filters, np.float32)
    acs = np.ones(2 * shp.blocks + 1, np.float32)
    assert _load_status(sp, b2, "int8") == az.AZ_ERR_INVALID_ARG
    assert _load_status(sp, b2, "int8", ws[:-1], acs) == az.AZ_ERR_INVALID_ARG
    assert _load_status(sp, b2, "fp8", ws, acs[:-1]) == az.AZ_ERR_INVALID_ARG
    assert _load_status(sp, b2, "bf16", ws, acs) == az.AZ_ERR_INVALID_ARG
    bad = ws.copy()
    bad[3] = 0.0
    assert _load_status(sp, b2, "int8", bad, acs) == az.AZ_ERR_INVALID_ARG
    bad = acs.copy()
    bad[0] = np.nan
    assert _load_status(sp, b2, "fp8", ws, bad) == az.AZ_ERR_INVALID_ARG


def test_eval_and_free_reject_null_handle():
    assert az.az_eval_batch(None, 0, 0, 4, 0, 0, 0, raise_on_error=False) == az.AZ_ERR_INVALID_ARG
    assert az.az_eval_batch_wdl(None, 0, 0, 4, 0, 0, 0, 0, raise_on_error=False) == az.AZ_ERR_INVALID_ARG
    assert az.lib().az_net_moves(None) == az.AZ_ERR_INVALID_ARG
    assert az.az_net_set_tiling(None, 1, raise_on_error=False) == az.AZ_ERR_INVALID_ARG
    assert az.az_net_device_bytes(None) == 0
    az.az_net_free(None)                                     # no-op
    with pytest.raises(az.AzError):
        az.az_eval_batch(None, 0, 0, 4, 0, 0, 0)


def test_compare_outputs_rejects_bad_arguments_before_device():
    L = az.lib()
    p = ctypes.c_void_p(16)  # never dereferenced: every call below fails validation first
    assert L.az_compare_outputs(p, p, p, p, p, -1, 4672, p, None) == az.AZ_ERR_INVALID_ARG
    assert L.az_compare_outputs(p, p, p, p, p, 4, 0, p, None) == az.AZ_ERR_INVALID_ARG
    assert L.az_compare_outputs(None, p, p, p, p, 4, 4672, p, None) == az.AZ_ERR_INVALID_ARG
    assert L.az_compare_outputs(p, p, p, p, p, 4, 4672, None, None) == az.AZ_ERR_INVALID_ARG
    q = ctypes.c_void_p(18)  # misaligned float buffer
    assert L.az_compare_outputs(q, p, p, p, p, 4, 4672, p, None) == az.AZ_ERR_INVALID_ARG
    assert b"aligned" in L.az_last_error()
    assert L.az_compare_outputs(None, None, None, None, None, 0, 4672, None, None) == az.AZ_OK


def test_pipeline_rejects_bad_arguments_before_device():
    L = az.lib()
    out = ctypes.c_void_p()
    assert L.az_pipeline_create(None, 4, 2, 0, 0, ctypes.byref(out)) == az.AZ_ERR_INVALID_ARG
    assert out.value is None
    p = ctypes.c_void_p(16)  # never dereferenced: slots, flags and max_legal are checked first
    assert L.az_pipeline_create(p, 4, 0, 0, 0, ctypes.byref(out)) == az.AZ_ERR_INVALID_ARG
    assert L.az_pipeline_create(p, 4, 65, 0, 0, ctypes.byref(out)) == az.AZ_ERR_INVALID_ARG
    assert L.az_pipeline_create(p, 4, 2, 0, 0, None) == az.AZ_ERR_INVALID_ARG
    assert L.az_pipeline_create(p, 4, 2, 8, 0, ctypes.byref(out)) == az.AZ_ERR_INVALID_ARG
    assert b"flags" in L.az_last_error()
    compact = az.AZ_PIPE_COMPACT_POLICY
    assert L.az_pipeline_create(p, 4, 2, compact, 0, ctypes.byref(out)) == az.AZ_ERR_INVALID_ARG
    assert L.az_pipeline_create(p, 4, 2, 0, 64, ctypes.byref(out)) == az.AZ_ERR_INVALID_ARG
    assert b"max_legal" in L.az_last_error()
    for fn in (L.az_pipeline_query, L.az_pipeline_wait):
        assert fn(None, 0) == az.AZ_ERR_INVALID_ARG
    assert L.az_pipeline_submit(None, 0, 1) == az.AZ_ERR_INVALID_ARG
    assert L.az_pipeline_slot(None, 0, None, None, None, None, None) == az.AZ_ERR_INVALID_ARG
    sec = ctypes.c_double()
    assert L.az_pipeline_drive(None, 1, 1, 1, 0, 1, ctypes.byref(sec)) == az.AZ_ERR_INVALID_ARG
    assert b"az_pipeline_drive" in L.az_last_error()
    L.az_pipeline_free(None)                                 # no-op
