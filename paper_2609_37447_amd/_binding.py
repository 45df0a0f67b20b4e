"""ctypes binding of the C ABI in include/az.h (argument marshalling only).

Every computation runs in the HIP library; this module only converts Python
arguments to the C types and raises on a non-zero status.  It fails loudly if
the library has not been built.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libaz_mi355x.so")

AZ_ABI_VERSION = 2
AZ_POLICY_PLANES, AZ_POLICY_FROMTO = 0, 1
AZ_VALUE_TANH, AZ_VALUE_WDL = 0, 1
AZ_F32, AZ_BF16, AZ_INT8, AZ_FP8_E4M3 = 0, 1, 2, 3
DTYPES = {"f32": AZ_F32, "bf16": AZ_BF16, "int8": AZ_INT8, "fp8": AZ_FP8_E4M3}
AZ_OK, AZ_ERR_INVALID_ARG, AZ_ERR_UNSUPPORTED, AZ_ERR_NOMEM, AZ_ERR_DEVICE = 0, -1, -2, -3, -4

# Every symbol include/az.h declares.
EXPORTS = ("az_weight_count", "az_net_load", "az_eval_batch", "az_eval_batch_wdl", "az_net_moves",
           "az_net_set_tiling",
           "az_net_tiling_for", "az_net_device_bytes", "az_net_free", "az_compare_outputs",
           "az_pipeline_create", "az_pipeline_slot", "az_pipeline_submit", "az_pipeline_query",
           "az_pipeline_wait", "az_pipeline_drive", "az_pipeline_free", "az_debug_fail_allocation",
           "az_debug_live_allocations", "az_eval_batch_compact_noalloc",
           "az_status_string", "az_last_error")


class az_layer_spec(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_int32), ("in_planes", ctypes.c_int32),
                ("blocks", ctypes.c_int32), ("filters", ctypes.c_int32),
                ("policy_planes", ctypes.c_int32), ("value_hidden", ctypes.c_int32),
                ("value_conv_relu", ctypes.c_int32), ("act_cap", ctypes.c_float),
                ("max_batch", ctypes.c_int32),
                # abi_version 2
                ("pool_every", ctypes.c_int32), ("policy_head", ctypes.c_int32),
                ("token_dim", ctypes.c_int32), ("value_head", ctypes.c_int32),
                ("value_channels", ctypes.c_int32)]


class az_layer_spec_v1(ctypes.Structure):
    """The version-1 layout (the first nine fields), as older callers pass it."""
    _fields_ = az_layer_spec._fields_[:9]


class AzError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


_lib = None


def lib():
    """The loaded library (CDLL); raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2609_37447_amd.build`")
        # torch ships its own HIP runtime under the same soname as ROCm's
        # (libamdhip64.so.7).  Loading torch first makes this library bind to
        # that one copy; loaded the other way round, torch would bring up a
        # second runtime beside it and find no GPU.
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        FP = ctypes.POINTER(ctypes.c_float)
        L.az_weight_count.argtypes, L.az_weight_count.restype = [ctypes.POINTER(az_layer_spec)], SZ
        L.az_net_load.argtypes = [ctypes.POINTER(az_layer_spec), FP, SZ, I32, FP, SZ, FP, SZ,
                                  ctypes.POINTER(P)]
        L.az_net_load.restype = ctypes.c_int
        L.az_eval_batch.argtypes = [P, P, P, I32, P, P, P]
        L.az_eval_batch.restype = ctypes.c_int
        L.az_eval_batch_wdl.argtypes = [P, P, P, I32, P, P, P, P]
        L.az_eval_batch_wdl.restype = ctypes.c_int
        L.az_net_moves.argtypes, L.az_net_moves.restype = [P], ctypes.c_int
        L.az_net_set_tiling.argtypes, L.az_net_set_tiling.restype = [P, I32], ctypes.c_int
        L.az_net_tiling_for.argtypes, L.az_net_tiling_for.restype = [P, I32], ctypes.c_int
        L.az_net_device_bytes.argtypes, L.az_net_device_bytes.restype = [P], SZ
        L.az_net_free.argtypes, L.az_net_free.restype = [P], None
        L.az_compare_outputs.argtypes = [P, P, P, P, P, I32, I32, P, P]
        L.az_compare_outputs.restype = ctypes.c_int
        L.az_pipeline_create.argtypes = [P, I32, I32, I32, I32, ctypes.POINTER(P)]
        L.az_pipeline_create.restype = ctypes.c_int
        L.az_pipeline_slot.argtypes = [P, I32, ctypes.POINTER(P), ctypes.POINTER(P), ctypes.POINTER(P),
                                       ctypes.POINTER(P), ctypes.POINTER(P)]
        L.az_pipeline_slot.restype = ctypes.c_int
        L.az_pipeline_submit.argtypes, L.az_pipeline_submit.restype = [P, I32, I32], ctypes.c_int
        L.az_pipeline_query.argtypes, L.az_pipeline_query.restype = [P, I32], ctypes.c_int
        L.az_pipeline_wait.argtypes, L.az_pipeline_wait.restype = [P, I32], ctypes.c_int
        L.az_pipeline_free.argtypes, L.az_pipeline_free.restype = [P], None
        L.az_pipeline_drive.argtypes = [P, I32, I32, I32, I32, I32, ctypes.POINTER(ctypes.c_double)]
        L.az_pipeline_drive.restype = ctypes.c_int
        L.az_eval_batch_compact_noalloc.argtypes = [P, P, P, I32, I32, P, P, P, P]
        L.az_eval_batch_compact_noalloc.restype = ctypes.c_int
        L.az_debug_fail_allocation.argtypes, L.az_debug_fail_allocation.restype = [I32], None
        L.az_debug_live_allocations.argtypes, L.az_debug_live_allocations.restype = [], ctypes.c_int64
        L.az_status_string.argtypes, L.az_status_string.restype = [ctypes.c_int], ctypes.c_char_p
        L.az_last_error.argtypes, L.az_last_error.restype = [], ctypes.c_char_p
        _lib = L
    return _lib


def make_spec(in_planes, blocks, filters, policy_planes, value_hidden, value_conv_relu=0,
              act_cap=0.0, max_batch=1, abi_version=AZ_ABI_VERSION, pool_every=0,
              policy_head=AZ_POLICY_PLANES, token_dim=0, value_head=AZ_VALUE_TANH,
              value_channels=1) -> az_layer_spec:
    return az_layer_spec(abi_version, in_planes, blocks, filters, policy_planes, value_hidden,
                         value_conv_relu, act_cap, max_batch, pool_every, policy_head, token_dim,
                         value_head, value_channels)


def spec_from_shape(shape, max_batch: int) -> az_layer_spec:
    """az_layer_spec from any object with the NetShape attribute names."""
    fromto = getattr(shape, "policy_head", "planes") == "fromto"
    wdl = getattr(shape, "value_head", "tanh") == "wdl"
    return make_spec(shape.in_planes, shape.blocks, shape.filters, shape.policy_planes,
                     shape.value_hidden, shape.value_conv_relu, shape.act_cap, max_batch,
                     pool_every=getattr(shape, "pool_every", 0),
                     policy_head=AZ_POLICY_FROMTO if fromto else AZ_POLICY_PLANES,
                     token_dim=shape.token_dim if fromto else 0,
                     value_head=AZ_VALUE_WDL if wdl else AZ_VALUE_TANH,
                     value_channels=getattr(shape, "value_channels", 1))


def _check(status: int, where: str) -> int:
    if status < 0:
        detail = lib().az_last_error().decode(errors="replace")
        raise AzError(status, where, detail or az_status_string(status))
    return status


def _fptr(a):
    if a is None:
        return None, 0
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a, a.size


def az_weight_count(spec: az_layer_spec) -> int:
    return int(lib().az_weight_count(ctypes.byref(spec)))


def az_net_load(spec: az_layer_spec, weights, dtype, w_scales=None, act_scales=None,
                raise_on_error: bool = True):
    """Returns the handle (int), or (status) when raise_on_error is False and it fails."""
    dt = DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
    w, nw = _fptr(weights)
    ws, nws = _fptr(w_scales)
    acs, nacs = _fptr(act_scales)
    FP = ctypes.POINTER(ctypes.c_float)
    cast = lambda a: a.ctypes.data_as(FP) if a is not None else None  # noqa: E731
    out = ctypes.c_void_p()
    st = lib().az_net_load(ctypes.byref(spec), cast(w), nw, dt, cast(ws), nws, cast(acs), nacs,
                           ctypes.byref(out))
    if not raise_on_error:
        return (st, out.value) if st == AZ_OK else (st, None)
    _check(st, "az_net_load")
    return out.value


def az_eval_batch(net, planes_ptr: int, legal_ptr: int, B: int, policy_ptr: int, value_ptr: int,
                  stream: int = 0, raise_on_error: bool = True) -> int:
    st = lib().az_eval_batch(net, planes_ptr, legal_ptr, int(B), policy_ptr, value_ptr, stream)
    return _check(st, "az_eval_batch") if raise_on_error else st


def az_eval_batch_wdl(net, planes_ptr: int, legal_ptr: int, B: int, policy_ptr: int, value_ptr: int,
                      wdl_ptr, stream: int = 0, raise_on_error: bool = True) -> int:
    st = lib().az_eval_batch_wdl(net, planes_ptr, legal_ptr, int(B), policy_ptr, value_ptr, wdl_ptr, stream)
    return _check(st, "az_eval_batch_wdl") if raise_on_error else st


def az_net_moves(net) -> int:
    return _check(lib().az_net_moves(net), "az_net_moves")


def az_net_set_tiling(net, tiling: int, raise_on_error: bool = True) -> int:
    st = lib().az_net_set_tiling(net, int(tiling))
    return _check(st, "az_net_set_tiling") if raise_on_error else st


def az_net_tiling_for(net, B: int) -> int:
    return _check(lib().az_net_tiling_for(net, int(B)), "az_net_tiling_for")


def az_net_device_bytes(net) -> int:
    return int(lib().az_net_device_bytes(net))


def az_net_free(net) -> None:
    lib().az_net_free(net)


def az_debug_fail_allocation(n: int) -> None:
    lib().az_debug_fail_allocation(int(n))


def az_debug_live_allocations() -> int:
    return int(lib().az_debug_live_allocations())


def az_status_string(status: int) -> str:
    return lib().az_status_string(int(status)).decode()


def az_last_error() -> str:
    return lib().az_last_error().decode(errors="replace")


# --------------------------------------------------------------------------- #
# torch convenience: device tensors and streams (PyTorch provides memory and
# streams only)
# --------------------------------------------------------------------------- #
def eval_tensors(net, planes, legal, policy, value, stream=None, wdl=None) -> int:
    """az_eval_batch (az_eval_batch_wdl when wdl is given) on torch CUDA tensors;
    stream defaults to torch's current one."""
    import torch
    B = planes.shape[0]
    named = [("planes", planes), ("legal", legal), ("policy", policy), ("value", value)]
    if wdl is not None:
        named.append(("wdl", wdl))
    for name, t in named:
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous device tensor")
    if planes.dtype != torch.float32 or legal.dtype != torch.uint8:
        raise ValueError("planes must be float32 and legal uint8")
    if policy.dtype != torch.float32 or value.dtype != torch.float32:
        raise ValueError("policy and value must be float32")
    if legal.shape[0] != B or policy.shape[0] != B or value.shape[0] != B:
        raise ValueError("batch sizes differ")
    s = torch.cuda.current_stream() if stream is None else stream
    if wdl is not None:
        if wdl.dtype != torch.float32 or tuple(wdl.shape) != (B, 3):
            raise ValueError("wdl must be float32 [B, 3]")
        return az_eval_batch_wdl(net, planes.data_ptr(), legal.data_ptr(), B, policy.data_ptr(),
                                 value.data_ptr(), wdl.data_ptr(), s.cuda_stream)
    return az_eval_batch(net, planes.data_ptr(), legal.data_ptr(), B, policy.data_ptr(),
                         value.data_ptr(), s.cuda_stream)


def az_compare_outputs(policy_ref, value_ref, policy_test, value_test, legal, B: int, n_moves: int,
                       row_metrics, stream) -> int:
    """Device pointers (ints); per-row {top-1 equal, KL(ref || test), |dV|} into row_metrics."""
    return _check(lib().az_compare_outputs(policy_ref, value_ref, policy_test, value_test, legal, B,
                                           n_moves, row_metrics, stream), "az_compare_outputs")


def validate(net_test, net_ref, planes, legal, min_top1: float = 0.8, max_kl: float = 0.1,
             max_dv: float = 0.25, stream=None) -> dict:
    """Deployment validation of a loaded network against a reference network on the
    same positions (torch device tensors planes [B][C][8][8] f32 and legal [B][P*64]
    u8): both are evaluated, the library compares them row by row, and the rows are
    summarised as the mean top-1 legal-move agreement (over rows with a legal move),
    the mean legal-policy KL(ref || test) and the largest value error.  The default
    bounds separate a faithful quantised network from a broken engine (the paper's
    faulty refit showed KL near 1); callers set their own."""
    import torch
    B, NM = legal.shape
    dev = planes.device
    out = {}
    for key, net in (("test", net_test), ("ref", net_ref)):
        pol = torch.empty((B, NM), device=dev)
        val = torch.empty((B,), device=dev)
        eval_tensors(net, planes, legal, pol, val, stream)
        out[key] = (pol, val)
    rows = torch.empty((B, 3), device=dev)
    s = torch.cuda.current_stream() if stream is None else stream
    az_compare_outputs(out["ref"][0].data_ptr(), out["ref"][1].data_ptr(), out["test"][0].data_ptr(),
                       out["test"][1].data_ptr(), legal.data_ptr(), B, NM, rows.data_ptr(), s.cuda_stream)
    s.synchronize()
    r = rows.cpu().numpy().astype(np.float64)
    has = (legal != 0).any(dim=1).cpu().numpy().astype(bool)
    top1 = float(r[has, 0].mean()) if has.any() else 1.0
    kl = float(r[:, 1].mean())
    dv = float(r[:, 2].max())
    return {"top1": top1, "kl": kl, "dv_max": dv, "rows": r,
            "passed": top1 >= min_top1 and kl <= max_kl and dv <= max_dv}


AZ_PIPE_GRAPHS = 1
AZ_PIPE_COMPACT_POLICY = 2


def az_pipeline_create(net, max_batch: int, slots: int, flags: int = 0, max_legal: int = 0,
                       raise_on_error: bool = True):
    """Returns the pipeline handle, or (status) when raise_on_error is False and it fails."""
    out = ctypes.c_void_p()
    st = lib().az_pipeline_create(net, max_batch, slots, flags, max_legal, ctypes.byref(out))
    if st != AZ_OK and not raise_on_error:
        return st
    _check(st, "az_pipeline_create")
    return out


def az_pipeline_slot(p, slot: int):
    """Host pointers (planes, legal, policy, value, legal_count) of a slot."""
    ptrs = [ctypes.c_void_p() for _ in range(5)]
    _check(lib().az_pipeline_slot(p, slot, *[ctypes.byref(x) for x in ptrs]), "az_pipeline_slot")
    return tuple(x.value for x in ptrs)


def az_pipeline_submit(p, slot: int, B: int) -> int:
    return _check(lib().az_pipeline_submit(p, slot, B), "az_pipeline_submit")


def az_pipeline_query(p, slot: int) -> int:
    return _check(lib().az_pipeline_query(p, slot), "az_pipeline_query")


def az_pipeline_wait(p, slot: int) -> int:
    return _check(lib().az_pipeline_wait(p, slot), "az_pipeline_wait")


def az_pipeline_drive(p, workers: int, slots_per_worker: int, B: int, warmup: int, batches: int) -> float:
    """Wall seconds of `batches` native round-robin submissions per worker thread."""
    sec = ctypes.c_double()
    _check(lib().az_pipeline_drive(p, workers, slots_per_worker, B, warmup, batches, ctypes.byref(sec)),
           "az_pipeline_drive")
    return sec.value


def az_pipeline_free(p) -> None:
    lib().az_pipeline_free(p)


class Pipeline:
    """A pipeline with numpy views of its slots' pinned host buffers:
    views[k] = (planes, legal, policy, value, legal_count or None)."""

    def __init__(self, net, spec, max_batch: int, slots: int, use_graphs: bool = False,
                 max_legal: int = 0):
        flags = (AZ_PIPE_GRAPHS if use_graphs else 0) | (AZ_PIPE_COMPACT_POLICY if max_legal else 0)
        self.p = az_pipeline_create(net, max_batch, slots, flags, max_legal)
        n_moves = az_net_moves(net)
        f32 = ctypes.POINTER(ctypes.c_float)
        u8 = ctypes.POINTER(ctypes.c_uint8)
        i32 = ctypes.POINTER(ctypes.c_int32)
        self.views = []
        for k in range(slots):
            pp, lp, po, vp, cp = az_pipeline_slot(self.p, k)
            self.views.append((
                np.ctypeslib.as_array(ctypes.cast(pp, f32), (max_batch, spec.in_planes, 8, 8)),
                np.ctypeslib.as_array(ctypes.cast(lp, u8), (max_batch, n_moves)),
                np.ctypeslib.as_array(ctypes.cast(po, f32), (max_batch, max_legal or n_moves)),
                np.ctypeslib.as_array(ctypes.cast(vp, f32), (max_batch,)),
                np.ctypeslib.as_array(ctypes.cast(cp, i32), (max_batch,)) if max_legal else None,
            ))

    def submit(self, slot: int, B: int) -> None:
        az_pipeline_submit(self.p, slot, B)

    def wait(self, slot: int) -> None:
        az_pipeline_wait(self.p, slot)

    def query(self, slot: int) -> bool:
        return az_pipeline_query(self.p, slot) == 0

    def drive(self, workers: int, slots_per_worker: int, B: int, warmup: int, batches: int) -> float:
        return az_pipeline_drive(self.p, workers, slots_per_worker, B, warmup, batches)

    def close(self) -> None:
        if self.p is not None:
            az_pipeline_free(self.p)
            self.p = None
