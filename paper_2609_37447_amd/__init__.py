"""MI355X (gfx950) library for batched policy/value evaluation of search leaves.

The computation lives in libaz_mi355x.so (HIP kernels behind the C ABI of
include/az.h); this package is its Python binding.
"""

from ._binding import (AZ_ABI_VERSION, AZ_BF16, AZ_ERR_DEVICE, AZ_ERR_INVALID_ARG,  # noqa: F401
                       AZ_ERR_NOMEM, AZ_ERR_UNSUPPORTED, AZ_F32, AZ_FP8_E4M3, AZ_INT8, AZ_OK,
                       DTYPES, EXPORTS, AzError, az_compare_outputs, az_eval_batch, az_last_error,
                       az_layer_spec, az_layer_spec_v1, az_eval_batch_wdl, az_net_moves,
                       AZ_POLICY_PLANES, AZ_POLICY_FROMTO, AZ_VALUE_TANH, AZ_VALUE_WDL,
                       az_net_device_bytes, az_net_free, az_net_load, az_net_set_tiling,
                       az_net_tiling_for, az_status_string, az_weight_count, eval_tensors, lib,
                       make_spec, spec_from_shape, validate, Pipeline, AZ_PIPE_COMPACT_POLICY, AZ_PIPE_GRAPHS,
                       az_pipeline_create,
                       az_pipeline_free, az_pipeline_query, az_pipeline_slot, az_pipeline_submit,
                       az_pipeline_wait, az_pipeline_drive, az_debug_fail_allocation, az_debug_live_allocations)
