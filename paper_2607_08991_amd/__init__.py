"""Routed, threshold-sparsified gated MLP for AMD Instinct MI355X (gfx950).

The computation lives in libsats.so (hand-written HIP kernels behind the C ABI
of include/sats.h).  This package is its ctypes binding, the build script and
nothing else.
"""
from ._lib import (  # noqa: F401
    SatsError, load, sats_mlp_forward, sats_mlp_dense, sats_mlp_forward_inspect,
    sats_reserve, sats_release, sats_device_status, sats_last_error, sats_timing_begin, sats_timing_end,
    sats_kernel_name, SATS_K_GATE, SATS_K_UP, SATS_K_DOWN, SATS_K_INSPECT, SATS_K_DENSE, LIB_PATH,
    SATS_K_DEC_LAYER, SATS_K_DEC_LORA_V, SATS_K_CAL_ERR, SATS_K_CAL_GATEUP, sats_calibration_curves,
    sats_calibrate_sats, sats_mlp_forward_lora, sats_route_table, SATS_K_ROUTE_ACCUM, SATS_K_LORA_V,
    sats_set_options, options, sats_query_path, SATS_BATCH_AUTO, SATS_BATCH_MFMA, SATS_BATCH_SPLIT,
    SATS_BATCH_COMPACT, SATS_SINGLE_AUTO, SATS_SINGLE_OFF, SATS_PATH_SINGLE_TOKEN, SATS_PATH_BATCH_MFMA,
    SATS_PATH_BATCH_SPLIT, SATS_PATH_BATCH_COMPACT, sats_mlp_forward_noalloc,
    SATS_K_DEC_REDUCE, SATS_K_DENSE_DOWN, SATS_K_DEC_REDUCE_LORA, SATS_K_ROUTE_MERGE,
)
