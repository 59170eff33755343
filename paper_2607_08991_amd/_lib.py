"""ctypes binding of libsats.so: the C ABI of include/sats.h, one Python
function per entry point with the same name.

Marshalling only: tensors are passed as device pointers, the stream defaults
to torch's current stream, and a nonzero return code raises SatsError with the
library's own message.  Every step of the computation runs in the library's
HIP kernels; there is no fallback of any kind.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsats.so")

SATS_OK, SATS_ERR_NULL, SATS_ERR_SHAPE, SATS_ERR_HIP, SATS_ERR_WORKSPACE, SATS_ERR_ARG = 0, -1, -2, -3, -4, -5
SATS_ERR_DEVICE = -6
SATS_K_GATE, SATS_K_UP, SATS_K_DOWN, SATS_K_INSPECT, SATS_K_DENSE = 0, 1, 2, 3, 4
SATS_K_DEC_LAYER, SATS_K_DEC_LORA_V, SATS_K_CAL_ERR, SATS_K_CAL_GATEUP, SATS_K_ROUTE_ACCUM = 5, 6, 7, 8, 9
SATS_K_LORA_V = 10
SATS_K_DEC_REDUCE = 11
SATS_K_DENSE_DOWN = 12
SATS_K_DEC_REDUCE_LORA = 13
SATS_K_ROUTE_MERGE = 14
SATS_BATCH_AUTO, SATS_BATCH_MFMA, SATS_BATCH_SPLIT, SATS_BATCH_COMPACT = 0, 1, 2, 3
SATS_SINGLE_AUTO, SATS_SINGLE_OFF = 0, 1
SATS_PATH_SINGLE_TOKEN, SATS_PATH_BATCH_MFMA, SATS_PATH_BATCH_SPLIT, SATS_PATH_BATCH_COMPACT = 1, 2, 3, 4


class SatsOptions(ctypes.Structure):
    """sats_options of include/sats.h."""
    _fields_ = [("batch_path", ctypes.c_int), ("single_token", ctypes.c_int), ("dec_block_cols", ctypes.c_int),
                ("lora_per_token", ctypes.c_int)]

# exported symbols and their argument types (p = pointer, i = int64, s = stream, n = int32)
_P, _I, _S, _N = ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
_FWD = [_P] * 8 + [_I] * 4 + [_S]
_DENSE = [_P] * 5 + [_I] * 4 + [_S]
_INSPECT = _FWD + [_P] * 4
SIGNATURES = {
    "sats_mlp_forward": (_FWD, _N),
    "sats_mlp_dense": (_DENSE, _N),
    "sats_mlp_forward_noalloc": (_FWD, _N),
    "sats_mlp_forward_f32": (_FWD, _N),
    "sats_mlp_dense_f32": (_DENSE, _N),
    "sats_mlp_forward_inspect": (_INSPECT, _N),
    "sats_mlp_forward_inspect_f32": (_INSPECT, _N),
    "sats_reserve": ([_I, _I, _I, _I, _N, _S], _N),
    "sats_device_status": ([_S], _N),
    "sats_release": ([], _N),
    "sats_last_error": ([], ctypes.c_char_p),
    "sats_timing_begin": ([_N, _N], _N),
    "sats_timing_end": ([_N, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)], _N),
    "sats_kernel_name": ([_N], ctypes.c_char_p),
    "sats_mlp_forward_lora": ([_P] * 11 + [_I, ctypes.c_float] + [_P] * 3 + [_I] * 4 + [_S] + [_P] * 4, _N),
    "sats_mlp_forward_lora_f32": ([_P] * 11 + [_I, ctypes.c_float] + [_P] * 3 + [_I] * 4 + [_S] + [_P] * 4, _N),
    "sats_route_table": ([_P] * 3 + [_I, _P, _I, _I, ctypes.c_double] + [_P] * 4 + [_S], _N),
    "sats_set_options": ([ctypes.POINTER(SatsOptions)], _N),
    "sats_query_path": ([_I, _I, _I, _N, _N, _N, ctypes.POINTER(ctypes.c_int)], _N),
    "sats_calibration_curves": ([_P] * 4 + [_I] * 3 + [_P, _I] + [_P] * 4 + [_S], _N),
    "sats_calibrate_sats": ([_P, _I] + [_P] * 3 + [_I] * 3 + [ctypes.c_double] * 3 + [_N] + [_P] * 3 + [_S], _N),
}


class SatsError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"sats error {code}: {msg}")
        self.code = code


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libsats.so (built by paper_2607_08991_amd.build); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2607_08991_amd.build` "
                          "(the HIP library is required: there is no other implementation)")
    # Load torch's HIP runtime first so that the library binds to the same one;
    # a second copy of the runtime in the process would not see the device.
    try:
        import torch  # noqa: F401
    except ImportError:  # pragma: no cover - the library also works without torch
        pass
    lib = ctypes.CDLL(path)
    for name, (args, res) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("device tensors are required")
    if not t.is_contiguous():
        raise ValueError("contiguous tensors are required")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(rc: int):
    if rc != SATS_OK:
        raise SatsError(rc, load().sats_last_error().decode())


def _call(name, *args):
    _check(getattr(load(), name)(*args))


def sats_mlp_forward(x, token_ids, W_gate_T, W_up_T, W_down, thresholds, route_lut, out,
                     n_tokens, d, d_ff, n_layers, stream=None):
    name = "sats_mlp_forward_f32" if _is_f32(x) else "sats_mlp_forward"
    _call(name, _ptr(x), _ptr(token_ids), _ptr(W_gate_T), _ptr(W_up_T), _ptr(W_down),
          _ptr(thresholds), _ptr(route_lut), _ptr(out), n_tokens, d, d_ff, n_layers, _stream(stream))


def sats_mlp_forward_noalloc(x, token_ids, W_gate_T, W_up_T, W_down, thresholds, route_lut, out,
                             n_tokens, d, d_ff, n_layers, stream=None):
    """sats_mlp_forward on the library's fixed scratch array (bf16; allocates nothing)."""
    _call("sats_mlp_forward_noalloc", _ptr(x), _ptr(token_ids), _ptr(W_gate_T), _ptr(W_up_T), _ptr(W_down),
          _ptr(thresholds), _ptr(route_lut), _ptr(out), n_tokens, d, d_ff, n_layers, _stream(stream))


def sats_mlp_dense(x, W_gate_T, W_up_T, W_down, out, n_tokens, d, d_ff, n_layers, stream=None):
    name = "sats_mlp_dense_f32" if _is_f32(x) else "sats_mlp_dense"
    _call(name, _ptr(x), _ptr(W_gate_T), _ptr(W_up_T), _ptr(W_down), _ptr(out), n_tokens, d, d_ff,
          n_layers, _stream(stream))


def sats_mlp_forward_inspect(x, token_ids, W_gate_T, W_up_T, W_down, thresholds, route_lut, out,
                             n_tokens, d, d_ff, n_layers, stream=None, route_out=None,
                             active_count=None, active_idx=None, layer_in=None):
    name = "sats_mlp_forward_inspect_f32" if _is_f32(x) else "sats_mlp_forward_inspect"
    _call(name, _ptr(x), _ptr(token_ids), _ptr(W_gate_T), _ptr(W_up_T), _ptr(W_down),
          _ptr(thresholds), _ptr(route_lut), _ptr(out), n_tokens, d, d_ff, n_layers,
          _stream(stream), _ptr(route_out), _ptr(active_count), _ptr(active_idx), _ptr(layer_in))


def sats_mlp_forward_lora(x, token_ids, W_gate_T, W_up_T, W_down, adapters, rank, scale, thresholds, route_lut,
                          out, n_tokens, d, d_ff, n_layers, stream=None, route_out=None, active_count=None,
                          active_idx=None, layer_in=None):
    """LoRA-aware routed sparse forward; adapters = (A_gate, B_gate, A_up, B_up_T, A_down, B_down)."""
    name = "sats_mlp_forward_lora_f32" if _is_f32(x) else "sats_mlp_forward_lora"
    if len(adapters) != 6:
        raise ValueError("adapters = (A_gate, B_gate, A_up, B_up_T, A_down, B_down)")
    _call(name, _ptr(x), _ptr(token_ids), _ptr(W_gate_T), _ptr(W_up_T), _ptr(W_down),
          *(_ptr(m) for m in adapters), int(rank), float(scale), _ptr(thresholds), _ptr(route_lut), _ptr(out),
          n_tokens, d, d_ff, n_layers, _stream(stream), _ptr(route_out), _ptr(active_count), _ptr(active_idx),
          _ptr(layer_in))


def sats_reserve(max_tokens, d, d_ff, n_layers, elem_bytes, stream=None):
    _call("sats_reserve", max_tokens, d, d_ff, n_layers, elem_bytes, _stream(stream))


def sats_device_status(stream=None):
    """Synchronise the stream; raise SatsError if a device-side bounded wait gave up."""
    _call("sats_device_status", _stream(stream))


def sats_release():
    _call("sats_release")


def sats_set_options(batch_path=0, single_token=0, dec_block_cols=0, lora_per_token=0):
    """Execution options of the calling thread's later forward calls (all 0: the defaults)."""
    o = SatsOptions(batch_path, single_token, dec_block_cols, lora_per_token)
    _call("sats_set_options", ctypes.byref(o))


class options:
    """Context manager: sats_set_options(**kw) inside, the defaults after."""

    def __init__(self, **kw):
        self.kw = kw

    def __enter__(self):
        sats_set_options(**self.kw)
        return self

    def __exit__(self, *exc):
        _call("sats_set_options", None)
        return False


def sats_query_path(n_tokens, d, d_ff, elem_bytes, aligned16=True, n_cus=0) -> int:
    """The SATS_PATH_* a forward call of this shape takes under the current options (host only)."""
    path = ctypes.c_int(-1)
    _call("sats_query_path", n_tokens, d, d_ff, elem_bytes, int(bool(aligned16)), n_cus, ctypes.byref(path))
    return path.value


def sats_last_error() -> str:
    return load().sats_last_error().decode()


def sats_timing_begin(kind: int, capacity: int):
    _call("sats_timing_begin", kind, capacity)


def sats_timing_end(kind: int):
    """Returns (total_ms, count) of the launches timed since sats_timing_begin."""
    ms = ctypes.c_double(0.0)
    cnt = ctypes.c_int64(0)
    _check(load().sats_timing_end(kind, ctypes.byref(ms), ctypes.byref(cnt)))
    return ms.value, cnt.value


def sats_kernel_name(kind: int) -> str:
    return load().sats_kernel_name(kind).decode()


def _is_f32(x) -> bool:
    if isinstance(x, int) or x is None:
        raise ValueError("pass a tensor for x so the element type is known, or call load() directly")
    import torch
    if x.dtype == torch.float32:
        return True
    if x.dtype == torch.bfloat16:
        return False
    raise ValueError(f"x must be bfloat16 or float32, got {x.dtype}")


def _host(a, dtype):
    import numpy as np
    return np.ascontiguousarray(a, dtype=dtype)


def sats_calibration_curves(h, W_gate_T, W_up_T, W_down, n, d, d_ff, levels, err_rows=None, stream=None):
    """SATS curves of one layer (Eq. 3 candidates at `levels`, Eq. 6 errors, sparsities).

    h and the weights are device tensors (bf16); levels is a host sequence.
    Returns host arrays (t float32, err float64, sp float64); synchronises.
    """
    import numpy as np
    lv = _host(levels, np.float64)
    t = np.zeros(len(lv), np.float32)
    err = np.zeros(len(lv), np.float64)
    sp = np.zeros(len(lv), np.float64)
    _call("sats_calibration_curves", _ptr(h), _ptr(W_gate_T), _ptr(W_up_T), _ptr(W_down), n, d, d_ff,
          lv.ctypes.data, len(lv), t.ctypes.data, err.ctypes.data, sp.ctypes.data, _ptr(err_rows),
          _stream(stream))
    return t, err, sp


def sats_calibrate_sats(x_cal, n_cal, W_gate_T, W_up_T, W_down, d, d_ff, n_layers, s_tar,
                        coarse_step=0.05, fine_step=0.005, guardrail=True, stream=None):
    """SATS thresholds of a stack (Eq. 7-10, coarse to fine, final-layer guardrail).

    Returns (thresholds float32 [n_layers], budget b*, realized sparsity S(b*)); synchronises.
    """
    import numpy as np
    ts = np.zeros(n_layers, np.float32)
    b = ctypes.c_double(0.0)
    s = ctypes.c_double(0.0)
    _call("sats_calibrate_sats", _ptr(x_cal), n_cal, _ptr(W_gate_T), _ptr(W_up_T), _ptr(W_down), d, d_ff,
          n_layers, float(s_tar), float(coarse_step), float(fine_step), int(bool(guardrail)),
          ts.ctypes.data, ctypes.addressof(b), ctypes.addressof(s), _stream(stream))
    return ts, b.value, s.value


def sats_route_table(loss_base, loss_sparse, token_ids, heldout_ids, vocab, r_tar, route_lut, scores=None,
                     stream=None):
    """Routing table of Eq. 11-14 into route_lut (device uint8 [vocab]); returns (tau*, R(tau*)).

    Synchronises.  Empty splits may be passed as None.
    """
    tau = ctypes.c_double(0.0)
    r = ctypes.c_double(0.0)
    n = 0 if token_ids is None else token_ids.numel()
    nh = 0 if heldout_ids is None else heldout_ids.numel()
    _call("sats_route_table", _ptr(loss_base), _ptr(loss_sparse), _ptr(token_ids), n, _ptr(heldout_ids), nh,
          int(vocab), float(r_tar), _ptr(route_lut), _ptr(scores), ctypes.addressof(tau), ctypes.addressof(r),
          _stream(stream))
    return tau.value, r.value
