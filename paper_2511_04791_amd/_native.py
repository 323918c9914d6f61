"""ctypes declarations of the C ABI in include/duet.h (argument marshalling only)."""
from __future__ import annotations

import ctypes
import os
import threading

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libduet.so")

c_int32, c_int64, c_double, c_size_t, c_void_p = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_size_t, ctypes.c_void_p

OK = 0
ERRORS = {-1: "EINVAL", -2: "EUNSUPPORTED", -3: "EWORKSPACE", -4: "EHIP", -5: "ENOMEM", -6: "EPAGE", -7: "EIO"}
BF16, F32 = 0, 1
KIND_PREFILL, KIND_DECODE = 0, 1
AGG, SPLIT, CONCURRENT = 0, 1, 2
STATUS_SLO_INFEASIBLE, STATUS_UNCALIBRATED = 1, 2
TOTAL_CUS, CU_STEP, SPLIT_STEP = 256, 8, 32


class Shape(ctypes.Structure):
    _fields_ = [("num_q_heads", c_int32), ("num_kv_heads", c_int32), ("head_dim", c_int32),
                ("page_size", c_int32), ("dtype", c_int32), ("num_layers", c_int32)]


class SeqMeta(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("q_start", c_int32), ("q_len", c_int32), ("cached_len", c_int32)]


class Batch(ctypes.Structure):
    _fields_ = [("reqs", ctypes.POINTER(SeqMeta)), ("num_reqs", c_int32)]


class CuSplit(ctypes.Structure):
    _fields_ = [("mode", c_int32), ("cus_prefill", c_int32), ("cus_decode", c_int32), ("k_decode_steps", c_int32)]


class BlockShape(ctypes.Structure):
    _fields_ = [("ffn_dim", c_int32), ("vocab_size", c_int32), ("flags", c_int32)]


class BlockWeights(ctypes.Structure):
    _fields_ = [("attn_norm", c_void_p), ("w_qkv", c_void_p), ("w_o", c_void_p), ("ffn_norm", c_void_p),
                ("w_gate_up", c_void_p), ("w_down", c_void_p)]


class KernelTimes(ctypes.Structure):
    _fields_ = [("decode_partial_us", c_double), ("decode_reduce_us", c_double), ("prefill_us", c_double),
                ("decode_total_us", c_double), ("iteration_us", c_double),
                ("decode_start_us", c_double), ("prefill_start_us", c_double), ("prefill_total_us", c_double),
                ("layers", c_double), ("decode_steps", c_double), ("decode_step_us", c_double),
                ("decode_first_step_us", c_double)]


P = ctypes.POINTER
_SIGS = {
    "duet_model_create": (c_int32, [P(c_void_p)]),
    "duet_model_destroy": (c_int32, [c_void_p]),
    "duet_batch_work": (c_int32, [P(Shape), P(Batch), c_int32, P(c_double), P(c_double)]),
    "duet_model_set_sharing_tables": (c_int32, [c_void_p, c_int32, P(c_int32), P(c_double), P(c_double)]),
    "duet_model_get_sharing_tables": (c_int32, [c_void_p, c_int32, P(c_int32), P(c_double), P(c_double),
                                                P(c_int32)]),
    "duet_model_set_tables": (c_int32, [c_void_p, c_int32, P(c_int32), P(c_double), P(c_double)]),
    "duet_model_get_tables": (c_int32, [c_void_p, c_int32, P(c_int32), P(c_double), P(c_double)]),
    "duet_model_set_efficiency": (c_int32, [c_void_p, c_double, c_double]),
    "duet_model_set_launch_tables": (c_int32, [c_void_p, c_int32, P(c_int32), P(c_double), P(c_double)]),
    "duet_model_get_launch_tables": (c_int32, [c_void_p, c_int32, P(c_int32), P(c_double), P(c_double)]),
    "duet_model_save": (c_int32, [c_void_p, ctypes.c_char_p]),
    "duet_model_load": (c_int32, [c_void_p, ctypes.c_char_p]),
    "duet_predict_iter_latency": (c_int32, [c_void_p, P(Shape), P(Batch), CuSplit, P(c_double)]),
    "duet_predict_partition_latency": (c_int32, [c_void_p, P(Shape), P(Batch), c_int32, c_int32, c_int32, P(c_double)]),
    "duet_choose_cu_split": (c_int32, [c_void_p, P(Shape), P(Batch), c_double, c_int32, P(CuSplit), P(c_double),
                                       P(c_double), P(c_int32)]),
    "duet_predict_model_latency": (c_int32, [c_void_p, P(Shape), P(BlockShape), P(Batch), CuSplit, P(c_double)]),
    "duet_choose_cu_split_model": (c_int32, [c_void_p, P(Shape), P(BlockShape), P(Batch), c_double, c_int32,
                                             P(CuSplit), P(c_double), P(c_double), P(c_int32)]),
    "duet_init": (c_int32, [c_int32, P(c_void_p)]),
    "duet_init_with_model": (c_int32, [c_int32, ctypes.c_char_p, P(c_void_p)]),
    "duet_destroy": (c_int32, [c_void_p]),
    "duet_ctx_model": (c_void_p, [c_void_p]),
    "duet_workspace_bytes": (c_int32, [P(Shape), P(Batch), P(c_size_t)]),
    "duet_block_workspace_bytes": (c_int32, [P(Shape), P(BlockShape), P(Batch), c_int32, P(c_size_t)]),
    "duet_engine_create": (c_int32, [c_int32, c_int32, c_int64, c_int32, ctypes.c_uint64, P(c_void_p)]),
    "duet_engine_destroy": (c_int32, [c_void_p]),
    "duet_engine_add_request": (c_int32, [c_void_p, c_int32, c_int32, P(c_int64)]),
    "duet_engine_step": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int32, P(c_int32)]),
    "duet_engine_step_lookahead": (c_int32, [c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_int32, P(c_int32)]),
    "duet_engine_complete": (c_int32, [c_void_p]),
    "duet_engine_complete_lookahead": (c_int32, [c_void_p, c_int32]),
    "duet_engine_stats": (c_int32, [c_void_p, P(c_int64), P(c_int64), P(c_int64)]),
    "duet_block_forward": (c_int32, [c_void_p, P(Shape), P(BlockShape), P(BlockWeights), ctypes.c_float, c_void_p,
                                     P(c_void_p), P(c_void_p), P(c_void_p), c_int64, c_void_p, c_int32, P(Batch), CuSplit,
                                     c_void_p, c_size_t, c_void_p]),
    "duet_block_buffers": (c_int32, [P(Shape), P(BlockShape), P(Batch), c_int32, P(c_size_t)]),
    "duet_rmsnorm": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_int32, ctypes.c_float, c_void_p]),
    "duet_swiglu": (c_int32, [c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_void_p]),
    "duet_qkv_split": (c_int32, [c_void_p, P(Shape), c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_void_p, c_int32,
                                 P(Batch), c_void_p, c_size_t, c_void_p]),
    "duet_attn_mixed_batch": (c_int32, [c_void_p, P(Shape), c_void_p, c_void_p, c_void_p, c_int64, c_void_p, c_int32,
                                        P(Batch), CuSplit, c_void_p, c_size_t, c_void_p, c_void_p]),
    "duet_attn_mixed_batch_noalloc": (c_int32, [c_void_p, P(Shape), c_void_p, c_void_p, c_void_p, c_int64, c_void_p,
                                                c_int32, P(Batch), CuSplit, c_void_p, c_void_p]),
    "duet_attn_iteration": (c_int32, [c_void_p, P(Shape), P(c_void_p), P(c_void_p), P(c_void_p), c_int64, c_void_p,
                                      c_int32, P(Batch), CuSplit, c_void_p, c_size_t, P(c_void_p), c_void_p]),
    "duet_lookahead_workspace_bytes": (c_int32, [P(Shape), P(Batch), c_int32, P(c_size_t)]),
    "duet_attn_lookahead": (c_int32, [c_void_p, P(Shape), P(c_void_p), P(c_void_p), P(c_void_p), P(c_void_p),
                                      P(c_void_p), P(c_void_p), c_int64, c_void_p, c_int32, P(Batch), CuSplit,
                                      c_void_p, c_size_t, P(c_void_p), P(c_void_p), c_void_p]),
    "duet_set_decode_graphs": (c_int32, [c_void_p, c_int32]),
    "duet_decode_graph_stats": (c_int32, [c_void_p, P(c_int64), P(c_int64), P(c_int64)]),
    "duet_check_device_error": (c_int32, [c_void_p, c_void_p, c_void_p]),
    "duet_gather_kv": (c_int32, [c_void_p, P(Shape), c_int32, c_void_p, c_int64, c_void_p, c_int32, c_int32, c_int32,
                                 c_void_p, c_void_p]),
    "duet_set_profiling": (c_int32, [c_void_p, c_int32]),
    "duet_last_kernel_times": (c_int32, [c_void_p, P(KernelTimes)]),
    "duet_probe_read_bw": (c_int32, [c_void_p, c_int32, c_void_p, c_size_t, c_int32, P(c_double)]),
    "duet_probe_mfma": (c_int32, [c_void_p, c_int32, c_int32, P(c_double)]),
    "duet_probe_placement": (c_int32, [c_void_p, c_int32, c_int32, c_int32, c_void_p]),
    "duet_calibrate": (c_int32, [c_void_p, c_void_p, c_void_p, c_size_t]),
    "duet_last_error": (ctypes.c_char_p, []),
}

_lock = threading.Lock()
_lib = None


def lib():
    """The loaded library.  Builds it first if no built library is present; raises if it cannot
    be built or loaded -- there is no fallback path."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                from . import build as _build
                _build.build()
            handle = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in _SIGS.items():
                fn = getattr(handle, name)
                fn.restype = res
                fn.argtypes = args
            _lib = handle
        return _lib


class DuetError(RuntimeError):
    def __init__(self, code: int, fn: str, msg: str):
        super().__init__(f"{fn} failed: {ERRORS.get(code, code)}: {msg}")
        self.code = code


def check(code: int, fn: str):
    if code != OK:
        raise DuetError(code, fn, lib().duet_last_error().decode())
    return code
