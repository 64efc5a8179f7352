"""ctypes declarations of the libaep C ABI (include/aep.h).

Argument marshalling only: every step of the path runs in the HIP library.
torch is imported first so that its HIP runtime is the one libaep binds to
(both carry the soname libamdhip64.so.7).  There is no fallback: if the
library is not built, loading fails loudly.
"""

from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (loads the HIP runtime libaep links against)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libaep.so")

AEP_OK, AEP_ERR_INVALID_ARG, AEP_ERR_CAPACITY, AEP_ERR_EMPTY, AEP_ERR_STATE, AEP_ERR_DEVICE, \
    AEP_ERR_UNSUPPORTED = range(7)
AEP_F32, AEP_BF16, AEP_FP8_E4M3 = range(3)
AEP_POLICY_MTFS, AEP_POLICY_FLFS, AEP_POLICY_DEFRAG = range(3)
AEP_STATIC_WORKSPACE_BYTES = 96 << 20   # include/aep.h

STATUS_NAMES = {0: "AEP_OK", 1: "AEP_ERR_INVALID_ARG", 2: "AEP_ERR_CAPACITY", 3: "AEP_ERR_EMPTY",
                4: "AEP_ERR_STATE", 5: "AEP_ERR_DEVICE", 6: "AEP_ERR_UNSUPPORTED"}


class AEPError(RuntimeError):
    def __init__(self, status: int, call: str):
        self.status = status
        super().__init__(f"{call} -> {STATUS_NAMES.get(status, status)}")


class Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_experts", ctypes.c_int32), ("n_shared", ctypes.c_int32),
                ("d_model", ctypes.c_int32), ("d_ffn", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("renorm", ctypes.c_int32), ("act_dtype", ctypes.c_int32), ("w_dtype", ctypes.c_int32),
                ("max_tokens_per_layer", ctypes.c_int32), ("token_pool", ctypes.c_int32)]


class Batch(ctypes.Structure):
    _fields_ = [("layer", ctypes.c_int32), ("n_tokens", ctypes.c_int32), ("n_routed", ctypes.c_int64),
                ("n_rows", ctypes.c_int64), ("epoch", ctypes.c_uint64), ("x_perm", ctypes.c_void_p),
                ("counts", ctypes.c_void_p), ("offsets", ctypes.c_void_p), ("row_token", ctypes.c_void_p),
                ("row_weight", ctypes.c_void_p), ("token_pos", ctypes.c_void_p),
                ("token_weight", ctypes.c_void_p)]


class SimConfig(ctypes.Structure):
    _fields_ = [("n_blocks", ctypes.c_int32), ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("n_frag", ctypes.c_int32), ("granularity", ctypes.c_int32), ("policy", ctypes.c_int32),
                ("delta", ctypes.c_double), ("lookahead", ctypes.c_int32), ("n_requests", ctypes.c_int32),
                ("attn_us", ctypes.c_int64), ("jitter_us", ctypes.c_int64), ("cost_fixed_us", ctypes.c_int64),
                ("cost_row_ns", ctypes.c_int64), ("horizon_us", ctypes.c_int64), ("seed", ctypes.c_uint64),
                ("arrival_us", ctypes.c_void_p), ("out_len", ctypes.c_void_p), ("expert_cdf", ctypes.c_void_p)]


class SimTrace(ctypes.Structure):
    _fields_ = [("capacity", ctypes.c_int64), ("t_start", ctypes.c_void_p), ("block", ctypes.c_void_p),
                ("expert", ctypes.c_void_p), ("rows", ctypes.c_void_p), ("queued_after", ctypes.c_void_p),
                ("blocks_busy_after", ctypes.c_void_p), ("block_rows_after", ctypes.c_void_p),
                ("done_us", ctypes.c_void_p)]


class SimSummary(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("steps", "rows", "busy_us", "end_us", "token_passes",
                                              "requests_done", "rows_queued_at_end", "recorded")]


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SIG = {
    "aep_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "aep_create": (ctypes.c_int, [ctypes.POINTER(Config), ctypes.POINTER(_P)]),
    "aep_destroy": (ctypes.c_int, [_P]),
    "aep_workspace_size": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_size_t)]),
    "aep_bind_workspace": (ctypes.c_int, [_P, _P, ctypes.c_size_t, _P]),
    "aep_bind_static_workspace": (ctypes.c_int, [_P, _P]),
    "aep_set_expert_weights": (ctypes.c_int, [_P, _I32, _I32, _P, _P, _P, _P, _P, _P]),
    "aep_route_enqueue": (ctypes.c_int, [_P, _I32, _P, _P, _I32, _P, _P, _P]),
    "aep_enqueue_rows": (ctypes.c_int, [_P, _I32, _I32, _P, _P, _P, _P, _I32, _I32, _P]),
    "aep_enqueue_rows_grouped": (ctypes.c_int, [_P, _I32, _P, _P, _P, _P, _P, _I32, _P]),
    "aep_queue_depth": (ctypes.c_int, [_P, _I32, ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "aep_expert_counts": (ctypes.c_int, [_P, _I32, _P, _P]),
    "aep_pick_layer": (ctypes.c_int, [_P, _I32, ctypes.c_double, _I32, ctypes.POINTER(_I32)]),
    "aep_rebatch": (ctypes.c_int, [_P, _I32, ctypes.POINTER(Batch), _P]),
    "aep_expert_ffn": (ctypes.c_int, [_P, ctypes.POINTER(Batch), _P, _P]),
    "aep_expert_gate_up": (ctypes.c_int, [_P, ctypes.POINTER(Batch), _P]),
    "aep_expert_down": (ctypes.c_int, [_P, ctypes.POINTER(Batch), _P, _P]),
    "aep_combine": (ctypes.c_int, [_P, ctypes.POINTER(Batch), _P, _P, _P]),
    "aep_release_batch": (ctypes.c_int, [_P, ctypes.POINTER(Batch)]),
    "aep_sync": (ctypes.c_int, [_P, _P]),
    "aep_set_clock_probe": (ctypes.c_int, [_P, _P, _I32]),
    "aep_fp8_e4m3_to_bf16": (ctypes.c_int, [_P, _P, _I64, _P]),
    "aep_route_enqueue_ids": (ctypes.c_int, [_P, _I32, _P, _P, _I32, _P, _P, _P, _P]),
    "aep_rebatch_expert": (ctypes.c_int, [_P, _I32, _I32, ctypes.POINTER(Batch), _P]),
    "aep_pool_accumulate": (ctypes.c_int, [_P, ctypes.POINTER(Batch), _P, _P]),
    "aep_pool_release": (ctypes.c_int, [_P, _I32, _P, _P, _P]),
    "aep_sched_pick": (ctypes.c_int, [_P, _I32, _I32, _I32, ctypes.c_double, _I32, ctypes.POINTER(_I32),
                                      ctypes.POINTER(_I32)]),
    "aep_sim_run": (ctypes.c_int, [ctypes.POINTER(SimConfig), ctypes.POINTER(SimTrace),
                                   ctypes.POINTER(SimSummary)]),
}

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2505_08944_amd.build`")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIG.items():
            fn = getattr(l, name)
            fn.restype = res
            fn.argtypes = args
        _lib = l
    return _lib


def check(status: int, call: str) -> None:
    if status != AEP_OK:
        raise AEPError(status, call)
