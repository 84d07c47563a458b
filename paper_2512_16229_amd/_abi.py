"""ctypes declarations of the liblopa C ABI (include/lopa.h) and the loader.

Kept free of PyTorch so that torch-less harnesses (the HBM-counter run of
bench.py) can drive the library with plain device pointers."""
from __future__ import annotations

import ctypes as C
import os


_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblopa.so")

LOPA_OK, LOPA_EINVAL, LOPA_ESHAPE, LOPA_ECAPACITY, LOPA_EHIP, LOPA_ENOMEM = 0, -1, -2, -3, -4, -5
MAX_BLOCK, MAX_ROWS, WINDOW_MAX_BLOCKS = 256, 2048, 16


class LopaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"liblopa status {status}: {msg}")
        self.status = status


class lopa_model_cfg(C.Structure):
    _fields_ = [("layers", C.c_int32), ("hidden", C.c_int32), ("heads", C.c_int32),
                ("kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
                ("vocab", C.c_int32), ("mask_id", C.c_int32), ("rms_eps", C.c_float),
                ("rope_theta", C.c_float), ("qkv_bias", C.c_int32)]


class lopa_layer_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("wq", "wk", "wv", "bq", "bk", "bv", "wo", "w_gate",
                                           "w_up", "w_down", "ln1", "ln2")]


class lopa_window(C.Structure):
    """The device-resident window state of include/lopa.h (field order)."""
    _fields_ = [(n, C.c_int32) for n in ("blocks", "eligible", "prefix_len", "need_initial", "done",
                                          "added", "committed", "last_commit", "last_commit_at",
                                          "error", "L", "w_max", "n_blocks", "mask_id", "add_min",
                                          "act_min")] + [("active", C.c_int32 * 16)]


class lopa_weight_ptrs(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("layers", C.POINTER(lopa_layer_weights)),
                ("final_norm", C.c_void_p), ("lm_head", C.c_void_p)]


EXPORTS = ["lopa_model_create", "lopa_model_create_ex", "lopa_model_destroy", "lopa_kv_create", "lopa_kv_destroy",
           "lopa_strerror", "lopa_last_error", "lopa_build_branches", "lopa_build_branches_window",
           "lopa_verify_forward",
           "lopa_branch_confidence_select", "lopa_branch_confidence_select_metric", "lopa_commit_kv",
           "lopa_commit_kv_rows", "lopa_kv_read", "lopa_kv_write",
           "lopa_kv_read_staging", "lopa_debug_hidden",
           "lopa_kv_set_block_causal", "lopa_kv_profile",
           "lopa_kv_profile_read", "lopa_verify_forward_noalloc", "lopa_window_init",
           "lopa_window_update", "lopa_window_commit"]
METRIC_MEAN, METRIC_WINDOW_MIN, METRIC_LOWEST_SEGMENT = 0, 1, 2
PRECISIONS = {"bf16": 0, "fp8_mlp": 1, "fp8": 2}
PROF_KINDS = ["qkv", "attn", "oproj", "gateup", "down", "lmhead", "norm", "merge"]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2512_16229_amd/build.py`")
    lib = C.CDLL(LIB_PATH)
    P, I32, F32 = C.c_void_p, C.c_int32, C.c_float
    sig = {
        "lopa_model_create": (C.c_int, [C.POINTER(lopa_model_cfg), C.POINTER(lopa_weight_ptrs), P,
                                        C.POINTER(C.c_void_p)]),
        "lopa_model_create_ex": (C.c_int, [C.POINTER(lopa_model_cfg), C.POINTER(lopa_weight_ptrs), I32, P,
                                        C.POINTER(C.c_void_p)]),
        "lopa_model_destroy": (None, [P]),
        "lopa_kv_create": (C.c_int, [P, I32, I32, I32, C.POINTER(C.c_void_p)]),
        "lopa_kv_destroy": (None, [P]),
        "lopa_strerror": (C.c_char_p, [C.c_int]),
        "lopa_last_error": (C.c_char_p, []),
        "lopa_build_branches": (C.c_int, [P, P, P, I32, I32, F32, I32, P, P, P, P, P]),
        "lopa_build_branches_window": (C.c_int, [P, P, P, I32, I32, I32, F32, I32, P, P, P, P, P]),
        "lopa_verify_forward": (C.c_int, [P, P, I32, P, I32, I32, P, P, P]),
        "lopa_branch_confidence_select": (C.c_int, [P, P, P, P, I32, I32, I32, P, P, P, P, P, P, P]),
        "lopa_branch_confidence_select_metric": (C.c_int, [P, P, P, P, I32, I32, I32, I32, I32, F32,
                                                           P, P, P, P, P, P, P]),
        "lopa_commit_kv": (C.c_int, [P, P, I32, I32, P, P]),
        "lopa_commit_kv_rows": (C.c_int, [P, P, I32, I32, I32, P, P]),
        "lopa_kv_read": (C.c_int, [P, I32, I32, I32, P, P, P]),
        "lopa_kv_write": (C.c_int, [P, I32, I32, I32, P, P, P]),
        "lopa_kv_read_staging": (C.c_int, [P, I32, I32, P, P, P]),
        "lopa_debug_hidden": (C.c_int, [P, P, I32, P, I32, I32, I32, P, P]),
        "lopa_kv_set_block_causal": (C.c_int, [P, I32]),
        "lopa_kv_profile": (C.c_int, [P, I32]),
        "lopa_kv_profile_read": (C.c_int, [P, C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
        "lopa_verify_forward_noalloc": (C.c_int, [P, P, I32, P, I32, I32, P, P, P]),
        "lopa_window_init": (C.c_int, [P, P, P, P, I32, I32, I32, I32, I32, C.c_double, C.c_double, P]),
        "lopa_window_update": (C.c_int, [P, P, P, P, P, P]),
        "lopa_window_commit": (C.c_int, [P, P, P, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    return lib


lib = _load()


