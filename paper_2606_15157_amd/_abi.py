"""ctypes declarations of librkv.so (the C ABI in include/rkv.h)."""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librkv.so")

RKV_OK = 0
STATUS_NAMES = {0: "RKV_OK", 1: "RKV_ERR_INVALID_ARG", 2: "RKV_ERR_SHAPE", 3: "RKV_ERR_PLAN",
                4: "RKV_ERR_UNSUPPORTED", 5: "RKV_ERR_WORKSPACE", 6: "RKV_ERR_HIP", 7: "RKV_ERR_DEVICE"}

FULL, STREAMING, SNAPKV, H2O, TOVA, H2O_FULL = 0, 1, 2, 3, 4, 5
PHASE_PREFILL, PHASE_DECODE = 0, 1
SCOPE_PREFILL, SCOPE_DECODE, SCOPE_BOTH = 0, 1, 2
T_IDENTITY, T_PPL_CAP = 0, 1
STATUS_TIMEOUT, STATUS_INVALID, STATUS_REPAIRED = 1, 2, 4

EXPORTED = [
    "rkv_allocate_budgets", "rkv_plan_create", "rkv_plan_destroy", "rkv_plan_num_layers",
    "rkv_plan_serialize", "rkv_plan_deserialize", "rkv_rule_phases", "rkv_plan_from_route",
    "rkv_plan_retained_counts", "rkv_prefill_workspace_size", "rkv_prefill_evict", "rkv_prefill_evict_noalloc", "rkv_prefill_check",
    "rkv_decode_step", "rkv_decode_init_from_prefill", "rkv_entropy_workspace_size", "rkv_entropy_profile", "rkv_profile_enable", "rkv_profile_read", "rkv_last_error",
    "rkv_version",
]


class Layer(C.Structure):
    _fields_ = [("rule_prefill", C.c_int32), ("budget_prefill", C.c_int32),
                ("rule_decode", C.c_int32), ("budget_decode", C.c_int32)]


class RouteLayer(C.Structure):
    _fields_ = [("rule", C.c_int32), ("scope", C.c_int32), ("budget", C.c_int32)]


class Params(C.Structure):
    _fields_ = [("window", C.c_int32), ("pool_kernel", C.c_int32), ("n_sink", C.c_int32),
                ("recent_num", C.c_int32), ("recent_den", C.c_int32)]


class Shape(C.Structure):
    _fields_ = [("batch", C.c_int32), ("seq_len", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32)]


class PrefillIO(C.Structure):
    _fields_ = [("q_win", C.POINTER(C.c_void_p)), ("k", C.POINTER(C.c_void_p)), ("v", C.POINTER(C.c_void_p)),
                ("k_out", C.POINTER(C.c_void_p)), ("v_out", C.POINTER(C.c_void_p)),
                ("idx_out", C.POINTER(C.c_void_p)), ("score_out", C.POINTER(C.c_void_p)),
                ("acc_out", C.POINTER(C.c_void_p))]


class DecodeState(C.Structure):
    _fields_ = [("k_cache", C.POINTER(C.c_void_p)), ("v_cache", C.POINTER(C.c_void_p)),
                ("pos", C.POINTER(C.c_void_p)), ("acc", C.POINTER(C.c_void_p))]


class DecodeInput(C.Structure):
    _fields_ = [("q", C.POINTER(C.c_void_p)), ("k", C.POINTER(C.c_void_p)), ("v", C.POINTER(C.c_void_p)),
                ("victim_out", C.POINTER(C.c_void_p))]


_lib = None


def lib():
    """Load librkv.so once; fail loudly when it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_15157_amd.build`")
        L = C.CDLL(LIB_PATH)
        L.rkv_allocate_budgets.argtypes = [C.POINTER(C.c_double), C.c_int32, C.c_int32, C.c_int64, C.c_int32,
                                           C.POINTER(C.c_int32)]
        L.rkv_plan_create.argtypes = [C.POINTER(Layer), C.c_int32, C.POINTER(Params), C.POINTER(C.c_void_p)]
        L.rkv_rule_phases.argtypes = [C.c_int32, C.POINTER(C.c_int32)]
        L.rkv_plan_from_route.argtypes = [C.POINTER(RouteLayer), C.c_int32, C.POINTER(Params), C.POINTER(C.c_void_p)]
        L.rkv_plan_destroy.argtypes = [C.c_void_p]
        L.rkv_plan_destroy.restype = None
        L.rkv_plan_num_layers.argtypes = [C.c_void_p, C.POINTER(C.c_int32)]
        L.rkv_plan_serialize.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.POINTER(C.c_size_t)]
        L.rkv_plan_deserialize.argtypes = [C.c_void_p, C.c_size_t, C.POINTER(C.c_void_p)]
        L.rkv_plan_retained_counts.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.POINTER(C.c_int32)]
        L.rkv_prefill_workspace_size.argtypes = [C.c_void_p, C.POINTER(Shape), C.POINTER(C.c_size_t)]
        L.rkv_prefill_evict.argtypes = [C.c_void_p, C.POINTER(Shape), C.POINTER(PrefillIO), C.c_void_p, C.c_size_t,
                                        C.c_void_p]
        L.rkv_prefill_evict_noalloc.argtypes = [C.c_void_p, C.POINTER(Shape), C.POINTER(PrefillIO), C.c_void_p,
                                                C.c_void_p]
        L.rkv_prefill_check.argtypes = [C.c_void_p, C.c_size_t, C.POINTER(C.c_int32)]
        L.rkv_decode_step.argtypes = [C.c_void_p, C.POINTER(Shape), C.POINTER(DecodeState), C.POINTER(DecodeInput),
                                      C.c_int32, C.c_void_p]
        L.rkv_decode_init_from_prefill.argtypes = [C.c_void_p, C.POINTER(Shape), C.POINTER(PrefillIO),
                                                   C.POINTER(DecodeState), C.c_void_p]
        L.rkv_entropy_workspace_size.argtypes = [C.POINTER(Shape), C.c_int32, C.c_int32, C.POINTER(C.c_size_t)]
        L.rkv_entropy_profile.argtypes = [C.POINTER(Shape), C.c_int32, C.c_int32, C.POINTER(C.c_void_p),
                                          C.POINTER(C.c_void_p), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                          C.c_size_t, C.c_void_p]
        L.rkv_profile_enable.argtypes = [C.c_int32]
        L.rkv_profile_read.argtypes = [C.POINTER(C.c_int32), C.POINTER(C.c_double)]
        L.rkv_last_error.restype = C.c_char_p
        L.rkv_last_error.argtypes = []
        L.rkv_version.argtypes = []
        for name in ("rkv_allocate_budgets", "rkv_plan_create", "rkv_plan_num_layers", "rkv_plan_retained_counts",
                     "rkv_plan_serialize", "rkv_plan_deserialize",
                     "rkv_prefill_workspace_size", "rkv_prefill_evict", "rkv_prefill_check", "rkv_decode_step",
                     "rkv_rule_phases", "rkv_plan_from_route", "rkv_decode_init_from_prefill", "rkv_prefill_evict_noalloc",
                     "rkv_entropy_workspace_size", "rkv_entropy_profile",
                     "rkv_profile_enable", "rkv_profile_read", "rkv_version"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


class RkvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def check(status: int):
    if status != RKV_OK:
        raise RkvError(status, lib().rkv_last_error().decode(errors="replace"))


def ptr_array(ptrs):
    arr = (C.c_void_p * len(ptrs))()
    for i, p in enumerate(ptrs):
        arr[i] = p if p else None
    return arr
