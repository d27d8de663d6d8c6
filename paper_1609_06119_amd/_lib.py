"""ctypes declarations of libfbdt's C ABI (include/fbdt.h).

The library is loaded from this package directory.  There is no fallback:
if the HIP library is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfbdt.so")

FBDT_OK = 0
STATUS = {
    -1: "FBDT_E_INVAL",
    -2: "FBDT_E_LABEL",
    -3: "FBDT_E_NAN",
    -4: "FBDT_E_WEIGHT",
    -5: "FBDT_E_SHAPE",
    -6: "FBDT_E_DEVICE",
}
KERNEL_KINDS = {"histogram": 0, "best_cuts": 1, "tree_prep": 2, "leaf": 3, "apply": 4,
                "encode": 5, "route": 6, "reference": 7}

EXPORTED = (
    "fbdt_bin", "fbdt_bin_transform", "fbdt_fit", "fbdt_apply", "fbdt_apply_float",
    "fbdt_model_export", "fbdt_model_import", "fbdt_model_set_boundaries", "fbdt_model_free",
    "fbdt_last_error", "fbdt_tree_weights", "fbdt_feature_importance", "fbdt_event_importance",
    "fbdt_histogram", "fbdt_best_cuts", "fbdt_best_cuts_noalloc", "fbdt_route",
    "fbdt_leaf_values",
    "fbdt_timing_enable", "fbdt_timing_read", "fbdt_set_option", "fbdt_hist_timeline",
    "fbdt_reference_pass",
)


class FitParams(C.Structure):
    _fields_ = [("depth", C.c_int32), ("n_trees", C.c_int32), ("shrinkage", C.c_double),
                ("subsample", C.c_double), ("seed", C.c_uint64)]


class ModelView(C.Structure):
    _fields_ = [("n_trees", C.c_int32), ("depth", C.c_int32), ("n_features", C.c_int32),
                ("n_bins", C.c_int32), ("f0", C.c_double),
                ("cut_feature", C.POINTER(C.c_uint8)), ("cut_bin", C.POINTER(C.c_uint8)),
                ("gain", C.POINTER(C.c_double)), ("leaf", C.POINTER(C.c_double)),
                ("boundaries", C.POINTER(C.c_float)), ("inner", C.POINTER(C.c_double))]


class FbdtError(RuntimeError):
    """A libfbdt call returned an error status."""

    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn}: {STATUS.get(code, code)}: {msg}")
        self.code = code
        self.status = STATUS.get(code, str(code))


_lib = None

P = C.c_void_p
I64 = C.c_int64
I32 = C.c_int32


def _declare(lib):
    sig = {
        "fbdt_bin": (C.c_int, [P, I64, I32, I64, I32, P, P, I64, P]),
        "fbdt_bin_transform": (C.c_int, [P, I64, I32, I64, I32, P, P, I64, P]),
        "fbdt_fit": (C.c_int, [P, I64, I32, I64, I32, P, P, C.POINTER(FitParams),
                               C.POINTER(P), P, P]),
        "fbdt_apply": (C.c_int, [P, P, I64, I32, I64, P, P, P]),
        "fbdt_apply_float": (C.c_int, [P, P, I64, I32, I64, P, P, P]),
        "fbdt_model_set_boundaries": (C.c_int, [P, P]),
        "fbdt_feature_importance": (C.c_int, [P, P]),
        "fbdt_event_importance": (C.c_int, [P, P, I64, I32, I64, P, I64, P]),
        "fbdt_model_export": (C.c_int, [P, C.POINTER(ModelView)]),
        "fbdt_model_import": (C.c_int, [C.POINTER(ModelView), C.POINTER(P)]),
        "fbdt_model_free": (None, [P]),
        "fbdt_last_error": (C.c_char_p, []),
        "fbdt_tree_weights": (C.c_int, [P, P, P, I64, C.c_uint64, I32, C.c_double, P, P]),
        "fbdt_histogram": (C.c_int, [P, I64, I32, I64, I32, P, P, I32, P, P]),
        "fbdt_best_cuts": (C.c_int, [P, I32, I32, I32, P, P, P, P]),
        "fbdt_best_cuts_noalloc": (C.c_int, [P, I32, I32, I32, P, P, P, P]),
        "fbdt_route": (C.c_int, [P, I64, I32, I64, P, P, P, I32, P]),
        "fbdt_leaf_values": (C.c_int, [P, P, P, P, I64, I32, C.c_uint64, I32, C.c_double,
                                       C.c_double, P, P]),
        "fbdt_timing_enable": (C.c_int, [I32]),
        "fbdt_timing_read": (C.c_int, [I32, C.POINTER(I64), C.POINTER(C.c_double),
                                       C.POINTER(C.c_double)]),
        "fbdt_set_option": (C.c_int, [C.c_char_p, I64]),
        "fbdt_hist_timeline": (C.c_int, [C.POINTER(I64), C.POINTER(I32),
                                         C.POINTER(C.POINTER(I32)),
                                         C.POINTER(C.POINTER(C.c_uint64)), C.POINTER(I64)]),
        "fbdt_reference_pass": (C.c_int, [I32, P, I64, I32, I64, I32, I32, P, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build the HIP library first "
                "(python -c 'import __graft_entry__ as g; g.build()')")
        handle = C.CDLL(LIB_PATH)
        _declare(handle)
        _lib = handle
    return _lib


def check(fn: str, rc: int):
    if rc != FBDT_OK:
        raise FbdtError(fn, rc, lib().fbdt_last_error().decode())
