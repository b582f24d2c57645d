"""ctypes declarations of libslorr.so (the C ABI in include/slorr.h).

Loading fails loudly when the library has not been built: there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libslorr.so")
# another build of the same library (e.g. the sanitizer build of the CPU tests)
if os.environ.get("SLORR_LIB"):
    LIB_PATH = os.environ["SLORR_LIB"]

# status codes
OK = 0
ERR_INVALID_ARGUMENT = 1
ERR_UNSUPPORTED = 2
ERR_PLAN_MISMATCH = 3
ERR_WORKSPACE = 4
ERR_HIP = 5
ERR_INTERNAL = 6

# enums and flags
HOYER, NUCLEAR = 0, 1
F32, BF16 = 0, 1
ACCUMULATE = 0x1
VALUES_ONLY = 0x2
NO_GRAPH = 0x4
AUX = 0x8
DEFER_GRAD = 0x10

OPS = ("sumsq", "norm", "prep", "gram", "poly", "update", "last", "finalize", "grad", "setsum", "gram_reduce")

EXPORTED = ("slorr_default_options", "slorr_pe_coefficients", "slorr_plan", "slorr_cache_config",
            "slorr_cache_clear",
            "slorr_plan_set_workspace", "slorr_reg_fwd_bwd", "slorr_reg_grad", "slorr_decoupled_apply",
            "slorr_reg_fwd_bwd_profiled", "slorr_reg_fwd_bwd_noalloc",
            "slorr_plan_destroy", "slorr_plan_get_info", "slorr_plan_get_launches", "slorr_status_string",
            "slorr_last_error")


class Shape(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int32), ("cols", ctypes.c_int32)]


class Options(ctypes.Structure):
    _fields_ = [("iters", ctypes.c_int32), ("degree", ctypes.c_int32), ("ell", ctypes.c_double),
                ("coeffs", ctypes.POINTER(ctypes.c_double)), ("eps", ctypes.c_float),
                ("flags", ctypes.c_uint32), ("grad_dtype", ctypes.c_int), ("safety", ctypes.c_double)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("groups", ctypes.c_int32), ("iters", ctypes.c_int32),
                ("launches", ctypes.c_int32), ("gemm_tiles", ctypes.c_int64),
                ("paper_flops", ctypes.c_double), ("mfma_flops", ctypes.c_double),
                ("weight_bytes", ctypes.c_double), ("workspace_bytes", ctypes.c_size_t)]


class SlorrError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        self.status = status
        super().__init__(f"{func}: {_status_name(status)}: {detail}")


_lib = None


def _status_name(s: int) -> str:
    return lib().slorr_status_string(s).decode()


def lib() -> ctypes.CDLL:
    """The loaded library (loaded once)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing; build it with "
                              "`python -m paper_2607_08754_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.slorr_default_options.argtypes = [ctypes.POINTER(Options)]
        L.slorr_default_options.restype = None
        L.slorr_pe_coefficients.argtypes = [ctypes.c_double, i32, i32, ctypes.POINTER(ctypes.c_double)]
        L.slorr_pe_coefficients.restype = ctypes.c_int
        L.slorr_plan.argtypes = [ctypes.POINTER(vp), i32, ctypes.POINTER(Shape), ctypes.c_int,
                                 ctypes.c_int, ctypes.POINTER(Options), ctypes.POINTER(sz)]
        L.slorr_plan.restype = ctypes.c_int
        L.slorr_cache_config.argtypes = [ctypes.c_int, ctypes.POINTER(Options)]
        L.slorr_cache_config.restype = None
        L.slorr_cache_clear.argtypes = []
        L.slorr_cache_clear.restype = ctypes.c_int
        L.slorr_plan_set_workspace.argtypes = [vp, vp, sz]
        L.slorr_plan_set_workspace.restype = ctypes.c_int
        L.slorr_reg_fwd_bwd.argtypes = [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(Shape), ctypes.c_int,
                                        i32, vp, ctypes.POINTER(vp), ctypes.c_float, vp]
        L.slorr_reg_fwd_bwd.restype = ctypes.c_int
        L.slorr_reg_grad.argtypes = [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(Shape), ctypes.c_int,
                                     i32, ctypes.POINTER(vp), vp, ctypes.c_float, vp]
        L.slorr_reg_grad.restype = ctypes.c_int
        L.slorr_decoupled_apply.argtypes = [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(Shape),
                                            ctypes.POINTER(vp), vp, ctypes.c_float, vp]
        L.slorr_decoupled_apply.restype = ctypes.c_int
        L.slorr_reg_fwd_bwd_profiled.argtypes = [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(Shape),
                                                 ctypes.c_int, i32, vp, ctypes.POINTER(vp), ctypes.c_float, vp,
                                                 ctypes.POINTER(ctypes.c_float), ctypes.POINTER(i32)]
        L.slorr_reg_fwd_bwd_profiled.restype = ctypes.c_int
        L.slorr_reg_fwd_bwd_noalloc.argtypes = [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(Shape), ctypes.c_int,
                                                i32, vp, ctypes.POINTER(vp), ctypes.c_float, vp]
        L.slorr_reg_fwd_bwd_noalloc.restype = ctypes.c_int
        L.slorr_plan_destroy.argtypes = [vp]
        L.slorr_plan_destroy.restype = ctypes.c_int
        L.slorr_plan_get_info.argtypes = [vp, ctypes.POINTER(PlanInfo)]
        L.slorr_plan_get_info.restype = ctypes.c_int
        L.slorr_plan_get_launches.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(i32)]
        L.slorr_plan_get_launches.restype = ctypes.c_int
        L.slorr_status_string.argtypes = [ctypes.c_int]
        L.slorr_status_string.restype = ctypes.c_char_p
        L.slorr_last_error.argtypes = []
        L.slorr_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def check(status: int, func: str) -> None:
    if status != OK:
        raise SlorrError(status, func, lib().slorr_last_error().decode())
