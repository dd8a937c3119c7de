"""ctypes binding of libmuon_mi355x.so (the C ABI declared in include/muon.h).

Argument marshalling only: every step of the Muon update runs in the HIP
library.  ``load()`` raises if the library has not been built -- there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os
import threading

LIB_NAME = "libmuon_mi355x.so"
LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), LIB_NAME)

# muon_status
MUON_OK = 0
MUON_ERR_INVALID_ARG = 1
MUON_ERR_UNSUPPORTED = 2
MUON_ERR_OUT_OF_MEMORY = 3
MUON_ERR_WORKSPACE_TOO_SMALL = 4
MUON_ERR_DEVICE = 5

# muon_dtype
MUON_F32 = 0
MUON_BF16 = 1

# muon_ns_precision
MUON_NS_BF16 = 0
MUON_NS_FP32 = 1
MUON_NS_FP16 = 2

MUON_PLAN_HOST_ONLY = 0x1
MUON_PLAN_CHECK_BUFFERS = 0x2
MUON_STATIC_WORKSPACE_BYTES = 64 << 20


class muon_matrix_desc(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("param_dtype", ctypes.c_int32), ("grad_dtype", ctypes.c_int32),
                ("momentum_dtype", ctypes.c_int32), ("tile_hint", ctypes.c_int32)]


class muon_plan_opts(ctypes.Structure):
    _fields_ = [("precision", ctypes.c_int32), ("max_ns_steps", ctypes.c_int32),
                ("a", ctypes.c_float), ("b", ctypes.c_float), ("c", ctypes.c_float),
                ("eps", ctypes.c_float), ("small_m_threshold", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("wave_bytes", ctypes.c_int64),
                ("gram_min_aspect", ctypes.c_float), ("gram_restart", ctypes.c_int32),
                ("abc_per_step", ctypes.POINTER(ctypes.c_float))]


class muon_plan_info(ctypes.Structure):
    _fields_ = [("n_matrices", ctypes.c_int32), ("n_waves", ctypes.c_int32),
                ("n_buckets", ctypes.c_int32), ("device", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_int64), ("launches_per_step", ctypes.c_int64),
                ("ns_flops_per_ns_step", ctypes.c_double),
                ("padded_flops_per_ns_step", ctypes.c_double),
                ("n_gram", ctypes.c_int32), ("gram_restart", ctypes.c_int32)]


class muon_matrix_info(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int64), ("n", ctypes.c_int64),
                ("m_pad", ctypes.c_int64), ("n_pad", ctypes.c_int64),
                ("transposed", ctypes.c_int32), ("kernel_class", ctypes.c_int32),
                ("tile", ctypes.c_int32), ("fp32_ns", ctypes.c_int32),
                ("wave", ctypes.c_int32), ("bucket", ctypes.c_int32),
                ("gram_space", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class muon_kernel_stat(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("kernel_class", ctypes.c_int32),
                ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double),
                ("algo_flops", ctypes.c_double), ("algo_bytes", ctypes.c_double)]


KERNEL_KINDS = ("momentum", "finalize", "gram", "poly", "bx", "apply", "symm")
KERNEL_CLASSES = ("bf16_t256", "bf16_t128", "bf16_t64", "f32_t128", "f32_t64", "f16_t256", "f16_t128", "f16_t64")

_VP = ctypes.c_void_p
_PP = ctypes.POINTER(ctypes.c_void_p)
_STEP_ARGS = [_VP, _PP, _PP, _PP, ctypes.c_float, ctypes.c_float, ctypes.c_float,
              ctypes.c_int32, ctypes.c_int32, _VP, ctypes.c_size_t, _VP]

# name -> (restype, argtypes); every function declared in include/muon.h
SIGNATURES = {
    "muon_plan_opts_default": (ctypes.c_int, [ctypes.POINTER(muon_plan_opts)]),
    "muon_plan_create": (ctypes.c_int, [ctypes.POINTER(muon_matrix_desc), ctypes.c_int32,
                                        ctypes.POINTER(muon_plan_opts), ctypes.POINTER(_VP)]),
    "muon_plan_destroy": (ctypes.c_int, [_VP]),
    "muon_plan_workspace_bytes": (ctypes.c_int, [_VP, ctypes.POINTER(ctypes.c_size_t)]),
    "muon_plan_get_info": (ctypes.c_int, [_VP, ctypes.POINTER(muon_plan_info)]),
    "muon_plan_ns_flops": (ctypes.c_int, [_VP, ctypes.c_int32, ctypes.POINTER(ctypes.c_double)]),
    "muon_plan_matrix_info": (ctypes.c_int, [_VP, ctypes.c_int32, ctypes.POINTER(muon_matrix_info)]),
    "muon_step": (ctypes.c_int, _STEP_ARGS),
    "muon_step_debug": (ctypes.c_int, _STEP_ARGS + [_PP]),
    "muon_step_static": (ctypes.c_int, [_VP, _PP, _PP, _PP, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                        ctypes.c_int32, ctypes.c_int32, _VP]),
    "muon_check_buffers": (ctypes.c_int, [_VP, _PP, _PP, _PP, _VP, ctypes.c_size_t, _PP]),
    "muon_plan_set_timing": (ctypes.c_int, [_VP, ctypes.c_int32]),
    "muon_plan_timing_read": (ctypes.c_int, [_VP, ctypes.POINTER(muon_kernel_stat), ctypes.c_int32,
                                             ctypes.POINTER(ctypes.c_int32), ctypes.c_int32]),
    "muon_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "muon_last_error": (ctypes.c_char_p, []),
    "muon_abi_version": (ctypes.c_int32, []),
}

_lock = threading.Lock()
_lib = None


class MuonError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


def load(path: str = LIB_PATH):
    """Loads the HIP library (once).  Raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(path):
            raise RuntimeError(
                f"{LIB_NAME} not found at {path}; build it first with "
                f"`python -m paper_2606_27153_amd.build` (there is no fallback path)")
        lib = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
        return lib


def status_string(status: int) -> str:
    return load().muon_status_string(status).decode()


def last_error() -> str:
    return load().muon_last_error().decode()


def check(status: int) -> None:
    if status != MUON_OK:
        raise MuonError(status, last_error())


def ptr_array(values):
    arr = (ctypes.c_void_p * len(values))()
    for i, v in enumerate(values):
        arr[i] = v
    return arr


def __getattr__(name):
    # muon_* entry points under their C names: _lib.muon_step(...)
    if name in SIGNATURES:
        return getattr(load(), name)
    raise AttributeError(name)
