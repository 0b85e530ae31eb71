"""ctypes declarations of the libvtrace C ABI (include/vtrace.h).

Loading fails loudly when the library has not been built: there is no
fallback implementation anywhere in this package.
"""

from __future__ import annotations

import ctypes
import os

# VTRACE_LIB names another build of the same library (the host-instrumented
# one of sanitize.py); by default the in-tree libvtrace.so.
LIB_PATH = os.environ.get("VTRACE_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                        "libvtrace.so")

VTRACE_F32 = 0
VTRACE_BF16 = 1
STATUS_NAMES = {
    0: "VTRACE_OK",
    1: "VTRACE_ERR_NULL",
    2: "VTRACE_ERR_SHAPE",
    3: "VTRACE_ERR_DTYPE",
    4: "VTRACE_ERR_PARAM",
    5: "VTRACE_ERR_ALIGN",
    6: "VTRACE_ERR_WORKSPACE",
    7: "VTRACE_ERR_HIP",
}

CORRECTIONS = {"vtrace": 0, "none": 1, "epsilon": 2, "one_step_is": 3}
Q_ESTIMATES = {"vtrace": 0, "baseline": 1}
BEHAVIOUR_INPUTS = {"logits": 0, "log_probs": 1}
REWARD_TRANSFORMS = {None: 0, "clip": 1, "asymmetric": 2}


class Variant(ctypes.Structure):
    """vtrace_variant: correction, Q estimate, epsilon, behaviour input kind,
    reward transform and gradient dtype."""
    _fields_ = [("correction", ctypes.c_int32), ("q_estimate", ctypes.c_int32),
                ("epsilon", ctypes.c_float), ("behaviour_input", ctypes.c_int32),
                ("reward_transform", ctypes.c_int32), ("grad_dtype", ctypes.c_int32)]


# Every symbol include/vtrace.h declares, with (restype, argtypes).
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_F = ctypes.c_float
_INPUTS = [_I64, _I64, _I64, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _F, _F, _F]
SIGNATURES = {
    "vtrace_abi_version": (ctypes.c_int, []),
    "vtrace_status_string": (ctypes.c_char_p, [ctypes.c_int32]),
    "vtrace_max_elements": (ctypes.c_int64, []),
    "vtrace_workspace_bytes": (ctypes.c_size_t, [_I64, _I64, _I64]),
    "vtrace_workspace_init": (ctypes.c_int, [_P, ctypes.c_size_t, _P]),
    "vtrace_targets": (ctypes.c_int, _INPUTS + [_P, _P, _P, ctypes.c_size_t, _P]),
    "vtrace_loss_grad": (ctypes.c_int, _INPUTS + [_F, _F, _P, _P, _P, _P, _P, _P, _P,
                                                  ctypes.c_size_t, _P]),
    "vtrace_targets_ex": (ctypes.c_int, _INPUTS + [ctypes.POINTER(Variant), _P, _P, _P,
                                                   ctypes.c_size_t, _P]),
    "vtrace_loss_grad_ex": (ctypes.c_int, _INPUTS + [_F, _F, ctypes.POINTER(Variant), _P, _P, _P,
                                                     _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "vtrace_loss_grad_static": (ctypes.c_int, _INPUTS + [_F, _F, ctypes.POINTER(Variant), _P, _P, _P, _P,
                                                         _P, _P, _P]),
    "vtrace_head_workspace_bytes": (ctypes.c_size_t, [_I64, _I64, _I64, _I64]),
    "vtrace_head_loss_grad": (ctypes.c_int, [_I64, _I64, _I64, _I64, ctypes.c_int, _P, _P, _P, _P, _P,
                                             _P, _P, _P, _F, _F, _F, _F, _F,
                                             ctypes.POINTER(Variant), _P, _P, _P, _P, _P, _P, _P,
                                             _P, _P, ctypes.c_size_t, _P]),
    "vtrace_gather_logits": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_int, _P, _P, _P, _P, _P]),
    "vtrace_error_flag": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int32), _P]),
}

_lib = None


class VtraceError(RuntimeError):
    def __init__(self, status: int, lib):
        msg = lib.vtrace_status_string(status).decode()
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def lib():
    """The loaded library, with argument types declared."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_1802_01561_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != 0:
        raise VtraceError(status, lib())
