"""ctypes view of libp4q.so (the C ABI declared in include/p4q.h).

Loading fails loudly when the library has not been built: there is no
fallback implementation of any entry point.
"""
from __future__ import annotations

import ctypes
import os

# P4Q_LIBRARY selects another build of the same library (for instance one
# whose host code is compiled with address and undefined-behaviour
# sanitizers); by default the in-tree build is loaded.
LIB_PATH = os.environ.get("P4Q_LIBRARY") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libp4q.so")

P4Q_OK, P4Q_ERR_INVALID_ARG, P4Q_ERR_UNSUPPORTED, P4Q_ERR_WORKSPACE, P4Q_ERR_HIP = range(5)
P4Q_FP16, P4Q_BF16 = 0, 1

_c_int, _c_size, _c_i64, _c_float, _vp = (ctypes.c_int, ctypes.c_size_t, ctypes.c_int64,
                                          ctypes.c_float, ctypes.c_void_p)

# name -> (restype, argtypes); mirrors include/p4q.h
SIGNATURES = {
    "p4q_version": (ctypes.c_char_p, []),
    "p4q_status_string": (ctypes.c_char_p, [_c_int]),
    "p4q_last_error": (ctypes.c_char_p, []),
    "p4q_select_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int, _c_int]),
    "p4q_select": (_c_int, [_c_int, _c_int, _c_int, _c_int, _vp, _vp, _c_int, _vp, _c_int,
                            _c_int, _c_float, _vp, _vp, _vp, _c_size, _vp]),
    "p4q_select_noalloc": (_c_int, [_c_int, _c_int, _c_int, _c_int, _vp, _vp, _c_int, _vp, _c_int,
                                    _c_int, _c_float, _vp, _vp, _vp]),
    "p4q_select_full_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int, _c_int, _c_int]),
    "p4q_select_budgets": (_c_int, [_c_int, ctypes.POINTER(_c_int), ctypes.POINTER(_c_int),
                                    ctypes.POINTER(_c_int)]),
    "p4q_select_full": (_c_int, [_c_int, _c_int, _c_int, _c_int, _vp, _vp, _c_int, _vp, _vp,
                                 _c_int, _c_int, _c_int, _c_int, _c_float, _vp, _vp, _vp, _vp,
                                 _c_size, _vp]),
    "p4q_quant_act": (_c_int, [_c_int, _c_int, _c_int, _vp, _c_i64, _c_float, _vp, _vp, _vp]),
    "p4q_rmsnorm_quant": (_c_int, [_c_int, _c_int, _c_int, _vp, _c_i64, _vp, _c_float, _c_float,
                                   _vp, _vp, _vp]),
    "p4q_attention_prefill": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _vp,
                                       _c_i64, _vp, _c_i64, _c_int, _vp]),
    "p4q_quant_scaled": (_c_int, [_c_int, _c_int, _c_int, _vp, _c_i64, _vp, _c_int, _c_float, _vp,
                                  _vp, _vp, _vp, _vp, _vp]),
    "p4q_calib_linear_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int]),
    "p4q_calib_linear_grad": (_c_int, [_c_int, _c_int, _c_int, _c_int, _vp, _c_i64, _vp, _c_i64,
                                       _vp, _c_i64, _vp, _c_float, _vp, _vp, _vp, _vp, _vp, _vp,
                                       _c_size, _vp]),
    "p4q_calib_block_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int, _c_int]),
    "p4q_calib_block_grad": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _vp, _vp, _c_i64,
                                      _vp, _vp, _vp, _vp, _vp, _vp, _c_float, _c_float, _vp,
                                      ctypes.POINTER(_c_float), _vp, _vp, _vp, _vp, _vp, _vp,
                                      _c_size, _vp]),
    "p4q_w4a4_linear_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int]),
    "p4q_w4a4_linear": (_c_int, [_c_int, _c_int, _c_int, _vp, _vp, _vp, _vp, _c_int, _vp,
                                 _c_i64, _vp, _vp, _c_size, _vp]),
    "p4q_diag_mfma_i8": (_c_int, [_c_int, _c_int, _vp, _vp]),
    "p4q_diag_stream_read": (_c_int, [_vp, _c_size, _c_int, _vp, _vp]),
}

_lib = None


class P4QError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_name(status)}: {message}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library (raises if libp4q.so is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is not built; run `python -m paper_2609_34867_amd.build` "
                "(or __graft_entry__.build()) first. There is no non-HIP fallback.")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def status_name(status: int) -> str:
    return lib().p4q_status_string(status).decode()


def check(status: int) -> None:
    if status != P4Q_OK:
        raise P4QError(status, lib().p4q_last_error().decode())
