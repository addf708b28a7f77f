"""P4Q hot path on MI355X: quantization-aware visual-token selection and W4A4
linear layers, as hand-written gfx950 HIP kernels behind the C ABI in
include/p4q.h.  This package only marshals torch tensors (device memory and
the current stream) into those calls; every step runs in libp4q.so.
"""
from ._lib import P4QError, lib, LIB_PATH  # noqa: F401
from .api import (select, select_workspace, select_noalloc, select_full, select_full_workspace,  # noqa: F401
                  select_budgets, quant_act, rmsnorm_quant, attention_prefill,
                  quant_scaled, calib_linear_grad, calib_linear_workspace, calib_block_grad,
                  calib_block_workspace,
                  w4a4_linear, w4a4_linear_workspace, diag_mfma_i8, diag_stream_read,
                  version)

__all__ = ["select", "select_workspace", "select_noalloc", "select_full", "select_full_workspace",
           "select_budgets", "quant_act", "rmsnorm_quant", "attention_prefill",
           "quant_scaled", "calib_linear_grad", "calib_linear_workspace", "calib_block_grad",
           "calib_block_workspace", "w4a4_linear", "w4a4_linear_workspace", "diag_mfma_i8", "diag_stream_read", "version",
           "P4QError", "lib", "LIB_PATH"]
