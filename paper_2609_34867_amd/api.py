"""torch-facing wrappers of the libp4q C ABI.

Only argument marshalling happens here: shape / dtype checks, output
allocation with torch (device memory), and passing the current HIP stream.
All computation runs in the library's kernels.
"""
from __future__ import annotations

import ctypes
from typing import Optional, Tuple

import torch

from ._lib import P4Q_BF16, P4Q_ERR_INVALID_ARG, P4Q_FP16, P4QError, check, lib


def version() -> str:
    return lib().p4q_version().decode()


def _dtype_code(t: torch.dtype) -> int:
    if t == torch.float16:
        return P4Q_FP16
    if t == torch.bfloat16:
        return P4Q_BF16
    raise TypeError(f"unsupported dtype {t} (fp16 or bf16)")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(dev: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _need_gpu(*ts):
    """Every given tensor on one GPU (checked after the shape and dtype checks,
    so that those can be exercised without a device)."""
    devs = {t.device for t in ts if t is not None}
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("p4q tensors must live on the GPU")
    if len(devs) > 1:
        raise ValueError(f"p4q tensors of one call must share a device, got {sorted(map(str, devs))}")


def _check(t: Optional[torch.Tensor], name: str, shape=None, dtype=None,
           contiguous: bool = True) -> None:
    """Shape, dtype and layout of a caller-supplied operand or output.  A
    buffer that is too small or of the wrong type would make a kernel read
    or write past its allocation, which the C ABI (plain pointers) cannot
    detect, so every such tensor is checked here before any call."""
    if t is None:
        return
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if dtype is not None:
        ok = t.dtype in dtype if isinstance(dtype, tuple) else t.dtype == dtype
        if not ok:
            raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_rows(t: torch.Tensor, name: str, rows: int, cols: int, dtype=None) -> None:
    """A 2-D operand or output whose rows may be strided: [rows, cols] with
    unit column stride and row stride >= cols."""
    if t.dim() != 2 or t.shape[0] != rows or t.shape[1] != cols:
        raise ValueError(f"{name} must have shape ({rows}, {cols}), got {tuple(t.shape)}")
    if t.stride(1) != 1 or (rows > 1 and t.stride(0) < cols):
        raise ValueError(f"{name} must have unit column stride and row stride >= {cols}")
    if dtype is not None:
        ok = t.dtype in dtype if isinstance(dtype, tuple) else t.dtype == dtype
        if not ok:
            raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


_F16 = (torch.float16, torch.bfloat16)


# --------------------------------------------------------------------------- selector
def select_workspace(B: int, N: int, d: int, J: int, device) -> torch.Tensor:
    """Workspace for select(); its first B*N*(J+1) int32 hold D and Nv per token."""
    n = lib().p4q_select_workspace_bytes(B, N, d, J)
    return torch.empty(n, dtype=torch.uint8, device=device)


def _selector_shapes(vis, concepts, text):
    """(B, N, d, J, T) of the selector's inputs, after checking that they
    agree and share a 16-bit float dtype."""
    if vis.dim() != 3 or concepts.dim() != 3 or (text is not None and text.dim() != 3):
        raise ValueError("vis, concepts and text must be 3-D [B, rows, d]")
    B, N, d = vis.shape
    J = concepts.shape[1]
    T = 0 if text is None else text.shape[1]
    if concepts.shape != (B, J, d) or (text is not None and text.shape != (B, T, d)):
        raise ValueError("shape mismatch between vis, concepts and text")
    for t, name in ((vis, "vis"), (concepts, "concepts"), (text, "text")):
        _check(t, name, None, _F16)
        if t is not None and t.dtype != vis.dtype:
            raise ValueError("vis/concepts/text must share a dtype")
    return B, N, d, J, T


def select(vis: torch.Tensor, concepts: torch.Tensor, text: Optional[torch.Tensor], K: int,
           clip: float = 1.0, idx_out: Optional[torch.Tensor] = None,
           tokens_out: Optional[torch.Tensor] = None,
           workspace: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Quantization-aware Query-Relevance selection (p4q_select).

    vis [B, N, d], concepts [B, J, d], text [B, T, d] or None; returns
    (idx int32 [B, K] ascending, tokens [B, K+T, d] = kept original rows + text)."""
    B, N, d, J, T = _selector_shapes(vis, concepts, text)
    _check(idx_out, "idx_out", (B, K), torch.int32)
    _check(tokens_out, "tokens_out", (B, K + T, d), vis.dtype)
    _check(workspace, "workspace", None, torch.uint8)
    _need_gpu(vis, concepts, text, idx_out, tokens_out, workspace)
    dev = vis.device
    if idx_out is None:
        idx_out = torch.empty((B, K), dtype=torch.int32, device=dev)
    if tokens_out is None:
        tokens_out = torch.empty((B, K + T, d), dtype=vis.dtype, device=dev)
    if workspace is None:
        workspace = select_workspace(B, N, d, J, dev)
    st = lib().p4q_select(_dtype_code(vis.dtype), B, N, d, _ptr(vis), _ptr(concepts), J,
                          _ptr(text) if T > 0 else None, T, K, ctypes.c_float(clip),
                          _ptr(idx_out), _ptr(tokens_out), _ptr(workspace),
                          workspace.numel() * workspace.element_size(), _stream(dev))
    check(st)
    return idx_out, tokens_out


def select_noalloc(vis: torch.Tensor, concepts: torch.Tensor, text: Optional[torch.Tensor],
                   K: int, clip: float = 1.0, idx_out: Optional[torch.Tensor] = None,
                   tokens_out: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """select() without a workspace (p4q_select_noalloc): the library's
    per-device scratch array serves instead, so with idx_out and tokens_out
    given nothing is allocated.  Calls that overlap on one device race."""
    B, N, d, J, T = _selector_shapes(vis, concepts, text)
    _check(idx_out, "idx_out", (B, K), torch.int32)
    _check(tokens_out, "tokens_out", (B, K + T, d), vis.dtype)
    _need_gpu(vis, concepts, text, idx_out, tokens_out)
    dev = vis.device
    if idx_out is None:
        idx_out = torch.empty((B, K), dtype=torch.int32, device=dev)
    if tokens_out is None:
        tokens_out = torch.empty((B, K + T, d), dtype=vis.dtype, device=dev)
    st = lib().p4q_select_noalloc(_dtype_code(vis.dtype), B, N, d, _ptr(vis), _ptr(concepts), J,
                                  _ptr(text) if T > 0 else None, T, K, ctypes.c_float(clip),
                                  _ptr(idx_out), _ptr(tokens_out), _stream(dev))
    check(st)
    return idx_out, tokens_out


def select_budgets(K: int) -> Tuple[int, int, int]:
    """The default (Query Relevance, Visual Saliency, Visual Diversity) token
    budgets for K kept tokens (p4q_select_budgets)."""
    kq, ks, kd = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    check(lib().p4q_select_budgets(K, ctypes.byref(kq), ctypes.byref(ks), ctypes.byref(kd)))
    return kq.value, ks.value, kd.value


def select_full_workspace(B: int, N: int, d: int, J: int, K: int, device) -> torch.Tensor:
    """Workspace for select_full() (holds the B N x N code Gram matrices)."""
    n = lib().p4q_select_full_workspace_bytes(B, N, d, J, K)
    return torch.empty(n, dtype=torch.uint8, device=device)


def select_full(vis: torch.Tensor, concepts: torch.Tensor, cls_attn: torch.Tensor,
                text: Optional[torch.Tensor], K: int, kq: Optional[int] = None,
                ks: Optional[int] = None, clip: float = 1.0,
                idx_out: Optional[torch.Tensor] = None,
                stages_out: Optional[torch.Tensor] = None,
                tokens_out: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None, return_stages: bool = False):
    """The three-stage selector (p4q_select_full): kq tokens by Query Relevance,
    ks by Visual Saliency (cls_attn fp32 [B, N]) over the rest, K - kq - ks by
    Visual Diversity.  kq / ks default to the paper's split of K.

    Returns (idx int32 [B, K] ascending, tokens [B, K+T, d]) and, when
    return_stages, also stages int32 [B, K] (query picks ascending, saliency
    picks ascending, diversity picks in pick order)."""
    B, N, d, J, T = _selector_shapes(vis, concepts, text)
    _check(cls_attn, "cls_attn", (B, N), torch.float32)
    _check(idx_out, "idx_out", (B, K), torch.int32)
    _check(stages_out, "stages_out", (B, K), torch.int32)
    _check(tokens_out, "tokens_out", (B, K + T, d), vis.dtype)
    _check(workspace, "workspace", None, torch.uint8)
    _need_gpu(vis, concepts, cls_attn, text, idx_out, stages_out, tokens_out, workspace)
    if kq is None or ks is None:
        dq, ds, _ = select_budgets(K)
        kq = dq if kq is None else kq
        ks = ds if ks is None else ks
    dev = vis.device
    if idx_out is None:
        idx_out = torch.empty((B, K), dtype=torch.int32, device=dev)
    if stages_out is None and return_stages:
        stages_out = torch.empty((B, K), dtype=torch.int32, device=dev)
    if tokens_out is None:
        tokens_out = torch.empty((B, K + T, d), dtype=vis.dtype, device=dev)
    if workspace is None:
        workspace = select_full_workspace(B, N, d, J, K, dev)
    st = lib().p4q_select_full(_dtype_code(vis.dtype), B, N, d, _ptr(vis), _ptr(concepts), J,
                               _ptr(cls_attn), _ptr(text) if T > 0 else None, T, K, kq, ks,
                               ctypes.c_float(clip), _ptr(idx_out), _ptr(stages_out),
                               _ptr(tokens_out), _ptr(workspace),
                               workspace.numel() * workspace.element_size(), _stream(dev))
    check(st)
    if return_stages:
        return idx_out, tokens_out, stages_out
    return idx_out, tokens_out


# --------------------------------------------------------------------------- quantizer
def quant_act(x: torch.Tensor, clip: float = 1.0, codes: Optional[torch.Tensor] = None,
              scales: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Per-row int4 quantize + pack (p4q_quant_act): x [M, K_in] (row stride may
    exceed K_in) -> (codes uint8 [M, K_in/2], scales fp32 [M])."""
    if x.dim() != 2:
        raise ValueError("x must be 2-D")
    M, K_in = x.shape
    _check_rows(x, "x", M, K_in, _F16)
    _check(codes, "codes", (M, K_in // 2), torch.uint8)
    _check(scales, "scales", (M,), torch.float32)
    _need_gpu(x, codes, scales)
    if codes is None:
        codes = torch.empty((M, K_in // 2), dtype=torch.uint8, device=x.device)
    if scales is None:
        scales = torch.empty((M,), dtype=torch.float32, device=x.device)
    st = lib().p4q_quant_act(_dtype_code(x.dtype), M, K_in, _ptr(x), x.stride(0),
                             ctypes.c_float(clip), _ptr(codes), _ptr(scales),
                             _stream(x.device))
    check(st)
    return codes, scales


def rmsnorm_quant(x: torch.Tensor, gamma: torch.Tensor, eps: float = 1e-5, clip: float = 1.0,
                  codes: Optional[torch.Tensor] = None,
                  scales: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Per-token int4 quantize + pack of RMSNorm(x) * gamma (p4q_rmsnorm_quant):
    x [M, d] (row stride may exceed d), gamma [d] of x's dtype -> (codes uint8
    [M, d/2], scales fp32 [M]); the normalized rows are never formed."""
    if x.dim() != 2:
        raise ValueError("x must be 2-D")
    M, d = x.shape
    _check_rows(x, "x", M, d, _F16)
    if gamma.shape != (d,) or gamma.dtype != x.dtype or not gamma.is_contiguous():
        raise ValueError("gamma must be a contiguous [d] tensor of x's dtype")
    _check(codes, "codes", (M, d // 2), torch.uint8)
    _check(scales, "scales", (M,), torch.float32)
    _need_gpu(x, gamma, codes, scales)
    if codes is None:
        codes = torch.empty((M, d // 2), dtype=torch.uint8, device=x.device)
    if scales is None:
        scales = torch.empty((M,), dtype=torch.float32, device=x.device)
    st = lib().p4q_rmsnorm_quant(_dtype_code(x.dtype), M, d, _ptr(x), x.stride(0), _ptr(gamma),
                                 ctypes.c_float(eps), ctypes.c_float(clip), _ptr(codes),
                                 _ptr(scales), _stream(x.device))
    check(st)
    return codes, scales


# --------------------------------------------------------------------------- attention
def attention_prefill(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, B: int, H: int,
                      causal: bool = True, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Attention prefill (p4q_attention_prefill) with head dimension 128.

    q, k, v: 2-D [B*L, >= H*128] views with a shared row stride (e.g. column
    slices of one fused q|k|v output); returns out [B*L, H*128] of the same
    dtype."""
    rows = q.shape[0]
    if rows % B:
        raise ValueError("rows must be B * L")
    L = rows // B
    D = 128
    for t in (q, k, v):
        if t.dim() != 2 or t.shape[0] != rows or t.shape[1] < H * D or t.stride(1) != 1:
            raise ValueError("q, k, v must be 2-D [B*L, >= H*D] with unit column stride")
        if t.stride(0) != q.stride(0) or t.dtype != q.dtype:
            raise ValueError("q, k, v must share row stride and dtype")
    if q.dtype not in _F16:
        raise ValueError(f"q, k, v must be fp16 or bf16, got {q.dtype}")
    if out is not None:
        _check_rows(out, "out", rows, H * D, q.dtype)
    _need_gpu(q, k, v, out)
    if out is None:
        out = torch.empty((rows, H * D), dtype=q.dtype, device=q.device)
    st = lib().p4q_attention_prefill(_dtype_code(q.dtype), B, L, H, D, _ptr(q), _ptr(k), _ptr(v),
                                     q.stride(0), _ptr(out), out.stride(0), int(causal),
                                     _stream(q.device))
    check(st)
    return out


# --------------------------------------------------------------------------- calibration
def quant_scaled(z: torch.Tensor, sigma: torch.Tensor, divide: bool, clip: float = 1.0,
                 clip_rows: Optional[torch.Tensor] = None):
    """Channel-scaled per-row quantizer (p4q_quant_scaled): z [R, K] (row
    stride may exceed K), sigma fp32 [K]; z' = z / sigma (divide) or z * sigma
    -> (codes uint8 [R, K/2], scales fp32 [R], absmax fp32 [R], kstar int32 [R])."""
    if z.dim() != 2:
        raise ValueError("z must be 2-D")
    R, K = z.shape
    _check_rows(z, "z", R, K, _F16)
    if sigma.shape != (K,) or sigma.dtype != torch.float32 or not sigma.is_contiguous():
        raise ValueError("sigma must be a contiguous fp32 [K] tensor")
    if clip_rows is not None and (clip_rows.shape != (R,) or clip_rows.dtype != torch.float32
                                  or not clip_rows.is_contiguous()):
        raise ValueError("clip_rows must be a contiguous fp32 [R] tensor")
    _need_gpu(z, sigma, clip_rows)
    dev = z.device
    codes = torch.empty((R, K // 2), dtype=torch.uint8, device=dev)
    scales = torch.empty((R,), dtype=torch.float32, device=dev)
    absmax = torch.empty((R,), dtype=torch.float32, device=dev)
    kstar = torch.empty((R,), dtype=torch.int32, device=dev)
    st = lib().p4q_quant_scaled(_dtype_code(z.dtype), R, K, _ptr(z), z.stride(0), _ptr(sigma),
                                int(bool(divide)), ctypes.c_float(clip),
                                _ptr(clip_rows) if clip_rows is not None else None, _ptr(codes),
                                _ptr(scales), _ptr(absmax), _ptr(kstar), _stream(dev))
    check(st)
    return codes, scales, absmax, kstar


def calib_linear_workspace(M: int, N: int, K: int, device) -> torch.Tensor:
    n = lib().p4q_calib_linear_workspace_bytes(M, N, K)
    if n == 0:
        raise P4QError(P4Q_ERR_INVALID_ARG, f"unsupported calibration shape M={M} N={N} K={K}")
    return torch.empty(n, dtype=torch.uint8, device=device)


def calib_linear_grad(x: torch.Tensor, w: torch.Tensor, target: torch.Tensor,
                      sigma: torch.Tensor, clip_a: float, clip_w: torch.Tensor,
                      workspace: Optional[torch.Tensor] = None, out=None):
    """One calibration step of a W4A4 fake-quantized linear
    (p4q_calib_linear_grad): x [M, K], w [N, K] (same dtype), target fp32
    [M, N], sigma fp32 [K], clip_w fp32 [N] -> (loss [1], grad_sigma [K],
    grad_clip_a [1], grad_clip_w [N]), all fp32 device tensors.  `out` may
    hold those four tensors to be written in place."""
    for t, name in ((x, "x"), (w, "w"), (target, "target")):
        if t.dim() != 2 or t.stride(1) != 1:
            raise ValueError(f"{name} must be 2-D with unit column stride")
    M, K = x.shape
    N = w.shape[0]
    if w.shape[1] != K or w.dtype != x.dtype:
        raise ValueError("w must be [N, K] of x's dtype")
    if target.shape != (M, N) or target.dtype != torch.float32:
        raise ValueError("target must be fp32 [M, N]")
    for t, n, name in ((sigma, K, "sigma"), (clip_w, N, "clip_w")):
        if t.shape != (n,) or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous fp32 [{n}] tensor")
    if x.dtype not in _F16:
        raise ValueError(f"x and w must be fp16 or bf16, got {x.dtype}")
    if out is not None:
        if len(out) != 4:
            raise ValueError("out must hold (loss, grad_sigma, grad_clip_a, grad_clip_w)")
        for t, n, name in zip(out, (1, K, 1, N), ("loss", "grad_sigma", "grad_clip_a", "grad_clip_w")):
            _check(t, name, (n,), torch.float32)
    _check(workspace, "workspace", None, torch.uint8)
    _need_gpu(x, w, target, sigma, clip_w, workspace, *(out or ()))
    dev = x.device
    if out is None:
        out = (torch.empty(1, dtype=torch.float32, device=dev),
               torch.empty(K, dtype=torch.float32, device=dev),
               torch.empty(1, dtype=torch.float32, device=dev),
               torch.empty(N, dtype=torch.float32, device=dev))
    if workspace is None:
        workspace = calib_linear_workspace(M, N, K, dev)
    loss, gs, gca, gcw = out
    st = lib().p4q_calib_linear_grad(_dtype_code(x.dtype), M, N, K, _ptr(x), x.stride(0), _ptr(w),
                                     w.stride(0), _ptr(target), target.stride(0), _ptr(sigma),
                                     ctypes.c_float(clip_a), _ptr(clip_w), _ptr(loss), _ptr(gs),
                                     _ptr(gca), _ptr(gcw), _ptr(workspace), workspace.numel(),
                                     _stream(dev))
    check(st)
    return loss, gs, gca, gcw


def calib_block_workspace(M: int, d: int, f: int, H: int, device) -> torch.Tensor:
    n = lib().p4q_calib_block_workspace_bytes(M, d, f, H)
    if n == 0:
        raise P4QError(P4Q_ERR_INVALID_ARG, f"unsupported block shape M={M} d={d} f={f} H={H}")
    return torch.empty(n, dtype=torch.uint8, device=device)


def calib_block_grad(x: torch.Tensor, target: torch.Tensor, w_qkv: torch.Tensor,
                     w_o: torch.Tensor, w_gu: torch.Tensor, w_down: torch.Tensor,
                     gamma1: torch.Tensor, gamma2: torch.Tensor, H: int, sigma: torch.Tensor,
                     clip_a, clip_w: torch.Tensor, eps: float = 1e-5, rope_base: float = 10000.0,
                     workspace: Optional[torch.Tensor] = None, out=None):
    """One calibration step of a W4A4 fake-quantized decoder block
    (p4q_calib_block_grad): x fp16 [M, d], target fp32 [M, d], weights fp16
    (q|k|v [3d, d], o [d, d], gate|up [2f, d], down [d, f]), RMSNorm weights
    fp16 [d]; sigma fp32 [3d + f] (groups q|k|v, o, gate|up, down), clip_a
    four floats (host), clip_w fp32 [5d + 2f].  Returns (loss [1],
    grad_sigma [3d + f], grad_clip_a [4], grad_clip_w [5d + 2f]) as fp32
    device tensors; `out` may hold those four to be written in place."""
    if x.dim() != 2:
        raise ValueError("x must be 2-D [M, d]")
    M, d = x.shape
    if w_down.dim() != 2 or w_down.shape[0] != d:
        raise ValueError("w_down must be [d, f]")
    f = w_down.shape[1]
    for t, shape, name in ((x, (M, d), "x"), (w_qkv, (3 * d, d), "w_qkv"), (w_o, (d, d), "w_o"),
                           (w_gu, (2 * f, d), "w_gu"), (w_down, (d, f), "w_down"),
                           (gamma1, (d,), "gamma1"), (gamma2, (d,), "gamma2")):
        _check(t, name, shape, torch.float16)
    _check(target, "target", (M, d), torch.float32)
    _check(sigma, "sigma", (3 * d + f,), torch.float32)
    _check(clip_w, "clip_w", (5 * d + 2 * f,), torch.float32)
    ca = [float(c) for c in clip_a]
    if len(ca) != 4:
        raise ValueError("clip_a must hold four factors (q|k|v, o, gate|up, down)")
    if out is not None:
        if len(out) != 4:
            raise ValueError("out must hold (loss, grad_sigma, grad_clip_a, grad_clip_w)")
        for t, n, name in zip(out, (1, 3 * d + f, 4, 5 * d + 2 * f),
                              ("loss", "grad_sigma", "grad_clip_a", "grad_clip_w")):
            _check(t, name, (n,), torch.float32)
    _check(workspace, "workspace", None, torch.uint8)
    _need_gpu(x, target, w_qkv, w_o, w_gu, w_down, gamma1, gamma2, sigma, clip_w, workspace,
              *(out or ()))
    dev = x.device
    if out is None:
        out = tuple(torch.empty(n, dtype=torch.float32, device=dev)
                    for n in (1, 3 * d + f, 4, 5 * d + 2 * f))
    if workspace is None:
        workspace = calib_block_workspace(M, d, f, H, dev)
    loss, gs, gca, gcw = out
    ca_arr = (ctypes.c_float * 4)(*ca)
    st = lib().p4q_calib_block_grad(P4Q_FP16, M, d, f, H, _ptr(x), _ptr(target), target.stride(0),
                                    _ptr(w_qkv), _ptr(w_o), _ptr(w_gu), _ptr(w_down),
                                    _ptr(gamma1), _ptr(gamma2), ctypes.c_float(eps),
                                    ctypes.c_float(rope_base), _ptr(sigma), ca_arr, _ptr(clip_w),
                                    _ptr(loss), _ptr(gs), _ptr(gca), _ptr(gcw), _ptr(workspace),
                                    workspace.numel(), _stream(dev))
    check(st)
    return loss, gs, gca, gcw


# --------------------------------------------------------------------------- W4A4 linear
def w4a4_linear_workspace(M: int, N_out: int, K_in: int, device) -> Optional[torch.Tensor]:
    n = lib().p4q_w4a4_linear_workspace_bytes(M, N_out, K_in)
    # zero-filled: its head holds arrival counters that must start at zero
    # (every call leaves them zero again)
    return None if n == 0 else torch.zeros(n, dtype=torch.uint8, device=device)


def w4a4_linear(a_codes: torch.Tensor, a_scales: torch.Tensor, w_codes: torch.Tensor,
                w_scales: torch.Tensor, out_dtype: torch.dtype = torch.bfloat16,
                y: Optional[torch.Tensor] = None, acc_out: Optional[torch.Tensor] = None,
                return_acc: bool = False, workspace: Optional[torch.Tensor] = None):
    """W4A4 linear (p4q_w4a4_linear): a_codes [M, K_in/2], w_codes [N_out, K_in/2]
    -> y [M, N_out] (out_dtype); also the int32 accumulators when return_acc.
    Without `workspace` one of the size the library asks for is allocated
    (small M splits K across work-groups with it); a smaller one, e.g.
    empty, runs the unsplit kernel.  Results are identical either way."""
    if a_codes.dim() != 2 or w_codes.dim() != 2:
        raise ValueError("a_codes and w_codes must be 2-D [rows, K_in/2]")
    M, kb = a_codes.shape
    N_out, kb2 = w_codes.shape
    if kb != kb2:
        raise ValueError("a_codes and w_codes disagree on K_in")
    _check(a_codes, "a_codes", (M, kb), torch.uint8)
    _check(w_codes, "w_codes", (N_out, kb), torch.uint8)
    _check(a_scales, "a_scales", (M,), torch.float32)
    _check(w_scales, "w_scales", (N_out,), torch.float32)
    if y is not None:
        _check_rows(y, "y", M, N_out, _F16)
    _check(acc_out, "acc_out", (M, N_out), torch.int32)
    _check(workspace, "workspace", None, torch.uint8)
    _need_gpu(a_codes, a_scales, w_codes, w_scales, y, acc_out, workspace)
    K_in = 2 * kb
    dev = a_codes.device
    if y is None:
        y = torch.empty((M, N_out), dtype=out_dtype, device=dev)
    if return_acc and acc_out is None:
        acc_out = torch.empty((M, N_out), dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = w4a4_linear_workspace(M, N_out, K_in, dev)
    ws_bytes = 0 if workspace is None else workspace.numel()
    st = lib().p4q_w4a4_linear(M, N_out, K_in, _ptr(a_codes), _ptr(a_scales), _ptr(w_codes),
                               _ptr(w_scales), _dtype_code(y.dtype), _ptr(y), y.stride(0),
                               _ptr(acc_out), _ptr(workspace), ws_bytes, _stream(dev))
    check(st)
    return (y, acc_out) if return_acc else y


# --------------------------------------------------------------------------- diagnostics
def diag_mfma_i8(blocks: int, iters: int, out: torch.Tensor) -> int:
    """Enqueue the int8 MFMA microbenchmark (p4q_diag_mfma_i8) writing its
    checksums to out (int32, >= blocks * 256 entries); returns the integer
    operations it performs."""
    _check(out, "out", None, torch.int32)
    if out.numel() < blocks * 256:
        raise ValueError(f"out needs {blocks * 256} entries")
    _need_gpu(out)
    check(lib().p4q_diag_mfma_i8(blocks, iters, _ptr(out), _stream(out.device)))
    return blocks * 4 * iters * 16 * 2 * 16 * 16 * 64


def diag_stream_read(src: torch.Tensor, blocks: int, out: torch.Tensor) -> int:
    """Enqueue the HBM read microbenchmark (p4q_diag_stream_read) over the
    bytes of src; returns the bytes read."""
    _check(src, "src", None, None)
    _check(out, "out", None, torch.int32)
    if out.numel() < blocks * 256:
        raise ValueError(f"out needs {blocks * 256} entries")
    nbytes = src.numel() * src.element_size()
    _need_gpu(src, out)
    check(lib().p4q_diag_stream_read(_ptr(src), nbytes, blocks, _ptr(out), _stream(src.device)))
    return nbytes
