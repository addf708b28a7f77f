"""Host-side argument checks of the Python binding (CPU, no GPU, no library
call).  Every caller-supplied operand and output is checked for shape, dtype
and layout before anything reaches the C ABI: a buffer of the wrong size or
type would otherwise be read or written past its end on the device, which
plain pointers cannot reveal.  The library is replaced by a stub that fails
the test if it is touched, so each error below is raised before any call."""
import pytest
import torch

import paper_2609_34867_amd.api as api


@pytest.fixture(autouse=True)
def no_library(monkeypatch):
    def forbidden():
        raise AssertionError("the library was called before the argument checks")
    monkeypatch.setattr(api, "lib", forbidden)


def f16(*shape):
    return torch.zeros(shape, dtype=torch.float16)


def u8(*shape):
    return torch.zeros(shape, dtype=torch.uint8)


def f32(*shape):
    return torch.zeros(shape, dtype=torch.float32)


def i32(*shape):
    return torch.zeros(shape, dtype=torch.int32)


def raises(match, fn, *a, **k):
    with pytest.raises(ValueError, match=match):
        fn(*a, **k)


# ------------------------------------------------------------------ W4A4 linear
def test_linear_checks_every_operand():
    a, sa, w, sw = u8(8, 64), f32(8), u8(16, 64), f32(16)
    raises("must live on the GPU", api.w4a4_linear, a, sa, w, sw)     # all shapes valid
    raises("disagree on K_in", api.w4a4_linear, a, sa, u8(16, 32), sw)
    raises("a_codes must be torch.uint8", api.w4a4_linear, a.to(torch.int8), sa, w, sw)
    raises("w_codes must be torch.uint8", api.w4a4_linear, a, sa, w.to(torch.int8), sw)
    raises(r"a_scales must have shape \(8,\)", api.w4a4_linear, a, f32(7), w, sw)
    raises("a_scales must be torch.float32", api.w4a4_linear, a, sa.half(), w, sw)
    raises(r"w_scales must have shape \(16,\)", api.w4a4_linear, a, sa, w, f32(17))
    raises("a_codes must be contiguous", api.w4a4_linear, u8(64, 8).t(), sa, w, sw)


def test_linear_checks_outputs():
    a, sa, w, sw = u8(8, 64), f32(8), u8(16, 64), f32(16)
    raises(r"y must have shape \(8, 16\)", api.w4a4_linear, a, sa, w, sw, y=f16(7, 16))
    raises(r"y must have shape \(8, 16\)", api.w4a4_linear, a, sa, w, sw, y=f16(8, 15))
    raises("unit column stride", api.w4a4_linear, a, sa, w, sw, y=f16(16, 8).t())
    raises("y must be", api.w4a4_linear, a, sa, w, sw, y=f32(8, 16))
    raises(r"acc_out must have shape \(8, 16\)", api.w4a4_linear, a, sa, w, sw, acc_out=i32(8, 8))
    raises("acc_out must be torch.int32", api.w4a4_linear, a, sa, w, sw, acc_out=f32(8, 16))
    raises("workspace must be torch.uint8", api.w4a4_linear, a, sa, w, sw, workspace=f32(64))
    # a wider row stride for y is allowed (a column slice of a larger output)
    raises("must live on the GPU", api.w4a4_linear, a, sa, w, sw, y=f16(8, 24)[:, :16])


# ------------------------------------------------------------------ quantizers
def test_quant_act_checks():
    x = f16(4, 64)
    raises("must live on the GPU", api.quant_act, x)
    raises("x must be 2-D", api.quant_act, f16(64))
    raises("x must be", api.quant_act, f32(4, 64))
    raises(r"codes must have shape \(4, 32\)", api.quant_act, x, codes=u8(4, 31))
    raises("codes must be torch.uint8", api.quant_act, x, codes=f16(4, 32))
    raises(r"scales must have shape \(4,\)", api.quant_act, x, scales=f32(3))
    raises("scales must be torch.float32", api.quant_act, x, scales=f16(4))
    raises("unit column stride", api.quant_act, f16(64, 4).t())


def test_rmsnorm_quant_checks():
    x, g = f16(4, 64), f16(64)
    raises("must live on the GPU", api.rmsnorm_quant, x, g)
    raises("gamma must be", api.rmsnorm_quant, x, f16(32))
    raises("gamma must be", api.rmsnorm_quant, x, g.bfloat16())
    raises(r"codes must have shape \(4, 32\)", api.rmsnorm_quant, x, g, codes=u8(5, 32))
    raises(r"scales must have shape \(4,\)", api.rmsnorm_quant, x, g, scales=f32(5))


def test_quant_scaled_checks():
    z, s = f16(3, 64), f32(64)
    raises("must live on the GPU", api.quant_scaled, z, s, True)
    raises("sigma must be", api.quant_scaled, z, f32(32), True)
    raises("clip_rows must be", api.quant_scaled, z, s, True, 1.0, f32(2))
    raises("z must be", api.quant_scaled, f32(3, 64), s, True)


# ------------------------------------------------------------------ selectors
def test_select_checks():
    vis, con, txt = f16(2, 10, 64), f16(2, 3, 64), f16(2, 4, 64)
    raises("must live on the GPU", api.select, vis, con, txt, 5)
    raises("shape mismatch", api.select, vis, f16(1, 3, 64), txt, 5)
    raises("share a dtype", api.select, vis, con.bfloat16(), txt, 5)
    raises("vis must be", api.select, vis.float(), con.float(), txt.float(), 5)
    raises(r"idx_out must have shape \(2, 5\)", api.select, vis, con, txt, 5, idx_out=i32(2, 4))
    raises("idx_out must be torch.int32", api.select, vis, con, txt, 5, idx_out=f32(2, 5))
    raises(r"tokens_out must have shape \(2, 9, 64\)", api.select, vis, con, txt, 5,
           tokens_out=f16(2, 8, 64))
    raises("tokens_out must be", api.select, vis, con, txt, 5, tokens_out=f16(2, 9, 64).bfloat16())
    raises("workspace must be torch.uint8", api.select, vis, con, txt, 5, workspace=f32(16))
    raises("vis must be contiguous", api.select, f16(2, 64, 10).transpose(1, 2), con, txt, 5)


def test_select_full_checks():
    vis, con, txt, cls = f16(2, 10, 64), f16(2, 3, 64), f16(2, 4, 64), f32(2, 10)
    raises("must live on the GPU", api.select_full, vis, con, cls, txt, 5, 1, 1)
    raises(r"cls_attn must have shape \(2, 10\)", api.select_full, vis, con, f32(2, 9), txt, 5, 1, 1)
    raises("cls_attn must be torch.float32", api.select_full, vis, con, cls.half(), txt, 5, 1, 1)
    raises(r"stages_out must have shape \(2, 5\)", api.select_full, vis, con, cls, txt, 5, 1, 1,
           stages_out=i32(2, 6))
    raises(r"tokens_out must have shape \(2, 9, 64\)", api.select_full, vis, con, cls, txt, 5, 1, 1,
           tokens_out=f16(2, 10, 64))


# ------------------------------------------------------------------ attention, calibration
def test_attention_checks():
    qkv = f16(2 * 6, 3 * 128)
    q, k, v = qkv[:, :128], qkv[:, 128:256], qkv[:, 256:]
    raises("must live on the GPU", api.attention_prefill, q, k, v, 2, 1)
    raises(r"out must have shape \(12, 128\)", api.attention_prefill, q, k, v, 2, 1, out=f16(12, 64))
    raises("out must be", api.attention_prefill, q, k, v, 2, 1, out=f32(12, 128))
    raises("rows must be B", api.attention_prefill, q, k, v, 5, 1)


def test_calib_checks():
    x, w, t, s, cw = f16(4, 128), f16(64, 128), f32(4, 64), f32(128), f32(64)
    raises("must live on the GPU", api.calib_linear_grad, x, w, t, s, 1.0, cw)
    raises("target must be", api.calib_linear_grad, x, w, f32(4, 63), s, 1.0, cw)
    raises("w must be", api.calib_linear_grad, x, w.bfloat16(), t, s, 1.0, cw)
    raises("clip_w must be", api.calib_linear_grad, x, w, t, s, 1.0, f32(63))
    bad = (f32(1), f32(128), f32(1), f32(63))
    raises(r"grad_clip_w must have shape \(64,\)", api.calib_linear_grad, x, w, t, s, 1.0, cw, out=bad)
