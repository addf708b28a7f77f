"""The C ABI library loads, exports every symbol include/p4q.h declares, and
rejects bad arguments on the host before any HIP call (no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_2609_34867_amd import _lib as L

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "p4q.h")



@pytest.fixture(scope="module", autouse=True)
def built_library():
    """The ABI tests need the library: build it when it is missing rather
    than skip (a CPU-only run must not report these tests green untested)."""
    if not os.path.exists(L.LIB_PATH):
        from paper_2609_34867_amd.build import build
        build()

ALIGNED = 0x10000       # fake device addresses: only validated, never dereferenced
F = ctypes.c_float


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(p4q_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = L.lib()
    names = declared_functions()
    assert len(names) >= 8
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L.SIGNATURES), "binding signatures out of sync with the header"


def test_version_and_status_strings():
    lib = L.lib()
    assert b"gfx950" in lib.p4q_version()
    assert lib.p4q_status_string(0) == b"P4Q_OK"
    assert lib.p4q_status_string(3) == b"P4Q_ERR_WORKSPACE"
    assert lib.p4q_status_string(99) == b"P4Q_ERR_UNKNOWN"


def quant(**kw):
    a = dict(dt=0, M=4, K=64, x=ALIGNED, ldx=64, clip=1.0, codes=ALIGNED, scales=ALIGNED)
    a.update(kw)
    return L.lib().p4q_quant_act(a["dt"], a["M"], a["K"], a["x"], a["ldx"], F(a["clip"]),
                                 a["codes"], a["scales"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(M=0), L.P4Q_ERR_INVALID_ARG),
    (dict(K=48), L.P4Q_ERR_INVALID_ARG),
    (dict(K=65536 + 32, ldx=65568), L.P4Q_ERR_UNSUPPORTED),
    (dict(ldx=32), L.P4Q_ERR_INVALID_ARG),
    (dict(ldx=68), L.P4Q_ERR_INVALID_ARG),
    (dict(x=None), L.P4Q_ERR_INVALID_ARG),
    (dict(x=ALIGNED + 8), L.P4Q_ERR_INVALID_ARG),
    (dict(clip=0.0), L.P4Q_ERR_INVALID_ARG),
    (dict(clip=1.5), L.P4Q_ERR_INVALID_ARG),
    (dict(clip=float("nan")), L.P4Q_ERR_INVALID_ARG),
    (dict(dt=7), L.P4Q_ERR_UNSUPPORTED),
])
def test_quant_act_validation(kw, status):
    assert quant(**kw) == status
    assert L.lib().p4q_last_error() != b""


def select(**kw):
    a = dict(dt=0, B=1, N=64, d=64, vis=ALIGNED, con=ALIGNED, J=2, text=ALIGNED, T=4, K=8,
             clip=1.0, idx=ALIGNED, tok=ALIGNED, ws=ALIGNED, ws_bytes=1 << 30)
    a.update(kw)
    return L.lib().p4q_select(a["dt"], a["B"], a["N"], a["d"], a["vis"], a["con"], a["J"],
                              a["text"], a["T"], a["K"], F(a["clip"]), a["idx"], a["tok"],
                              a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(K=65), L.P4Q_ERR_INVALID_ARG),
    (dict(K=0), L.P4Q_ERR_INVALID_ARG),
    (dict(J=0), L.P4Q_ERR_INVALID_ARG),
    (dict(J=9), L.P4Q_ERR_UNSUPPORTED),
    (dict(d=48), L.P4Q_ERR_INVALID_ARG),
    (dict(N=9000, K=8), L.P4Q_ERR_UNSUPPORTED),
    (dict(text=None), L.P4Q_ERR_INVALID_ARG),
    (dict(T=0), L.P4Q_ERR_INVALID_ARG),
    (dict(vis=None), L.P4Q_ERR_INVALID_ARG),
    (dict(vis=ALIGNED + 4), L.P4Q_ERR_INVALID_ARG),
    (dict(ws=None), L.P4Q_ERR_WORKSPACE),
    (dict(ws_bytes=100), L.P4Q_ERR_WORKSPACE),
    (dict(ws=ALIGNED + 16), L.P4Q_ERR_INVALID_ARG),
    (dict(clip=2.0), L.P4Q_ERR_INVALID_ARG),
    (dict(dt=2), L.P4Q_ERR_UNSUPPORTED),
    (dict(J=5, d=8224), L.P4Q_ERR_UNSUPPORTED),
])
def test_select_validation(kw, status):
    assert select(**kw) == status


def test_select_workspace_size_covers_documented_stats():
    n = L.lib().p4q_select_workspace_bytes(16, 2880, 4096, 4)
    assert n >= 16 * 2880 * 5 * 4
    assert L.lib().p4q_select_workspace_bytes(0, 1, 1, 1) == 0


def select_full(**kw):
    a = dict(dt=0, B=1, N=64, d=64, vis=ALIGNED, con=ALIGNED, J=2, cls=ALIGNED, text=ALIGNED,
             T=4, K=10, kq=3, ks=2, clip=1.0, idx=ALIGNED, stages=None, tok=ALIGNED,
             ws=ALIGNED, ws_bytes=1 << 30)
    a.update(kw)
    return L.lib().p4q_select_full(a["dt"], a["B"], a["N"], a["d"], a["vis"], a["con"], a["J"],
                                   a["cls"], a["text"], a["T"], a["K"], a["kq"], a["ks"],
                                   F(a["clip"]), a["idx"], a["stages"], a["tok"], a["ws"],
                                   a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(K=65), L.P4Q_ERR_INVALID_ARG),
    (dict(kq=-1), L.P4Q_ERR_INVALID_ARG),
    (dict(ks=-1), L.P4Q_ERR_INVALID_ARG),
    (dict(kq=6, ks=5), L.P4Q_ERR_INVALID_ARG),
    (dict(cls=None), L.P4Q_ERR_INVALID_ARG),
    (dict(cls=ALIGNED + 2), L.P4Q_ERR_INVALID_ARG),
    (dict(stages=ALIGNED + 1), L.P4Q_ERR_INVALID_ARG),
    (dict(d=8224), L.P4Q_ERR_UNSUPPORTED),
    (dict(N=9000), L.P4Q_ERR_UNSUPPORTED),
    (dict(J=9), L.P4Q_ERR_UNSUPPORTED),
    (dict(ws_bytes=1000), L.P4Q_ERR_WORKSPACE),
    (dict(ws=ALIGNED + 64), L.P4Q_ERR_INVALID_ARG),
    (dict(text=None), L.P4Q_ERR_INVALID_ARG),
    (dict(dt=3), L.P4Q_ERR_UNSUPPORTED),
])
def test_select_full_validation(kw, status):
    assert select_full(**kw) == status
    assert L.lib().p4q_last_error() != b""


def test_select_full_workspace_holds_gram_matrices():
    n = L.lib().p4q_select_full_workspace_bytes(16, 2880, 4096, 4, 640)
    assert n >= 16 * 2880 * 2880 * 4 + L.lib().p4q_select_workspace_bytes(16, 2880, 4096, 4)
    assert L.lib().p4q_select_full_workspace_bytes(1, 1, 32, 1, 0) == 0


def test_select_budgets_match_the_oracle():
    import ctypes
    import oracle
    for K in (0, 1, 2, 64, 192, 320, 640, 2879):
        kq, ks, kd = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        assert L.lib().p4q_select_budgets(K, ctypes.byref(kq), ctypes.byref(ks),
                                          ctypes.byref(kd)) == L.P4Q_OK
        assert (kq.value, ks.value, kd.value) == oracle.stage_budgets(K)
    assert L.lib().p4q_select_budgets(-1, ctypes.byref(kq), ctypes.byref(ks),
                                      ctypes.byref(kd)) == L.P4Q_ERR_INVALID_ARG
    assert L.lib().p4q_select_budgets(5, None, ctypes.byref(ks),
                                      ctypes.byref(kd)) == L.P4Q_ERR_INVALID_ARG


def rmsq(**kw):
    a = dict(dt=0, M=4, d=64, x=ALIGNED, ldx=64, g=ALIGNED, eps=1e-5, clip=1.0, codes=ALIGNED,
             scales=ALIGNED)
    a.update(kw)
    return L.lib().p4q_rmsnorm_quant(a["dt"], a["M"], a["d"], a["x"], a["ldx"], a["g"],
                                     F(a["eps"]), F(a["clip"]), a["codes"], a["scales"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(M=0), L.P4Q_ERR_INVALID_ARG),
    (dict(d=48, ldx=48), L.P4Q_ERR_INVALID_ARG),
    (dict(d=16416, ldx=16416), L.P4Q_ERR_UNSUPPORTED),
    (dict(ldx=60), L.P4Q_ERR_INVALID_ARG),
    (dict(ldx=68), L.P4Q_ERR_INVALID_ARG),
    (dict(g=None), L.P4Q_ERR_INVALID_ARG),
    (dict(g=ALIGNED + 2), L.P4Q_ERR_INVALID_ARG),
    (dict(eps=-1.0), L.P4Q_ERR_INVALID_ARG),
    (dict(eps=float("nan")), L.P4Q_ERR_INVALID_ARG),
    (dict(clip=0.0), L.P4Q_ERR_INVALID_ARG),
    (dict(dt=9), L.P4Q_ERR_UNSUPPORTED),
])
def test_rmsnorm_quant_validation(kw, status):
    assert rmsq(**kw) == status
    assert L.lib().p4q_last_error() != b""


def attn(**kw):
    a = dict(dt=0, B=1, L=16, H=2, D=128, q=ALIGNED, k=ALIGNED, v=ALIGNED, ld=768, o=ALIGNED,
             ldo=256, causal=1)
    a.update(kw)
    return L.lib().p4q_attention_prefill(a["dt"], a["B"], a["L"], a["H"], a["D"], a["q"], a["k"],
                                         a["v"], a["ld"], a["o"], a["ldo"], a["causal"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(L=0), L.P4Q_ERR_INVALID_ARG),
    (dict(D=64), L.P4Q_ERR_UNSUPPORTED),
    (dict(causal=2), L.P4Q_ERR_INVALID_ARG),
    (dict(ld=200), L.P4Q_ERR_INVALID_ARG),
    (dict(ld=772), L.P4Q_ERR_INVALID_ARG),
    (dict(ldo=255), L.P4Q_ERR_INVALID_ARG),
    (dict(k=None), L.P4Q_ERR_INVALID_ARG),
    (dict(v=ALIGNED + 8), L.P4Q_ERR_INVALID_ARG),
    (dict(o=ALIGNED + 2), L.P4Q_ERR_INVALID_ARG),
    (dict(dt=4), L.P4Q_ERR_UNSUPPORTED),
])
def test_attention_validation(kw, status):
    assert attn(**kw) == status
    assert L.lib().p4q_last_error() != b""


def linear(**kw):
    a = dict(M=4, N=8, K=64, a=ALIGNED, sa=ALIGNED, w=ALIGNED, sw=ALIGNED, dt=1, y=ALIGNED,
             ldy=8, acc=None, ws=None, ws_bytes=0)
    a.update(kw)
    return L.lib().p4q_w4a4_linear(a["M"], a["N"], a["K"], a["a"], a["sa"], a["w"], a["sw"],
                                   a["dt"], a["y"], a["ldy"], a["acc"], a["ws"], a["ws_bytes"],
                                   None)


@pytest.mark.parametrize("kw,status", [
    (dict(M=0), L.P4Q_ERR_INVALID_ARG),
    (dict(N=-1), L.P4Q_ERR_INVALID_ARG),
    (dict(K=40), L.P4Q_ERR_INVALID_ARG),
    (dict(K=131072 + 32), L.P4Q_ERR_UNSUPPORTED),
    (dict(ldy=4), L.P4Q_ERR_INVALID_ARG),
    (dict(a=None), L.P4Q_ERR_INVALID_ARG),
    (dict(w=ALIGNED + 1), L.P4Q_ERR_INVALID_ARG),
    (dict(y=ALIGNED + 2), L.P4Q_ERR_INVALID_ARG),
    (dict(dt=5), L.P4Q_ERR_UNSUPPORTED),
])
def test_linear_validation(kw, status):
    assert linear(**kw) == status


def qscaled(**kw):
    a = dict(dt=0, R=4, K=64, z=ALIGNED, ldz=64, sigma=ALIGNED, divide=1, clip=1.0, clip_rows=None,
             codes=ALIGNED, scales=ALIGNED, absmax=None, kstar=None)
    a.update(kw)
    return L.lib().p4q_quant_scaled(a["dt"], a["R"], a["K"], a["z"], a["ldz"], a["sigma"],
                                    a["divide"], ctypes.c_float(a["clip"]), a["clip_rows"],
                                    a["codes"], a["scales"], a["absmax"], a["kstar"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(R=0), L.P4Q_ERR_INVALID_ARG),
    (dict(K=48), L.P4Q_ERR_INVALID_ARG),
    (dict(K=16384 + 32, ldz=16384 + 32), L.P4Q_ERR_UNSUPPORTED),
    (dict(ldz=60), L.P4Q_ERR_INVALID_ARG),
    (dict(ldz=68), L.P4Q_ERR_INVALID_ARG),
    (dict(divide=2), L.P4Q_ERR_INVALID_ARG),
    (dict(clip=0.0), L.P4Q_ERR_INVALID_ARG),
    (dict(clip=1.5), L.P4Q_ERR_INVALID_ARG),
    (dict(sigma=None), L.P4Q_ERR_INVALID_ARG),
    (dict(sigma=ALIGNED + 4), L.P4Q_ERR_INVALID_ARG),
    (dict(codes=ALIGNED + 8), L.P4Q_ERR_INVALID_ARG),
    (dict(dt=3), L.P4Q_ERR_UNSUPPORTED),
])
def test_quant_scaled_validation(kw, status):
    assert qscaled(**kw) == status
    assert L.lib().p4q_last_error() != b""


def calib(**kw):
    a = dict(dt=0, M=8, N=64, K=128, x=ALIGNED, ldx=128, w=ALIGNED, ldw=128, t=ALIGNED, ldt=64,
             sigma=ALIGNED, clip_a=1.0, clip_w=ALIGNED, loss=ALIGNED, gs=ALIGNED, gca=ALIGNED,
             gcw=ALIGNED, ws=ALIGNED, ws_bytes=1 << 30)
    a.update(kw)
    return L.lib().p4q_calib_linear_grad(a["dt"], a["M"], a["N"], a["K"], a["x"], a["ldx"],
                                         a["w"], a["ldw"], a["t"], a["ldt"], a["sigma"],
                                         ctypes.c_float(a["clip_a"]), a["clip_w"], a["loss"],
                                         a["gs"], a["gca"], a["gcw"], a["ws"], a["ws_bytes"],
                                         None)


@pytest.mark.parametrize("kw,status", [
    (dict(M=0), L.P4Q_ERR_INVALID_ARG),
    (dict(N=96), L.P4Q_ERR_INVALID_ARG),
    (dict(K=192, ldx=192, ldw=192), L.P4Q_ERR_INVALID_ARG),
    (dict(K=16384 + 128, ldx=16384 + 128, ldw=16384 + 128), L.P4Q_ERR_UNSUPPORTED),
    (dict(ldx=120), L.P4Q_ERR_INVALID_ARG),
    (dict(ldw=132), L.P4Q_ERR_INVALID_ARG),
    (dict(ldt=62), L.P4Q_ERR_INVALID_ARG),
    (dict(clip_a=0.0), L.P4Q_ERR_INVALID_ARG),
    (dict(clip_a=1.01), L.P4Q_ERR_INVALID_ARG),
    (dict(clip_w=None), L.P4Q_ERR_INVALID_ARG),
    (dict(t=ALIGNED + 4), L.P4Q_ERR_INVALID_ARG),
    (dict(ws=ALIGNED + 16), L.P4Q_ERR_INVALID_ARG),
    (dict(ws=None), L.P4Q_ERR_WORKSPACE),
    (dict(ws_bytes=1024), L.P4Q_ERR_WORKSPACE),
    (dict(dt=2), L.P4Q_ERR_UNSUPPORTED),
])
def test_calib_validation(kw, status):
    assert calib(**kw) == status
    assert L.lib().p4q_last_error() != b""


def test_calib_workspace_size():
    f = L.lib().p4q_calib_linear_workspace_bytes
    assert f(8, 96, 128) == 0 and f(0, 64, 128) == 0
    small, big = f(384, 12288, 4096), f(385, 12288, 4096)
    # at least codes, transposed bf16 codes, acc and the two bf16 operands
    assert small >= 384 * 12288 * (4 + 2 + 2) + 4096 * (384 + 12288) * 2
    assert big > small


def test_binding_refuses_cpu_tensors():
    import torch
    import paper_2609_34867_amd as p4q
    with pytest.raises(ValueError):
        p4q.quant_act(torch.zeros(4, 64, dtype=torch.float16))


INT_MAX = 2 ** 31 - 1


@pytest.mark.parametrize("args", [(INT_MAX, INT_MAX, INT_MAX, INT_MAX), (1, 1, 32, INT_MAX),
                                  (INT_MAX, 8192, 16384, 8), (INT_MAX, 8192, 8192, 8),
                                  (1, INT_MAX, 32, 1),
                                  (-1, 5, 32, 1), (1, 5, 32, -3)])
def test_select_workspace_size_extremes(args):
    """Sizes outside the documented limits give 0 (the call would reject
    them), and no size computation overflows (checked under the
    sanitizers)."""
    n = L.lib().p4q_select_workspace_bytes(*args)
    B, N, d, J = args
    if B >= 1 and 1 <= N <= 8192 and 32 <= d <= 16384 and 1 <= J <= 8 and not (J > 4 and d > 8192):
        assert n >= B * N * (J + 1) * 4
    else:
        assert n == 0


@pytest.mark.parametrize("args", [(INT_MAX, INT_MAX, INT_MAX, INT_MAX, INT_MAX),
                                  (1, 8192, 8192, 8, INT_MAX), (1, 100, 64, 2, 200)])
def test_select_full_workspace_size_extremes(args):
    n = L.lib().p4q_select_full_workspace_bytes(*args)
    B, N, d, J, K = args
    if K > N or N > 8192 or d > 8192 or J > 8:
        assert n == 0
    else:
        assert n >= B * N * N * 4


@pytest.mark.parametrize("args", [(INT_MAX, INT_MAX, 131072), (INT_MAX, 1, 32), (1, INT_MAX, 32),
                                  (512, 4096, 2 ** 30), (384, 4096, 4096), (-5, 10, 32)])
def test_linear_workspace_size_extremes(args):
    M, N, K = args
    n = L.lib().p4q_w4a4_linear_workspace_bytes(M, N, K)
    if (M, N, K) == (384, 4096, 4096):
        assert n > 0                          # split-K at batch 1
    if M <= 0 or K > 131072:
        assert n == 0


@pytest.mark.parametrize("args", [(INT_MAX, INT_MAX, INT_MAX), (INT_MAX, 64, 128),
                                  (384, 12288, 16384), (384, 12288, 2 ** 30)])
def test_calib_workspace_size_extremes(args):
    n = L.lib().p4q_calib_linear_workspace_bytes(*args)
    M, N, K = args
    if K > 16384 or M * N >= 2 ** 31 or N * K >= 2 ** 31:
        assert n == 0
    else:
        assert n > 0


def test_long_error_message_is_truncated():
    """An error message longer than the per-thread buffer is cut, not
    overflowed (checked under the sanitizers)."""
    st = L.lib().p4q_quant_act(0, -123456789, -987654321, None, -1, F(float("nan")), None, None,
                               None)
    assert st == L.P4Q_ERR_INVALID_ARG
    assert 0 < len(L.lib().p4q_last_error()) < 512
