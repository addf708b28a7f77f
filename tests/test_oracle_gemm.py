"""Pins for the oracle's W4A4 linear (O4): integer GEMM on int4 codes and the
dequant epilogue (W4A4 setting of Appendix A / B.3)."""
import numpy as np
import pytest
import torch

import oracle
from workload import random_features


def _triple_loop(a, w):
    M, K = a.shape
    N = w.shape[0]
    out = [[0] * N for _ in range(M)]
    for m in range(M):
        for n in range(N):
            acc = 0
            for k in range(K):
                acc += int(a[m, k]) * int(w[n, k])
            out[m][n] = acc
    return np.array(out, dtype=np.int64)


@pytest.mark.parametrize("shape", [(3, 5, 8), (7, 4, 32), (1, 9, 64)])
def test_int_gemm_equals_triple_loop(shape):
    M, N, K = shape
    rng = np.random.default_rng(M * 100 + N)
    a = rng.integers(-8, 8, size=(M, K)).astype(np.int8)
    w = rng.integers(-8, 8, size=(N, K)).astype(np.int8)
    assert np.array_equal(oracle.int_gemm(a, w), _triple_loop(a, w))


def test_int_gemm_extremes_exact():
    """Worst-case magnitudes (all -8) at K = 13824: acc = 64*K exactly."""
    K = 13824
    a = np.full((2, K), -8, dtype=np.int8)
    w = np.full((3, K), -8, dtype=np.int8)
    w[1] = 7
    acc = oracle.int_gemm(a, w)
    assert acc[0, 0] == 64 * K and acc[1, 1] == -56 * K
    assert abs(int(acc.max())) < 2 ** 24


def test_int_gemm_identity_closed_form():
    rng = np.random.default_rng(9)
    a = rng.integers(-8, 8, size=(6, 16)).astype(np.int8)
    eye = np.eye(16, dtype=np.int8)
    assert np.array_equal(oracle.int_gemm(a, eye), a.astype(np.int64))
    ones = np.ones((1, 16), dtype=np.int8)
    assert np.array_equal(oracle.int_gemm(a, ones)[:, 0], a.astype(np.int64).sum(1))


def test_packed_linear_matches_unpacked():
    rng = np.random.default_rng(11)
    a = rng.integers(-8, 8, size=(5, 64)).astype(np.int8)
    w = rng.integers(-8, 8, size=(7, 64)).astype(np.int8)
    sa = rng.uniform(0.1, 2, size=5).astype(np.float32)
    sw = rng.uniform(0.001, 0.01, size=7).astype(np.float32)
    acc, y = oracle.w4a4_linear(oracle.pack_int4(a), sa, oracle.pack_int4(w), sw, "fp16")
    assert np.array_equal(acc, _triple_loop(a, w))
    for m in range(5):
        for n in range(7):
            acc1, y1 = oracle.w4a4_linear_entry(oracle.pack_int4(a), sa, oracle.pack_int4(w),
                                                sw, m, n, "fp16")
            assert acc1 == acc[m, n] and y1 == y[m, n]


@pytest.mark.parametrize("out_dtype", ["fp16", "bf16"])
def test_epilogue_rounding_matches_torch(out_dtype):
    """The epilogue's two fp32 products and final RNE, against torch CPU ops
    (torch's own float32 multiply and dtype conversion)."""
    rng = np.random.default_rng(13)
    # ~1e6 outputs: a reordered epilogue changes the rounded result only
    # about once per 1e4 elements, so the sample must be large
    acc = rng.integers(-200000, 200000, size=(1024, 1000)).astype(np.int64)
    sa = rng.uniform(1e-3, 5, size=1024).astype(np.float32)
    sw = rng.uniform(1e-4, 1e-2, size=1000).astype(np.float32)
    y = oracle.epilogue(acc, sa, sw, out_dtype)
    t = torch.from_numpy(acc).to(torch.float32) * torch.from_numpy(sa)[:, None]
    t = t * torch.from_numpy(sw)[None, :]
    tdt = torch.float16 if out_dtype == "fp16" else torch.bfloat16
    ref = t.to(tdt).view(torch.int16).numpy().view(np.uint16)
    got = y.view(np.uint16)
    assert np.array_equal(got, ref)


def test_bf16_rne_ties_and_overflow():
    vals = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 3.3895e38, 1e-40],
                    dtype=np.float32)
    got = oracle.f32_to_bf16_rne(vals)
    ref = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref)
    assert got[0] == 0x3F80 and got[1] == 0x3F82      # ties to even


def test_w4a4_approximates_float_linear():
    """y = s_a s_w acc approximates x @ w^T within the per-element rounding
    bound |x - s c| <= s/2 (clip 1): catches transposed operands or a
    misplaced scale."""
    x = random_features(31, 12, 256)
    w = random_features(32, 10, 256, outliers=0, std=0.02)
    ap, sa = oracle.quant_act(x)
    wp, sw = oracle.quant_act(w)
    acc, y = oracle.w4a4_linear(ap, sa, wp, sw, "fp16")
    exact = sa.astype(np.float64)[:, None] * sw.astype(np.float64)[None, :] * acc
    ref = x.astype(np.float64) @ w.astype(np.float64).T
    bound = (np.abs(x.astype(np.float64)).sum(1)[:, None] * sw[None, :] / 2
             + np.abs(w.astype(np.float64)).sum(1)[None, :] * sa[:, None] / 2
             + 256 * sa[:, None] * sw[None, :] / 4)
    assert np.all(np.abs(exact - ref) <= bound * (1 + 1e-9))
    # and the rounded output stays within fp16 rounding of the exact product
    rel = np.abs(y.astype(np.float64) - exact) / np.maximum(np.abs(exact), 1e-30)
    assert np.all((rel <= 2 ** -10) | (np.abs(exact) < 6e-5))
