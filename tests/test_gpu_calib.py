"""GPU parity of the calibration mechanics against the oracle (O7).

* p4q_quant_scaled: codes, scales, row maxima and their lowest indices
  bit-exact (every step is a correctly rounded fp32 operation or an exact
  decision taken in the same fp32 precision on both sides).
* p4q_calib_linear_grad against the plain float64 definition
  (oracle.calib_linear, operands="fp64").  The quantizer outputs are
  bit-identical on both sides; the GPU then rounds the residual in fp32, the
  two backward contraction operands to bf16 and accumulates in fp32.  The
  oracle propagates exactly those roundings, in magnitude, through the
  backward pass (bounds=True) and every component must lie within that
  bound, plus 2^-24 relative for the fp32 store of the result.  The bound is
  a worst case; the measured error is reported as a fraction of it.
* As a diagnostic of the arithmetic alone, the GPU is also compared with
  the oracle's bf16-operand mode, which rounds the same operands the same
  way: there only fp32 summation order differs, so components agree to
  |gpu - ref| <= 1e-3 |ref| + 2e-4 max|ref| and the loss to 1e-5."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34867_amd as p4q
from workload import calib_problem, random_features
from gpu_util import first_mismatch, to_gpu, to_np

pytestmark = pytest.mark.gpu


def sigma_vec(seed, K):
    g = np.random.default_rng(seed)
    return np.exp(0.4 * g.standard_normal(K)).astype(np.float32)


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("K", [32, 160, 4096, 11008, 16384])
@pytest.mark.parametrize("divide", [True, False])
def test_quant_scaled(dtype, K, divide):
    R = 19
    z = random_features(60 + K % 97, R, K, dtype)
    z[3] = 0
    sig = sigma_vec(K, K)
    clip_rows = np.random.default_rng(K).uniform(0.5, 1.0, R).astype(np.float32)
    for clip, rows in ((1.0, None), (0.8, None), (1.0, clip_rows)):
        codes, s, a, ks = p4q.quant_scaled(to_gpu(z, dtype), to_gpu(sig), divide, clip,
                                           None if rows is None else to_gpu(rows))
        torch.cuda.synchronize()
        rc, rs, ra, rk, _ = oracle.quant_rows_scaled(z, sig, divide,
                                                     clip if rows is None else rows, dtype)
        assert (m := first_mismatch(to_np(codes), oracle.pack_int4(rc))) is None, f"codes: {m}"
        assert (m := first_mismatch(to_np(s), rs)) is None, f"scales: {m}"
        assert (m := first_mismatch(to_np(a), ra)) is None, f"absmax: {m}"
        assert (m := first_mismatch(to_np(ks).astype(np.int64), rk)) is None, f"kstar: {m}"


def test_quant_scaled_ties_and_stride():
    K = 256
    z = np.zeros((4, K + 64), dtype=np.float16)
    z[0, [200, 7, 100]] = [5.0, -5.0, 5.0]          # three equal maxima -> 7
    z[1, :K] = random_features(61, 1, K)[0]
    z[2, [K - 1, 0]] = [-2.0, 2.0]                  # first and last
    sig = np.ones(K, dtype=np.float32)
    zt = to_gpu(z)[:, :K]
    codes, s, a, ks = p4q.quant_scaled(zt, to_gpu(sig), True, 1.0)
    torch.cuda.synchronize()
    rc, rs, ra, rk, _ = oracle.quant_rows_scaled(z[:, :K], sig, True, 1.0, "fp16")
    assert to_np(ks).tolist() == rk.tolist() and rk[0] == 7 and rk[2] == 0
    assert np.array_equal(to_np(codes), oracle.pack_int4(rc))
    assert np.array_equal(to_np(s), rs) and np.array_equal(to_np(a), ra)


def run_calib(p):
    x, w = to_gpu(p.x, p.dtype), to_gpu(p.w, p.dtype)
    out = p4q.calib_linear_grad(x, w, to_gpu(p.target), to_gpu(p.sigma), p.clip_a,
                                to_gpu(p.clip_w))
    torch.cuda.synchronize()
    return [to_np(t).astype(np.float64) for t in out]


def compare(p, got):
    """The GPU step against the float64 definition, within the oracle's
    propagated bound (see the module docstring), then the bf16-operand
    diagnostic.  Returns the float64 reference."""
    ref = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, p.dtype, "fp64",
                              bounds=True)
    loss, gs, gca, gcw = got
    store = 2.0 ** -24                                   # fp32 store of each result
    worst = 0.0
    for name, g, r, b in (("loss", loss, np.array([ref["loss"]]), np.array([ref["bound_loss"]])),
                          ("grad_sigma", gs, ref["grad_sigma"], ref["bound_grad_sigma"]),
                          ("grad_clip_a", gca, np.array([ref["grad_clip_a"]]),
                           np.array([ref["bound_grad_clip_a"]])),
                          ("grad_clip_w", gcw, ref["grad_clip_w"], ref["bound_grad_clip_w"])):
        tol = b + store * np.abs(r)
        err = np.abs(g - r)
        bad = err > tol
        assert not bad.any(), (f"{name} vs float64: {bad.sum()} off, first {np.argwhere(bad)[0]}: "
                               f"{g[bad][:3]} vs {r[bad][:3]} (bound {tol[bad][:3]})")
        nz = tol > 0
        if nz.any():
            worst = max(worst, float(np.max(err[nz] / tol[nz])))
    print(f"calibration {p.x.shape[0]}x{p.w.shape[0]}x{p.x.shape[1]}: largest error "
          f"{worst:.3f} of the propagated bound")
    diag = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, p.dtype, "bf16")
    assert loss[0] == pytest.approx(diag["loss"], rel=1e-5)
    for name, g, r in (("grad_sigma", gs, diag["grad_sigma"]), ("grad_clip_w", gcw, diag["grad_clip_w"])):
        tol = 1e-3 * np.abs(r) + 2e-4 * np.abs(r).max()
        bad = np.abs(g - r) > tol
        assert not bad.any(), (f"{name} vs bf16 operands: {bad.sum()} off, first "
                               f"{np.argwhere(bad)[0]}: {g[bad][:3]} vs {r[bad][:3]}")
    assert gca[0] == pytest.approx(diag["grad_clip_a"], rel=1e-3,
                                   abs=1e-6 * abs(diag["grad_clip_a"]))
    return ref


@pytest.mark.parametrize("dtype,M,N,K,clip_a", [
    ("fp16", 1, 64, 128, 1.0),          # one token
    ("fp16", 37, 128, 256, 0.9),        # ragged M inside one tile
    ("bf16", 200, 192, 384, 0.7),       # ragged M over two tiles, 3 k-tiles
    ("fp16", 300, 320, 512, 1.0),
])
def test_calib_small(dtype, M, N, K, clip_a):
    p = calib_problem(M + N + K, M, N, K, dtype, clip_a=clip_a)
    compare(p, run_calib(p))


def test_calib_zero_rows_and_repeat():
    p = calib_problem(71, 96, 128, 256, "fp16")
    p.x[5] = 0
    p.w[17] = 0
    got = run_calib(p)
    ref = compare(p, got)
    assert got[3][17] == 0.0 and ref["grad_clip_w"][17] == 0.0
    again = run_calib(p)          # fp64 scatter order aside, the same fp32 results
    for a, b in zip(got, again):
        assert np.allclose(a, b, rtol=1e-6, atol=0)


def test_calib_split_contraction():
    """Enough tiles that neither backward product splits (M = 512, N = 1024,
    K = 1024), against a shape whose act-side product splits its
    contraction over several work-groups (small M, long N)."""
    for M, N, K in ((512, 1024, 1024), (64, 4096, 256)):
        p = calib_problem(M * 7 + N, M, N, K, "bf16", clip_a=0.85)
        compare(p, run_calib(p))


def test_calib_llava_next_qkv():
    """The calibration step at the measured size: LLaVA-NeXT-7B q/k/v (fused,
    N = 12288, K = 4096) on one pruned calibration sample (M = 320 + 64)."""
    p = calib_problem(72, 384, 12288, 4096, "fp16", clip_a=0.9)
    compare(p, run_calib(p))


def test_calib_llava_next_down_proj_bf16():
    """down_proj's shape (K = 11008 inputs, 86 channel tiles) in bf16, on the
    same pruned calibration sample."""
    p = calib_problem(73, 384, 4096, 11008, "bf16", clip_a=0.8)
    compare(p, run_calib(p))


def test_calib_workspace_reuse_across_shapes():
    """One workspace sized for the larger problem serves a smaller one; the
    second call's results do not depend on what the first left behind."""
    big = calib_problem(74, 256, 512, 1024, "fp16")
    small = calib_problem(75, 40, 128, 256, "fp16")
    ws = p4q.calib_linear_workspace(256, 512, 1024, torch.device("cuda:0"))
    for p in (big, small):
        out = p4q.calib_linear_grad(to_gpu(p.x), to_gpu(p.w), to_gpu(p.target), to_gpu(p.sigma),
                                    p.clip_a, to_gpu(p.clip_w), workspace=ws)
        torch.cuda.synchronize()
        compare(p, [to_np(t).astype(np.float64) for t in out])


def test_calib_heavy_clamping():
    """Small clipping factors (most values saturate: the clamp's gradient
    mask and the code range edges -8 / 7 dominate) on both sides."""
    p = calib_problem(76, 130, 192, 512, "fp16", clip_a=0.2)
    p.clip_w = np.random.default_rng(76).uniform(0.1, 0.3, 192).astype(np.float32)
    ref = compare(p, run_calib(p))
    # the activations' outlier channels set their row maxima, so fewer of
    # their values saturate than the weights'
    assert np.mean(np.abs(ref["a_codes"]) >= 7) > 0.02 and np.mean(np.abs(ref["w_codes"]) >= 7) > 0.3
