"""Pins for the oracle's calibration mechanics (O7: reconstruction loss of a
W4A4 fake-quantized linear on a pruned sequence and its gradients with respect
to the diagonal channel scales and the clipping factors).

None of these checks re-types the oracle's backward formulas:
* a hand-derived worked example (tests/golden/calib_worked_example.txt);
* torch autograd, float64, through a forward written with torch ops
  (rounding passed straight through by the detach trick);
* central finite differences of a surrogate forward in which every rounding
  decision is frozen at the evaluation point -- the function whose exact
  derivative the straight-through gradient is;
* the invariance of the product under sigma -> lambda sigma, which forces
  sum_k sigma_k dL/dsigma_k = 0 (both sides of the transform must agree);
* closed forms on the quantization grid, and degenerate rows."""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from workload import calib_problem, random_features

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "calib_worked_example.txt")


def load_golden():
    vals = {}
    for line in open(GOLDEN):
        line = line.split("#", 1)[0].split()
        if line:
            vals[line[0]] = line[1:]
    return vals


def test_worked_example():
    g = load_golden()
    x = np.array([[float(v) for v in g["x"]]], dtype=np.float16)
    w = np.array([[float(v) for v in g["w"]]], dtype=np.float16)
    sigma = np.array([float(v) for v in g["sigma"]], dtype=np.float32)
    out = oracle.calib_linear(x, w, np.array([[float(g["target"][0])]], np.float32), sigma,
                              float(g["clip_a"][0]), np.array([float(g["clip_w"][0])]),
                              g["dtype"][0])
    assert out["a_codes"][0].tolist() == [int(v) for v in g["a_codes"]]
    assert out["w_codes"][0].tolist() == [int(v) for v in g["w_codes"]]
    frac = lambda s: float(Fraction(s))
    assert out["loss"] == pytest.approx(frac(g["loss"][0]), rel=1e-12)
    assert out["grad_clip_a"] == pytest.approx(frac(g["grad_clip_a"][0]), rel=1e-12)
    assert out["grad_clip_w"][0] == pytest.approx(frac(g["grad_clip_w"][0]), rel=1e-12)
    np.testing.assert_allclose(out["grad_sigma"], [frac(v) for v in g["grad_sigma"]],
                               rtol=1e-12)


def small_problem(seed, M=6, N=5, K=48, clip_a=0.8, clip_lo=0.6):
    p = calib_problem(seed, M, N, K, "fp16", clip_a=clip_a, w_std=0.05)
    rng = np.random.default_rng(seed)
    p.clip_w = rng.uniform(clip_lo, 1.0, N).astype(np.float32)
    return p


def torch_forward(p, sigma, clip_a, clip_w, frozen=None):
    """Loss through a forward written with torch ops (float64).

    frozen=None: straight-through rounding (value rne(u), gradient of u),
    clamp on the rounded value.  frozen=(q, inside, u0) per side: the surrogate
    s * (q + inside * (u - u0)) whose rounding decisions are fixed."""
    x = torch.tensor(oracle.as_f32(p.x, p.dtype), dtype=torch.float64)
    w = torch.tensor(oracle.as_f32(p.w, p.dtype), dtype=torch.float64)
    T = torch.tensor(p.target, dtype=torch.float64)

    def fq(z, c, fr):
        a = z.abs().max(dim=1).values
        s = c * a / 7
        u = z / s[:, None]
        if fr is None:
            q = torch.clamp(u + (torch.round(u) - u).detach(), -8, 7)
        else:
            q0, ins, u0 = fr
            q = q0 + ins * (u - u0)
        return q * s[:, None], u.detach()

    fx, ux = fq(x / sigma, clip_a.expand(x.shape[0]), None if frozen is None else frozen[0])
    fw, uw = fq(w * sigma, clip_w, None if frozen is None else frozen[1])
    y = fx @ fw.T
    M, N = y.shape
    return ((y - T) ** 2).sum() / (M * N), ux, uw


def params(p):
    return (torch.tensor(p.sigma, dtype=torch.float64, requires_grad=True),
            torch.tensor(p.clip_a, dtype=torch.float64, requires_grad=True),
            torch.tensor(p.clip_w, dtype=torch.float64, requires_grad=True))


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_autograd(seed):
    p = small_problem(seed)
    ref = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, p.dtype)
    sig, ca, cw = params(p)
    loss, _, _ = torch_forward(p, sig, ca, cw)
    loss.backward()
    assert ref["loss"] == pytest.approx(loss.item(), rel=1e-5)
    scale = np.abs(sig.grad.numpy()).max()
    np.testing.assert_allclose(ref["grad_sigma"], sig.grad.numpy(), rtol=1e-5, atol=1e-6 * scale)
    assert ref["grad_clip_a"] == pytest.approx(ca.grad.item(), rel=1e-5, abs=1e-9)
    np.testing.assert_allclose(ref["grad_clip_w"], cw.grad.numpy(), rtol=1e-5,
                               atol=1e-6 * np.abs(cw.grad.numpy()).max())
    # the case exercises clamping (clip < 1) on both sides
    assert np.any(np.abs(ref["a_codes"]) == 8) or np.any(ref["a_codes"] == 7)


def frozen_state(p, sig, ca, cw):
    with torch.no_grad():
        _, ux, uw = torch_forward(p, sig, ca, cw)
    out = []
    for u in (ux, uw):
        r = torch.round(u)
        ins = ((r >= -8) & (r <= 7)).double()
        out.append((torch.clamp(r, -8, 7), ins, u.clone()))
    return out


@pytest.mark.parametrize("seed", [4, 5])
def test_finite_differences(seed):
    p = small_problem(seed)
    ref = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, p.dtype)
    sig0, ca0, cw0 = params(p)
    fr = frozen_state(p, sig0, ca0, cw0)

    def F(sig, ca, cw):
        with torch.no_grad():
            return torch_forward(p, sig, ca, cw, frozen=fr)[0].item()

    h = 1e-6
    # sigma: an activation outlier channel (an argmax column), two ordinary ones
    ks = [int(ref["a_kstar"][0]), 0, p.sigma.shape[0] - 1]
    for k in ks:
        e = torch.zeros_like(sig0)
        e[k] = h * sig0[k]
        fd = (F(sig0 + e, ca0, cw0) - F(sig0 - e, ca0, cw0)) / (2 * e[k].item())
        assert ref["grad_sigma"][k] == pytest.approx(fd, rel=1e-4, abs=1e-7 * abs(ref["loss"]))
    d = h * ca0.item()
    fd = (F(sig0, ca0 + d, cw0) - F(sig0, ca0 - d, cw0)) / (2 * d)
    assert ref["grad_clip_a"] == pytest.approx(fd, rel=1e-4, abs=1e-7 * abs(ref["loss"]))
    for n in (0, p.clip_w.shape[0] - 1):
        e = torch.zeros_like(cw0)
        e[n] = h * cw0[n]
        fd = (F(sig0, ca0, cw0 + e) - F(sig0, ca0, cw0 - e)) / (2 * e[n].item())
        assert ref["grad_clip_w"][n] == pytest.approx(fd, rel=1e-4, abs=1e-7 * abs(ref["loss"]))


@pytest.mark.parametrize("seed,M,N,K", [(6, 16, 24, 128), (7, 33, 17, 256)])
def test_scale_invariance(seed, M, N, K):
    p = calib_problem(seed, M, N, K, "fp16")
    ref = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, p.dtype)
    t = p.sigma.astype(np.float64) * ref["grad_sigma"]
    # exact in real arithmetic; the fp32 transformed rows and scales leave
    # a residue of a few fp32 ulps of the terms
    assert abs(t.sum()) <= 1e-6 * np.abs(t).sum()
    assert np.abs(t).sum() > 0


def test_power_of_two_sigma_is_exact():
    """sigma = 2^e on every channel scales each row exactly: the codes are
    the plain quantizer's and the scales move by 2^-e (divide) / 2^e."""
    x = random_features(11, 7, 64, "fp16")
    codes, scales = oracle.quantize_rows(x, "fp16", 0.9)
    for e, divide in ((3, True), (-2, True), (4, False)):
        sig = np.full(64, 2.0 ** e, dtype=np.float32)
        c, s, a, ks, _ = oracle.quant_rows_scaled(x, sig, divide, 0.9, "fp16")
        f = 2.0 ** (-e if divide else e)
        assert np.array_equal(c, codes)
        assert np.array_equal(s, (scales * f).astype(np.float32))
        mag = np.abs(x.astype(np.float32))
        assert np.array_equal(a, (mag.max(axis=1) * f).astype(np.float32))
        assert ks.tolist() == [int(np.argmax(r)) for r in mag]


def test_kstar_takes_lowest_tie():
    x = np.zeros((2, 8), dtype=np.float16)
    x[0, [5, 2]] = [3.0, -3.0]
    x[1, [7, 6]] = [-1.5, 1.5]
    _, _, a, ks, _ = oracle.quant_rows_scaled(x, np.ones(8, np.float32), True, 1.0, "fp16")
    assert ks.tolist() == [2, 6] and a.tolist() == [3.0, 1.5]


def grid_rows(rng, R, K, e):
    """Rows s * integers with max |code| = 7 exactly and s = 2^e: Q4 at clip 1
    reproduces them exactly."""
    c = rng.integers(-7, 8, (R, K))
    c[:, 0] = 7
    return (c * 2.0 ** e).astype(np.float16)


def test_grid_closed_form():
    rng = np.random.default_rng(8)
    x = grid_rows(rng, 5, 32, -3)
    w = grid_rows(rng, 4, 32, -5)
    xf, wf = x.astype(np.float64), w.astype(np.float64)
    E = rng.standard_normal((5, 4)).astype(np.float32) * np.float32(0.25)
    T = (xf @ wf.T + E).astype(np.float32)
    one = np.ones(32, np.float32)
    ref = oracle.calib_linear(x, w, T, one, 1.0, np.ones(4, np.float32), "fp16")
    assert np.array_equal(ref["a_codes"].astype(np.float64) * 2.0 ** -3, xf)
    R = xf @ wf.T - T.astype(np.float64)
    assert ref["loss"] == pytest.approx(np.mean(R * R), rel=1e-12)
    exact = oracle.calib_linear(x, w, (xf @ wf.T).astype(np.float32), one, 1.0,
                                np.ones(4, np.float32), "fp16")
    assert exact["loss"] == 0.0
    assert not np.any(exact["grad_sigma"]) and exact["grad_clip_a"] == 0.0
    assert not np.any(exact["grad_clip_w"])


def test_zero_rows():
    p = calib_problem(9, 6, 5, 64, "fp16")
    p.x[2] = 0
    p.w[3] = 0
    ref = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, p.dtype)
    assert ref["a_scales"][2] == 0 and not np.any(ref["a_codes"][2])
    assert ref["w_scales"][3] == 0 and ref["grad_clip_w"][3] == 0.0
    assert np.all(np.isfinite(ref["grad_sigma"]))


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_bf16_operands_close(dtype):
    """Rounding the two contraction operands to bf16 perturbs each product
    by < 2^-8 relative; the gradients stay within a few 2^-8 of the float64
    ones, measured against the largest component."""
    p = calib_problem(10, 24, 32, 256, dtype)
    a = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, dtype, "fp64")
    b = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, dtype, "bf16")
    assert np.array_equal(a["a_codes"], b["a_codes"])
    assert b["loss"] == pytest.approx(a["loss"], rel=1e-5)
    for key in ("grad_sigma", "grad_clip_w"):
        ref = np.abs(a[key]).max()
        assert np.abs(a[key] - b[key]).max() <= 2 ** -6 * ref
    assert b["grad_clip_a"] == pytest.approx(a["grad_clip_a"], rel=2 ** -6)


@pytest.mark.parametrize("dtype,M,N,K,clip_a", [("fp16", 40, 64, 256, 0.9),
                                                ("bf16", 96, 192, 512, 0.7),
                                                ("fp16", 130, 128, 1024, 1.0)])
def test_bound_covers_rounded_operands(dtype, M, N, K, clip_a):
    """The propagated bound around the float64 result (bounds=True) covers
    an evaluation that rounds the contraction operands to bf16 (the oracle's
    bf16-operand mode, computed independently of the bound), and it is not
    vacuous: it stays a small fraction of each component's own magnitude
    scale (the operand rounding is 2^-8 relative)."""
    p = calib_problem(M * 3 + N + K, M, N, K, dtype, clip_a=clip_a)
    r64 = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, dtype, "fp64",
                              bounds=True)
    r16 = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, dtype, "bf16")
    for key in ("grad_sigma", "grad_clip_w", "grad_clip_a", "loss"):
        err = np.abs(np.asarray(r16[key]) - np.asarray(r64[key]))
        assert np.all(err <= np.asarray(r64["bound_" + key])), key
    # not vacuous: for most components the bound is well below the value
    # itself (sigma's components are differences of larger activation- and
    # weight-side sums, so their bound is the larger fraction)
    rel = lambda k: np.median(r64["bound_" + k] / np.maximum(np.abs(r64[k]), 1e-30))
    assert rel("grad_clip_w") < 0.25 and rel("grad_sigma") < 0.6
    assert r64["bound_loss"] < 1e-2 * r64["loss"]


def test_bound_fails_for_a_wrong_gradient():
    """A planted mistake (the weight-side argmax share dropped) moves the
    gradient by far more than the propagated bound, so a GPU step carrying
    that mistake could not pass the float64 comparison."""
    p = calib_problem(5, 48, 64, 256, "fp16", clip_a=0.9)
    r64 = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, "fp16", "fp64",
                              bounds=True)
    orig = oracle.p4q_oracle.fq_row_backward

    def dropped(zp, s, clip, codes, absmax, kstar, g, absolute=False):
        dz, dc = orig(zp, s, clip, codes, absmax, kstar, g, absolute)
        if not absolute and zp.shape[0] == p.w.shape[1] and s != 0:
            dz = g * (np.abs(np.rint(zp / np.float32(s))) <= 8)
        return dz, dc
    oracle.p4q_oracle.fq_row_backward = dropped
    try:
        bad = oracle.calib_linear(p.x, p.w, p.target, p.sigma, p.clip_a, p.clip_w, "fp16", "fp64")
    finally:
        oracle.p4q_oracle.fq_row_backward = orig
    err = np.abs(bad["grad_sigma"] - r64["grad_sigma"])
    assert np.any(err > r64["bound_grad_sigma"])
