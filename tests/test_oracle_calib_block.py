"""Pins for the oracle's block-level calibration (O8: a decoder block's
W4A4 fake-quantized forward, block-output MSE and the gradients for every
linear group's diagonal scales and clipping factors).

Each pin is independent of the oracle's code path:
* torch float64 autograd through a forward written here with torch ops
  (straight-through rounding by the detach trick for the quantizer codes and
  for every 16-bit intermediate), against every gradient;
* central finite differences of a surrogate forward whose rounding
  decisions (codes, clamp masks, 16-bit roundings) are frozen at the
  evaluation point -- the function whose exact derivative the
  straight-through gradient is;
* scale invariance per linear group (X W^T is unchanged when sigma is
  multiplied by a constant, so sum_k sigma_k dL/dsigma_k = 0);
* zero loss and zero gradients when the target is the block's own output;
* planted mistakes in the chain rule fail the autograd pin."""
import numpy as np
import pytest
import torch

import oracle
from oracle import p4q_oracle as O
from workload import calib_block_problem

GROUPS = oracle.BLOCK_GROUPS


def problem(seed, M=24, d=256, f=384, H=2):
    p = calib_block_problem(seed, M, d, f, H)
    fp = oracle.calib_block(p.x, p.weights, p.gamma1, p.gamma2, p.H, quantize=False)
    target = oracle.as_f32(fp["out"], p.dtype).astype(np.float32)
    return p, target


def torch_block(p, target, sigma, clip_a, clip_w, frozen=None, record=None, eps=1e-5):
    """The block's loss written with torch ops in float64.  frozen=None:
    straight-through rounding; with `record` (a list) the rounding decisions
    are appended in order; frozen (such a list): every rounding replaced by
    its frozen decision (codes and masks fixed, 16-bit roundings as fixed
    offsets), a smooth surrogate of the loss."""
    t = lambda a: torch.tensor(oracle.as_f32(a, p.dtype), dtype=torch.float64)
    X, g1, g2 = t(p.x), t(p.gamma1), t(p.gamma2)
    W = {k: t(v) for k, v in p.weights.items()}
    it = iter(frozen) if frozen is not None else None

    def r16(v):
        if it is not None:
            return v + next(it)
        off = (v.detach().to(torch.float16).to(torch.float64) - v.detach())
        if record is not None:
            record.append(off)
        return v + off

    def st(v64, v32):
        """value of the fp32 computation, gradient of the real one; in the
        frozen surrogate the real value alone (a smooth function with the
        same derivative)"""
        if it is not None:
            return v64
        return v64 + (v32.double() - v64).detach()

    def fq(z, z32, c):
        """Q4 rows of z (values: the fp32 transformed rows z32, fp32 scale
        and fp32 quotient, as the quantizer defines them); returns the codes
        (straight-through) and the scales."""
        a32 = z32.abs().max(dim=1).values
        s32 = (c.detach().float() * a32) / 7.0
        s = st(c * z.abs().max(dim=1).values / 7, s32)
        u = st(z, z32) / s[:, None]
        if it is not None:
            q0, ins, u0 = next(it)
            q = q0 + ins * (u - u0)
        else:
            r = torch.round(z32 / s32[:, None]).double()
            if record is not None:
                record.append((torch.clamp(r, -8, 7), ((r >= -8) & (r <= 7)).double(),
                               u.detach().clone()))
            q = torch.clamp(u + (r - u).detach(), -8, 7)
        return q, s, s32

    def lin(name, A):
        sg = sigma[name]
        qa, sa, sa32 = fq(A / sg, (A.float() / sg.detach().float()),
                          clip_a[name].expand(A.shape[0]))
        qw, sw, sw32 = fq(W[name] * sg, (W[name].float() * sg.detach().float()), clip_w[name])
        y = (qa * sa[:, None]) @ (qw * sw[:, None]).T
        acc = (qa.detach() @ qw.detach().T).float()
        y32 = (acc * sa32[:, None]) * sw32[None, :]           # the W4A4 epilogue in fp32
        return r16(st(y, y32))

    def rms(x, g):
        return x * torch.rsqrt((x * x).mean(dim=1, keepdim=True) + eps) * g

    M, d = X.shape
    H = p.H
    D = d // H
    n1 = r16(rms(X, g1))
    qkv = lin("qkv", n1)
    i = torch.arange(D // 2, dtype=torch.float64)
    ang = torch.arange(M, dtype=torch.float64)[:, None] * (10000.0 ** (-2 * i / D))[None, :]
    c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]

    def rope(z):
        a, b = z[..., :D // 2], z[..., D // 2:]
        return torch.cat([a * c - b * s, b * c + a * s], dim=-1)
    q = r16(rope(qkv[:, :d].reshape(M, H, D)))
    k = r16(rope(qkv[:, d:2 * d].reshape(M, H, D)))
    v = qkv[:, 2 * d:].reshape(M, H, D)
    S = torch.einsum("mhd,nhd->hmn", q, k) / D ** 0.5
    mask = torch.tril(torch.ones(M, M, dtype=torch.bool))
    S = S.masked_fill(~mask, float("-inf"))
    P = torch.softmax(S, dim=-1)
    O_ = r16(torch.einsum("hmn,nhd->mhd", P, v).reshape(M, d))
    h = r16(X + lin("o", O_))
    n2 = r16(rms(h, g2))
    gu = lin("gu", n2)
    f = gu.shape[1] // 2
    a = r16(torch.nn.functional.silu(gu[:, :f]) * gu[:, f:])
    out = r16(h + lin("down", a))
    T = torch.tensor(target, dtype=torch.float64)
    return ((out - T) ** 2).sum() / (M * d)


def params(p):
    sig = {k: torch.tensor(p.sigma[k], dtype=torch.float64, requires_grad=True) for k in GROUPS}
    ca = {k: torch.tensor(np.float32(p.clip_a[k]), dtype=torch.float64, requires_grad=True)
          for k in GROUPS}
    cw = {k: torch.tensor(p.clip_w[k], dtype=torch.float64, requires_grad=True) for k in GROUPS}
    return sig, ca, cw


def run_oracle(p, target):
    return oracle.calib_block(p.x, p.weights, p.gamma1, p.gamma2, p.H, target, p.sigma, p.clip_a,
                              p.clip_w)


def check_against_autograd(ref, p, target):
    sig, ca, cw = params(p)
    loss = torch_block(p, target, sig, ca, cw)
    loss.backward()
    # Both sides evaluate the same roundings in float64, in different orders
    # (softmax, SiLU, sums): a 16-bit intermediate that sits on a rounding
    # tie can come out one unit apart and flip a downstream code, which
    # moves a few components by ~1e-4 of the largest; every planted mistake
    # below moves them by far more than the 2e-3 allowed here.
    assert ref["loss"] == pytest.approx(loss.item(), rel=1e-5)
    for g in GROUPS:
        gs = sig[g].grad.numpy()
        np.testing.assert_allclose(ref["grad_sigma"][g], gs, rtol=2e-3,
                                   atol=2e-3 * np.abs(gs).max(), err_msg=f"sigma {g}")
        gw = cw[g].grad.numpy()
        np.testing.assert_allclose(ref["grad_clip_w"][g], gw, rtol=2e-3,
                                   atol=2e-3 * np.abs(gw).max(), err_msg=f"clip_w {g}")
        assert ref["grad_clip_a"][g] == pytest.approx(ca[g].grad.item(), rel=2e-3), g


@pytest.mark.parametrize("seed", [1, 2])
def test_autograd(seed):
    p, target = problem(seed)
    ref = run_oracle(p, target)
    assert ref["loss"] > 0
    check_against_autograd(ref, p, target)


def test_autograd_two_heads_longer_sequence():
    p, target = problem(3, M=70, d=256, f=256, H=2)
    check_against_autograd(run_oracle(p, target), p, target)


def test_finite_differences():
    p, target = problem(4)
    ref = run_oracle(p, target)
    sig0, ca0, cw0 = params(p)
    rec = []
    with torch.no_grad():
        torch_block(p, target, sig0, ca0, cw0, record=rec)

    def F(sig, ca, cw):
        with torch.no_grad():
            return torch_block(p, target, sig, ca, cw, frozen=rec).item()

    hrel = 1e-6
    for g in GROUPS:
        n_in = p.sigma[g].shape[0]
        for kk in (0, n_in // 3, n_in - 1):
            e = {k: v.detach().clone() for k, v in sig0.items()}
            em = {k: v.detach().clone() for k, v in sig0.items()}
            dd = hrel * float(sig0[g][kk].detach())
            e[g][kk] += dd
            em[g][kk] -= dd
            fd = (F(e, ca0, cw0) - F(em, ca0, cw0)) / (2 * dd)
            assert ref["grad_sigma"][g][kk] == pytest.approx(fd, rel=2e-4, abs=1e-6 * ref["loss"]), \
                (g, kk)
        dd = hrel * float(ca0[g].detach())
        up = {k: v.detach().clone() for k, v in ca0.items()}
        dn = {k: v.detach().clone() for k, v in ca0.items()}
        up[g] += dd
        dn[g] -= dd
        fd = (F(sig0, up, cw0) - F(sig0, dn, cw0)) / (2 * dd)
        assert ref["grad_clip_a"][g] == pytest.approx(fd, rel=2e-4, abs=1e-6 * ref["loss"]), g
        n = p.clip_w[g].shape[0] // 2
        up = {k: v.detach().clone() for k, v in cw0.items()}
        dn = {k: v.detach().clone() for k, v in cw0.items()}
        dd = hrel * float(cw0[g][n].detach())
        up[g][n] += dd
        dn[g][n] -= dd
        fd = (F(sig0, ca0, up) - F(sig0, ca0, dn)) / (2 * dd)
        assert ref["grad_clip_w"][g][n] == pytest.approx(fd, rel=2e-4, abs=1e-6 * ref["loss"]), g


def test_scale_invariance_per_group():
    p, target = problem(5)
    ref = run_oracle(p, target)
    for g in GROUPS:
        t = p.sigma[g].astype(np.float64) * ref["grad_sigma"][g]
        assert abs(t.sum()) <= 1e-5 * np.abs(t).sum(), g


def test_zero_residual():
    p, _ = problem(6)
    own = oracle.calib_block(p.x, p.weights, p.gamma1, p.gamma2, p.H, None, p.sigma, p.clip_a,
                             p.clip_w)
    target = oracle.as_f32(own["out"], p.dtype).astype(np.float32)
    ref = run_oracle(p, target)
    assert ref["loss"] == 0.0
    for g in GROUPS:
        assert not np.any(ref["grad_sigma"][g]) and not np.any(ref["grad_clip_w"][g])
        assert ref["grad_clip_a"][g] == 0.0


def test_full_precision_block_matches_torch():
    """The unquantized block (the calibration target) against the same block
    in torch float64 with the 16-bit roundings applied at the same points."""
    p, target = problem(7)
    t = lambda a: torch.tensor(oracle.as_f32(a, p.dtype), dtype=torch.float64)
    r16 = lambda v: v.to(torch.float16).to(torch.float64)
    X, g1, g2 = t(p.x), t(p.gamma1), t(p.gamma2)
    W = {k: t(v) for k, v in p.weights.items()}
    M, d = X.shape
    D = d // p.H
    rms = lambda x, g: x * torch.rsqrt((x * x).mean(dim=1, keepdim=True) + 1e-5) * g
    qkv = r16(r16(rms(X, g1)) @ W["qkv"].T)
    i = torch.arange(D // 2, dtype=torch.float64)
    ang = torch.arange(M, dtype=torch.float64)[:, None] * (10000.0 ** (-2 * i / D))[None, :]
    c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
    rope = lambda z: torch.cat([z[..., :D // 2] * c - z[..., D // 2:] * s,
                                z[..., D // 2:] * c + z[..., :D // 2] * s], dim=-1)
    q = r16(rope(qkv[:, :d].reshape(M, p.H, D))).transpose(0, 1)
    k = r16(rope(qkv[:, d:2 * d].reshape(M, p.H, D))).transpose(0, 1)
    v = qkv[:, 2 * d:].reshape(M, p.H, D).transpose(0, 1)
    O_ = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True)
    O_ = r16(O_.transpose(0, 1).reshape(M, d))
    h = r16(X + r16(O_ @ W["o"].T))
    gu = r16(r16(rms(h, g2)) @ W["gu"].T)
    f = gu.shape[1] // 2
    a = r16(torch.nn.functional.silu(gu[:, :f]) * gu[:, f:])
    out = r16(h + r16(a @ W["down"].T))
    got = oracle.as_f32(oracle.calib_block(p.x, p.weights, p.gamma1, p.gamma2, p.H,
                                           quantize=False)["out"], p.dtype)
    # identical up to ties of the 16-bit roundings (float64 evaluation order),
    # whose one-unit differences propagate through the residual stream
    ref = out.numpy().astype(np.float32)
    assert np.mean(got == ref) > 0.99
    np.testing.assert_allclose(got, ref, rtol=2.0 ** -8, atol=2.0 ** -12 * np.abs(ref).max())


@pytest.mark.parametrize("mistake", ["rope_not_inverted", "rmsnorm_first_term_only",
                                     "silu_derivative", "attention_no_centering",
                                     "attention_dk_transposed", "dx_not_divided_by_sigma"])
def test_planted_mistakes_fail_the_autograd_pin(mistake, monkeypatch):
    p, target = problem(8)
    if mistake == "rope_not_inverted":
        orig = O._rope
        monkeypatch.setattr(O, "_rope", lambda z, c, s, inverse=False: orig(z, c, s, False))
    elif mistake == "rmsnorm_first_term_only":
        monkeypatch.setattr(O, "_rmsnorm_backward",
                            lambda x, g, r, dn: r[:, None] * g[None, :] * dn)
    elif mistake == "silu_derivative":          # dSiLU/dg taken as sig(g) only
        def wrong(g, u, da):
            sg = 1.0 / (1.0 + np.exp(-g))
            return da * u * sg, da * g * sg
        monkeypatch.setattr(O, "_silu_mul_backward", wrong)
    elif mistake == "attention_no_centering":   # dS = P dP, the row sum dropped
        def wrong(q, k, v, P, dO):
            M, H, D = q.shape
            dq, dk, dv = (np.empty((M, H, D)) for _ in range(3))
            for hh in range(H):
                dv[:, hh, :] = P[hh].T @ dO[:, hh, :]
                dS = P[hh] * (dO[:, hh, :] @ v[:, hh, :].T)
                dq[:, hh, :] = dS @ k[:, hh, :] / np.sqrt(D)
                dk[:, hh, :] = dS.T @ q[:, hh, :] / np.sqrt(D)
            return dq, dk, dv
        monkeypatch.setattr(O, "_attention_backward", wrong)
    elif mistake == "attention_dk_transposed":  # dk = dS q instead of dS^T q
        orig = O._attention_backward

        def wrong(q, k, v, P, dO):
            dq, dk, dv = orig(q, k, v, P, dO)
            M, H, D = q.shape
            for hh in range(H):
                dP = dO[:, hh, :] @ v[:, hh, :].T
                dS = P[hh] * (dP - np.sum(P[hh] * dP, axis=1, keepdims=True))
                dk[:, hh, :] = dS @ q[:, hh, :] / np.sqrt(D)
            return dq, dk, dv
        monkeypatch.setattr(O, "_attention_backward", wrong)
    elif mistake == "dx_not_divided_by_sigma":
        orig_back = O._fq_linear_backward

        def no_div(q, G):
            dX, ds, dca, dcw = orig_back(q, G)
            return dX * q["sigma"].astype(np.float64)[None, :] ** 2, ds, dca, dcw
        monkeypatch.setattr(O, "_fq_linear_backward", no_div)
    ref = run_oracle(p, target)
    monkeypatch.undo()
    with pytest.raises(AssertionError):
        check_against_autograd(ref, p, target)
