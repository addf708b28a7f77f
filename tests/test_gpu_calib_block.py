"""GPU parity of the block-level calibration step (p4q_calib_block_grad)
against the oracle's float64 block (O8).

The two sides compute the same block with the same roundings but not the
same arithmetic: the GPU evaluates RMSNorm, RoPE, attention and SiLU in
fp32 (the oracle: float64), and each linear group's two backward
contractions take bf16 operands (8 significant bits) with fp32
accumulation.  Some gradient components are ill-conditioned with respect to
the first: a 16-bit intermediate on a rounding tie comes out one unit
apart, a row's largest value changes its index, and a row maximum's share
of a scale's gradient -- a large term that nearly cancels -- moves between
channels and down the chain.  On the LLaVA-NeXT block the oracle's own fp32
evaluation of those operations (fp32_ops=True, a probe of each component's
sensitivity, not the reference) moves 92 of the 12288 q|k|v weight-clip
gradients by more than the tight bound below; the GPU moves 94; rounding the
backward operands to bf16 alone moves none.

Per group and gradient vector, with sens = |fp32-evaluated - float64| from
the oracle and mag the sum of the magnitudes of a component's terms:
* every component: |gpu - ref| <= 2^-5 |ref| + 2^-6 max|ref| + 8 sens +
  share + 2^-8 mag, where share is the row-maximum share the component can
  receive from rows whose largest values lie within 2^-9 of each other and
  2^-8 mag the first-order bound of the bf16 operand rounding;
* all but a fraction 2^-9 of the components also without the 2^-8 mag term;
* the loss to 2^-10 relative, each activation clipping factor's gradient
  (a sum over all rows) to 2^-5 relative plus 8 sens.
A planted mistake in any derivative moves most components by O(1) of their
size (the oracle's pins), so it cannot pass; the measured errors are
printed."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34867_amd as p4q
from workload import calib_block_problem
from gpu_util import Guarded, check_canaries, to_gpu, to_np

pytestmark = pytest.mark.gpu

GROUPS = oracle.BLOCK_GROUPS
REL, ABS = 2.0 ** -5, 2.0 ** -6


def flat(p, key):
    return np.concatenate([np.asarray(getattr(p, key)[g], dtype=np.float32) for g in GROUPS])


def run(p, target):
    d = p.x.shape[1]
    f = p.weights["down"].shape[1]
    M = p.x.shape[0]
    outs = [Guarded((n,), torch.float32, name) for n, name in
            ((1, "loss"), (3 * d + f, "grad_sigma"), (4, "grad_clip_a"), (5 * d + 2 * f, "grad_clip_w"))]
    w = {k: to_gpu(v) for k, v in p.weights.items()}
    res = p4q.calib_block_grad(to_gpu(p.x), to_gpu(target), w["qkv"], w["o"], w["gu"], w["down"],
                               to_gpu(p.gamma1), to_gpu(p.gamma2), p.H, to_gpu(flat(p, "sigma")),
                               [p.clip_a[g] for g in GROUPS], to_gpu(flat(p, "clip_w")),
                               out=tuple(g.t for g in outs))
    torch.cuda.synchronize()
    check_canaries(*outs)
    return [to_np(t).astype(np.float64) for t in res]


def split(v, d, f, kind):
    sizes = {"sigma": (d, d, d, f), "clip_w": (3 * d, d, 2 * f, d)}[kind]
    out, o = {}, 0
    for g, n in zip(GROUPS, sizes):
        out[g] = v[o:o + n]
        o += n
    return out


def fragile_shares(st, sigma):
    """Per channel, the row-maximum shares of the scale's gradient that an
    evaluation can move to it: rows whose largest |X'| values lie within
    2^-9 of each other, each candidate channel of such a row getting the
    row's share |dL/dclip_row| clip_a / sigma_k."""
    a = np.abs(st["xp"].astype(np.float64))
    mx = a.max(axis=1, keepdims=True)
    cand = (a >= mx * (1.0 - 2.0 ** -9)) & (mx > 0)
    fragile = cand.sum(axis=1) > 1
    share = np.abs(st["a_dclip_rows"]) * float(st["clip_a"])
    out = (cand[fragile] * share[fragile, None]).sum(axis=0)
    return out / sigma.astype(np.float64)


def check(p, target, label):
    d = p.x.shape[1]
    f = p.weights["down"].shape[1]
    args = (p.x, p.weights, p.gamma1, p.gamma2, p.H, target, p.sigma, p.clip_a, p.clip_w)
    ref = oracle.calib_block(*args, bounds=True)
    r32 = oracle.calib_block(*args, fp32_ops=True)
    loss, gs, gca, gcw = run(p, target)
    worst, outliers = 0.0, 0
    assert loss[0] == pytest.approx(ref["loss"], rel=2.0 ** -10), label
    for kind, got in (("sigma", split(gs, d, f, "sigma")), ("clip_w", split(gcw, d, f, "clip_w"))):
        for g in GROUPS:
            r, mag = ref["grad_" + kind][g], ref["mag_grad_" + kind][g]
            sens = np.abs(r32["grad_" + kind][g] - r)
            share = fragile_shares(ref["state"][g], p.sigma[g]) if kind == "sigma" else 0.0
            tight = REL * np.abs(r) + ABS * np.abs(r).max() + 8.0 * sens + share
            err = np.abs(got[g] - r)
            off = err > tight
            loose = err > tight + 2.0 ** -8 * mag
            assert not loose.any(), (f"{label} {kind} {g}: {loose.sum()} of {r.size} beyond the worst-case "
                                     f"bound, first {np.argwhere(loose)[0]}: {got[g][loose][:3]} vs "
                                     f"{r[loose][:3]}")
            assert off.sum() <= max(1, r.size // 512), (
                f"{label} {kind} {g}: {off.sum()} of {r.size} beyond the tight bound, first "
                f"{np.argwhere(off)[0]}: {got[g][off][:3]} vs {r[off][:3]}")
            outliers += int(off.sum())
            worst = max(worst, float(np.median(err / (np.abs(r) + np.abs(r).max()))))
    for i, g in enumerate(GROUPS):
        r = ref["grad_clip_a"][g]
        sens = abs(r32["grad_clip_a"][g] - r)
        assert abs(gca[i] - r) <= REL * abs(r) + 8.0 * sens + 1e-30, (label, g, gca[i], r)
    print(f"{label}: loss {loss[0]:.6e} vs {ref['loss']:.6e}; median error {worst:.2e} of "
          f"(|ref| + max|ref|) in the worst vector; {outliers} components beyond the tight bound")


def target_of(p):
    fp = oracle.calib_block(p.x, p.weights, p.gamma1, p.gamma2, p.H, quantize=False)
    return oracle.as_f32(fp["out"], p.dtype).astype(np.float32)


@pytest.mark.parametrize("seed,M,d,f,H", [(1, 24, 256, 384, 2), (2, 130, 256, 256, 2),
                                          (3, 200, 512, 768, 4), (4, 64, 384, 640, 3)])
def test_block_small(seed, M, d, f, H):
    p = calib_block_problem(seed, M, d, f, H)
    check(p, target_of(p), f"block M={M} d={d} f={f} H={H}")


def test_block_repeat_is_stable():
    """Two calls on one workspace give the same results (the float64
    scatter order aside)."""
    p = calib_block_problem(5, 96, 256, 384, 2)
    t = target_of(p)
    a, b = run(p, t), run(p, t)
    for x, y in zip(a, b):
        assert np.allclose(x, y, rtol=1e-5, atol=1e-6 * np.abs(y).max())


@pytest.mark.slow
def test_block_llava_next_7b():
    """The measured shape: one LLaVA-NeXT-7B decoder block (d = 4096, f =
    11008, 32 heads) on one pruned calibration sample of 320 kept visual +
    64 text tokens."""
    p = calib_block_problem(6, 384, 4096, 11008, 32)
    check(p, target_of(p), "LLaVA-NeXT-7B block M=384")
