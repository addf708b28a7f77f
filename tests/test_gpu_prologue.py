"""GPU parity of p4q_rmsnorm_quant (per-token int4 of RMSNorm(x) * gamma)
against the oracle: codes bit-exact; scales within 1e-5 relative (the GPU sums
x^2 in fp32 in its own order)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34867_amd as p4q
from workload import CONFIGS, random_features, selector_inputs
from gpu_util import Guarded, check_canaries, first_mismatch, to_gpu, to_np

pytestmark = pytest.mark.gpu


def gamma_row(seed, d, dtype):
    g = random_features(seed, 1, d, "fp16", outliers=4, scale=6.0, std=0.3)[0].astype(np.float32)
    g = np.where(np.abs(g) < 1e-3, np.float32(0.5), g)
    if dtype == "fp16":
        return g.astype(np.float16)
    u = g.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def check(x, g, dtype="fp16", eps=1e-5, clip=1.0, ldx=None, rows=None):
    M, d = x.shape
    xs = x
    if ldx is not None and ldx > d:
        pad = np.zeros((M, ldx), dtype=x.dtype)
        pad[:, :d] = x
        xs = pad
    xt = to_gpu(xs, dtype)[:, :d]
    gt = to_gpu(g, dtype)
    gc, gs = Guarded((M, d // 2), torch.uint8, "codes"), Guarded((M,), torch.float32, "scales")
    codes, scales = p4q.rmsnorm_quant(xt, gt, eps, clip, codes=gc.t, scales=gs.t)
    torch.cuda.synchronize()
    check_canaries(gc, gs)
    codes, scales = to_np(codes), to_np(scales)
    sel = np.arange(M) if rows is None else np.asarray(rows)
    rc, rs = oracle.rmsnorm_quant(x[sel], g, eps, dtype, clip)
    assert (m := first_mismatch(codes[sel], rc)) is None, f"codes: {m}"
    ok = np.isclose(scales[sel], rs, rtol=1e-5, atol=0)
    assert ok.all(), f"scales: {np.argwhere(~ok)[:3].ravel()} {scales[sel][~ok][:3]} vs {rs[~ok][:3]}"


@pytest.mark.parametrize("d", [32, 256, 4096, 5120, 16384])
def test_widths(d):
    x = random_features(41, 37, d)
    check(x, gamma_row(42, d, "fp16"))


def test_bf16_clip_strided_zero_rows():
    x = random_features(43, 300, 2048, "bf16")
    x[[0, 17, 299]] = 0
    g = gamma_row(44, 2048, "bf16")
    check(x, g, "bf16")
    check(x, g, "bf16", clip=0.6)
    check(x, g, "bf16", eps=0.0, ldx=2048 + 64)


def test_negative_and_unit_gamma():
    x = random_features(45, 64, 1024)
    check(x, (-gamma_row(46, 1024, "fp16").astype(np.float32)).astype(np.float16))
    check(x, np.ones(1024, np.float16))


def test_near_tie_rows():
    """With max |u| = 7 the step is exactly 1, so u = k + 1/2 lands on
    rounding ties (ties to even): the exact fall-back decides."""
    d = 512
    rng = np.random.default_rng(47)
    k = rng.integers(-7, 7, size=(16, d)).astype(np.float32)
    x = (k + 0.5).astype(np.float16)
    x[:, 0] = 7
    check(x, np.ones(d, np.float16))
    check(x, np.full(d, 2.0, np.float16))


def test_llava_next_b16_pruned_sequence_sampled():
    """The bench shape: M = 11264 rows of d = 4096; 256 sampled rows."""
    cfg = CONFIGS["next7b_b16"]
    si = selector_inputs(cfg, samples=[0, 1])
    x = np.concatenate([si.vis.reshape(-1, cfg.d)] * 2)[:cfg.M]
    g = gamma_row(48, cfg.d, "fp16")
    rows = np.random.default_rng(49).choice(cfg.M, 256, replace=False)
    check(x, g, rows=np.sort(rows))
