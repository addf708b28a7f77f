"""GPU parity of p4q_quant_act (fused per-row int4 quantize + pack) against
the oracle: packed codes and fp32 scales must match bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34867_amd as p4q
from workload import CONFIGS, random_features, mlp_standin, attn_standin, f32_to_bf16_bits
from gpu_util import Guarded, check_canaries, first_mismatch, to_gpu, to_np

pytestmark = pytest.mark.gpu


def check(x, dtype, clip=1.0, ldx=None):
    M, K = x.shape
    if ldx is not None and ldx > K:                      # strided rows
        wide = np.zeros((M, ldx), dtype=x.dtype)
        wide[:, :K] = x
        xt = to_gpu(wide, dtype)[:, :K]
    else:
        xt = to_gpu(x, dtype)
    gc, gs = Guarded((M, K // 2), torch.uint8, "codes"), Guarded((M,), torch.float32, "scales")
    codes, scales = p4q.quant_act(xt, clip, codes=gc.t, scales=gs.t)
    torch.cuda.synchronize()
    check_canaries(gc, gs)
    ref_codes, ref_scales = oracle.quant_act(x, dtype, clip)
    got_c, got_s = to_np(codes), to_np(scales)
    assert (m := first_mismatch(got_s.view(np.uint32), ref_scales.view(np.uint32))) is None, m
    assert (m := first_mismatch(got_c, ref_codes)) is None, m


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("K", [32, 96, 512, 4096, 5120, 11008, 13824, 16384, 20480])
def test_shapes(dtype, K):
    M = 67 if K <= 16384 else 9                          # ragged block of 4 rows
    check(random_features(K, M, K, dtype), dtype)


@pytest.mark.parametrize("clip", [0.9, 0.5, 2.0 ** -16])
@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_clip(clip, dtype):
    check(random_features(3, 33, 4096, dtype), dtype, clip)


def test_strided_rows():
    check(random_features(4, 21, 1024), "fp16", ldx=1048)


def test_adversarial_rows():
    d = 4096
    rows = []
    rows.append(np.zeros(d))                              # all zero -> scale 0
    r = np.zeros(d); r[17] = -3.0; rows.append(r)         # single nonzero
    rows.append(np.full(d, 2.5))                          # all equal
    r = np.zeros(d); r[:] = 65504.0; r[1::2] = -65504.0; rows.append(r)  # fp16 max
    rng = np.random.default_rng(0)
    for a in (61.4375, 1.6630859375, 95.8125, 91.375, 7.0):  # quotients on .5 boundaries
        r = np.zeros(d)
        r[0] = a
        k = rng.integers(-6, 6, size=d - 1) + 0.5
        s = np.float32(np.float32(a) / np.float32(7))
        r[1:] = (k * s).astype(np.float16)
        rows.append(r)
    r = rng.standard_normal(d) * 1e-6; rows.append(r)     # fp16 subnormal range
    x = np.stack(rows).astype(np.float16)
    check(x, "fp16")
    check(x, "fp16", 0.7)


def test_bf16_tiny_rows():
    """bf16 rows whose scale underflows to a subnormal take the exact path."""
    d = 512
    x = np.zeros((3, d), dtype=np.float32)
    x[0, :] = np.linspace(-1e-38, 1e-38, d)
    x[1, :] = np.linspace(-3e-39, 2e-39, d)
    x[2, :5] = [1e-40, -2e-40, 3e-40, 0, 5e-41]
    check(f32_to_bf16_bits(x), "bf16")


@pytest.mark.slow
def test_full_size_layer_inputs():
    """The two activation widths of a LLaVA-NeXT-7B decoder layer at batch 16
    (M = 11264): all rows of the o_proj input, sampled rows of the down_proj
    input, quantized by one launch each."""
    cfg = CONFIGS["next7b_b16"]
    x = attn_standin(cfg)
    check(x, "fp16")
    xm = mlp_standin(cfg)
    xt = to_gpu(xm)
    codes, scales = p4q.quant_act(xt)
    torch.cuda.synchronize()
    rows = np.r_[0:64, np.random.default_rng(1).integers(0, cfg.M, 192), cfg.M - 64:cfg.M]
    rc, rs = oracle.quant_act(xm[rows], "fp16")
    assert np.array_equal(to_np(scales)[rows].view(np.uint32), rs.view(np.uint32))
    assert np.array_equal(to_np(codes)[rows], rc)
