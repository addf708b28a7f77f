"""GPU parity of p4q_attention_prefill against the oracle (float64 softmax
attention).  Tolerance, from the arithmetic: the softmax weights are rounded
to the input dtype before the P V product (at most half an ulp each, so at
most 2^-11 (fp16) / 2^-8 (bf16) of max|v| in total), and both results are
rounded to that dtype (one ulp of |o| between them); the bound used is twice
that: |o - ref| <= 2^-10 max|v| + 2^-9 |ref| (fp16), 2^-7 max|v| + 2^-6 |ref|
(bf16)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34867_amd as p4q
from workload import random_features
from gpu_util import Guarded, check_canaries, to_gpu, to_np

pytestmark = pytest.mark.gpu
D = 128


def make_qkv(seed, B, L, H, dtype, std=1.0):
    """One fused [B*L, 3*H*D] q|k|v buffer, as the q|k|v projection writes it."""
    return random_features(seed, B * L, 3 * H * D, dtype, outliers=0, std=std)


def tol(dtype):
    return (2.0 ** -10, 2.0 ** -9) if dtype == "fp16" else (2.0 ** -7, 2.0 ** -6)


def check(qkv, B, L, H, causal=True, dtype="fp16", samples=None):
    t = to_gpu(qkv, dtype)
    HD = H * D
    go = Guarded((B * L, HD), t.dtype, "out")
    out = p4q.attention_prefill(t[:, :HD], t[:, HD:2 * HD], t[:, 2 * HD:], B, H, causal, out=go.t)
    torch.cuda.synchronize()
    check_canaries(go)
    got = oracle.as_f32(to_np(out), dtype).astype(np.float64).reshape(B, L, H, D)
    a, r = tol(dtype)
    for b in (range(B) if samples is None else samples):
        blk = qkv[b * L:(b + 1) * L].reshape(L, 3, H, D)
        ref = oracle.attention_prefill(blk[:, 0], blk[:, 1], blk[:, 2], causal, dtype)
        ref = oracle.as_f32(ref, dtype).astype(np.float64)
        vmax = np.abs(oracle.as_f32(blk[:, 2], dtype)).max(axis=(0, 2))          # per head
        err = np.abs(got[b] - ref)
        bound = a * vmax[None, :, None] + r * np.abs(ref)
        bad = np.argwhere(err > bound)
        assert bad.size == 0, (f"b={b}: {len(bad)} elements out of tolerance, first {tuple(bad[0])}: "
                               f"{got[b][tuple(bad[0])]} vs {ref[tuple(bad[0])]}")


@pytest.mark.parametrize("L", [1, 5, 32, 33, 127, 128, 129, 300])
def test_lengths_causal(L):
    check(make_qkv(61, 2, L, 3, "fp16"), 2, L, 3)


@pytest.mark.parametrize("L", [7, 200])
def test_non_causal(L):
    check(make_qkv(62, 1, L, 2, "fp16"), 1, L, 2, causal=False)


def test_bf16_and_large_logits():
    check(make_qkv(63, 1, 257, 2, "bf16", std=2.0), 1, 257, 2, dtype="bf16")
    check(make_qkv(64, 1, 160, 2, "fp16", std=3.0), 1, 160, 2)


def test_separate_buffers_and_strided_output():
    B, L, H = 2, 96, 2
    q, k, v = (to_gpu(random_features(65 + i, B * L, H * D, "fp16", outliers=0)) for i in range(3))
    out = torch.zeros((B * L, H * D + 64), dtype=torch.float16, device=q.device)
    p4q.attention_prefill(q, k, v, B, H, True, out=out[:, :H * D])
    torch.cuda.synchronize()
    assert torch.count_nonzero(out[:, H * D:]) == 0
    fused = np.concatenate([to_np(q), to_np(k), to_np(v)], axis=1)
    got = to_np(out[:, :H * D]).reshape(B, L, H, D).astype(np.float64)
    for b in range(B):
        blk = fused[b * L:(b + 1) * L].reshape(L, 3, H, D)
        ref = oracle.attention_prefill(blk[:, 0], blk[:, 1], blk[:, 2], True).astype(np.float64)
        assert np.all(np.abs(got[b] - ref) <= 2.0 ** -10 * 4 + 2.0 ** -9 * np.abs(ref))


def test_llava_next_b16_layer_sampled():
    """The bench shape: 16 samples x 704 tokens (640 kept + 64 text), 32 heads;
    first and last samples checked."""
    B, L, H = 16, 704, 32
    check(make_qkv(66, B, L, H, "fp16"), B, L, H, samples=[0, B - 1])
