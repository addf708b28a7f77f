"""Pins for the oracle's attention prefill (O6): special cases with closed
forms, and the library routine torch.nn.functional.scaled_dot_product_attention
(float64, CPU) as an independent implementation of the same definition."""
import numpy as np
import pytest
import torch

import oracle
from workload import random_features


def qkv(seed, L, H, D, dtype="fp16", std=1.0):
    a = random_features(seed, 3 * L, H * D, dtype, outliers=0, std=std)
    return tuple(x.reshape(L, H, D) for x in np.split(a, 3))


def dec(a, dtype):
    return oracle.as_f32(a, dtype).astype(np.float64)


def test_first_token_sees_only_itself():
    q, k, v = qkv(51, 17, 2, 64)
    o = oracle.attention_prefill(q, k, v, causal=True)
    assert np.array_equal(o[0].view(np.uint16), v[0].view(np.uint16))


def test_equal_keys_give_running_means():
    q, k, v = qkv(52, 33, 2, 32)
    k[:] = k[0]                                  # every key identical: uniform weights
    o = oracle.attention_prefill(q, k, v, causal=True).astype(np.float64)
    vf = dec(v, "fp16")
    means = np.cumsum(vf, axis=0) / np.arange(1, 34)[:, None, None]
    assert np.allclose(o, means, rtol=0, atol=np.abs(means).max() * 2.0 ** -10)


def test_dominant_diagonal_copies_values():
    q, k, v = qkv(53, 40, 1, 64)
    k[:] = (q.astype(np.float32) * 8).astype(np.float16)   # <q_t, k_t> dominates
    o = oracle.attention_prefill(q, k, v, causal=False).astype(np.float64)
    assert np.allclose(o, dec(v, "fp16"), rtol=0, atol=1e-2)


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_matches_torch_sdpa_float64(causal, dtype):
    L, H, D = 45, 3, 128
    q, k, v = qkv(54, L, H, D, dtype, std=2.0)
    o = dec(oracle.attention_prefill(q, k, v, causal, dtype), dtype)
    t = lambda a: torch.from_numpy(dec(a, dtype)).permute(1, 0, 2)      # [H, L, D]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=causal)
    ref = ref.permute(1, 0, 2).numpy()
    ulp = 2.0 ** -10 if dtype == "fp16" else 2.0 ** -7
    assert np.all(np.abs(o - ref) <= np.abs(ref) * ulp + 1e-6)
