"""Pins for the oracle's fused decoder prologue (O5: per-token Q4 of
RMSNorm(x) * gamma, scale carrying 1/rms).

Each check is independent of the oracle's own code path: a hand-derived
worked example, the plain quantizer (gamma = 1), exact power-of-two
invariances, and the reconstruction bound against a float64 RMSNorm
computed directly."""
import os

import numpy as np
import pytest

import oracle
from workload import random_features

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "rmsnorm_quant_worked_example.txt")


def load_golden():
    meta, rows, cur = {}, [], {}
    for line in open(GOLDEN):
        line = line.split("#", 1)[0].split()
        if not line:
            if cur:
                rows.append(cur)
                cur = {}
            continue
        if line[0] in ("dtype", "eps", "clip"):
            meta[line[0]] = line[1]
        else:
            cur[line[0]] = [float(v) for v in line[1:]]
    if cur:
        rows.append(cur)
    return meta, rows


def test_worked_example():
    meta, rows = load_golden()
    for r in rows:
        x = np.array([r["x"]], dtype=np.float16)
        g = np.array(r["gamma"], dtype=np.float16)
        packed, scales = oracle.rmsnorm_quant(x, g, float(meta["eps"]), meta["dtype"],
                                              float(meta["clip"]))
        codes = oracle.unpack_int4(packed)[0]
        assert codes.tolist() == [int(c) for c in r["codes"]]
        assert scales[0] == pytest.approx(r["scale"][0], rel=1e-6, abs=0)


@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
def test_unit_gamma_is_the_plain_quantizer(dtype):
    x = random_features(31, 40, 256, dtype)
    one = np.ones(256, np.float16) if dtype == "fp16" else np.full(256, 0x3F80, np.uint16)
    packed, _ = oracle.rmsnorm_quant(x, one, 1e-5, dtype)
    ref_packed, _ = oracle.quant_act(x, dtype)
    assert np.array_equal(packed, ref_packed)


def test_power_of_two_invariances():
    x = random_features(32, 24, 128)
    g = random_features(33, 1, 128, outliers=0)[0]
    p0, s0 = oracle.rmsnorm_quant(x, g, 0.0)
    # gamma * 4: same codes, scale * 4 exactly
    p1, s1 = oracle.rmsnorm_quant(x, (g.astype(np.float32) * 4).astype(np.float16), 0.0)
    assert np.array_equal(p0, p1) and np.array_equal(s1, s0 * np.float32(4))
    # x * 8 (eps = 0): same codes, same scale
    p2, s2 = oracle.rmsnorm_quant((x.astype(np.float32) * 8).astype(np.float16), g, 0.0)
    assert np.array_equal(p0, p2) and np.array_equal(s0, s2)


def test_reconstruction_bound_against_float64_rmsnorm():
    x = random_features(34, 64, 512)
    g = random_features(35, 1, 512, outliers=0, std=0.5)[0]
    eps = 1e-6
    packed, scales = oracle.rmsnorm_quant(x, g, eps)
    codes = oracle.unpack_int4(packed).astype(np.float64)
    xf = x.astype(np.float64)
    y = xf / np.sqrt(np.mean(xf * xf, axis=1, keepdims=True) + eps) * g.astype(np.float64)
    err = np.abs(y - codes * scales.astype(np.float64)[:, None])
    assert np.all(err <= scales[:, None] * (0.5 + 1e-5))
    # every row uses the full range (clip 1: a code of magnitude 7 per row)
    assert np.all(np.max(np.abs(codes), axis=1) == 7)


def test_zero_row_and_negative_gamma():
    x = random_features(36, 4, 64)
    x[2] = 0
    g = -np.abs(random_features(37, 1, 64, outliers=0)[0])
    packed, scales = oracle.rmsnorm_quant(x, g, 1e-5)
    codes = oracle.unpack_int4(packed)
    assert scales[2] == 0 and np.all(codes[2] == 0)
    # eps = 0: a zero row still has scale 0 (not 0 * inf)
    _, s0 = oracle.rmsnorm_quant(x, g, 0.0)
    assert s0[2] == 0 and np.all(np.isfinite(s0))
    # negating gamma negates every code (no -8 at clip 1)
    p2, s2 = oracle.rmsnorm_quant(x, (-g.astype(np.float32)).astype(np.float16), 1e-5)
    assert np.array_equal(oracle.unpack_int4(p2), -codes) and np.array_equal(s2, scales)
