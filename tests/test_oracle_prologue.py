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


def plain_codes_exact(x, g, dtype, clip):
    """Codes of the plain definition Q4(RMSNorm(x) * gamma) in exact real
    arithmetic, together with the exact quotients q_k = v_k / s, where
    v = RMSNorm(x) * gamma and s = clip max|v| / 7.  The row factor 1/rms
    cancels, so q_k = 7 u_k / (clip a) with u = x * gamma and a = max|u|.

    Everything is exact in float64: u_k is a product of two 16-bit floats (at
    most 22 significant bits), 14 u_k has at most 26, clip * a at most 46 and
    (2n + 1) clip a at most 50, so the side of the half-integer n + 1/2 on
    which q_k lies is the exact sign of 14 u_k - (2n + 1) clip a (ties to
    even when it is zero)."""
    u = oracle.as_f32(x, dtype).astype(np.float64) * oracle.as_f32(g, dtype).astype(np.float64)[None, :]
    a = np.max(np.abs(u), axis=1, keepdims=True)
    c = float(np.float32(clip))
    ca = c * a
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.where(ca > 0, 7.0 * u / np.where(ca > 0, ca, 1.0), 0.0)
    n0 = np.floor(q)
    d = 14.0 * u - (2.0 * n0 + 1.0) * ca
    up = (d > 0) | ((d == 0) & (np.mod(n0, 2) != 0))
    codes = np.clip(n0 + up, -8, 7).astype(np.int8)
    codes[(ca == 0)[:, 0]] = 0
    return codes, q


@pytest.mark.parametrize("dtype,clip,seed", [("fp16", 1.0, 1), ("fp16", 0.7, 2), ("bf16", 1.0, 3),
                                             ("bf16", 0.55, 4)])
def test_fused_codes_equal_the_plain_definition_except_at_near_ties(dtype, clip, seed):
    """The oracle (and the kernel) quantize u = x * gamma in fp32 and put
    1/rms into the scale.  Against the plain definition -- Q4 of the real
    RMSNorm(x) * gamma -- the fused fp32 quotient fl32(u / fl32(fl32(c a) / 7))
    is within 3 fp32 roundings, 3 * 2^-24 * |q| <= 1.5 * 2^-21 < 2^-20 for
    |q| <= 8, of the exact quotient, so a code can differ only where the
    exact quotient lies within 2^-20 of a half-integer.  Rows include exact
    ties (x = 2.5 with max 7 at gamma 1).  The count of differing codes is
    printed: 0 of 2^21 at clip 1 (where fl32(1 * a) is exact), 3 and 1 of
    2^21 at clips 0.7 and 0.55, each at a quotient within 2^-20 of a
    half-integer."""
    rng = np.random.default_rng(seed)
    M, d = 512, 4096
    x = random_features(100 + seed, M, d, dtype)
    g = (1.0 + 0.1 * rng.standard_normal(d)).astype(np.float32)
    g = g.astype(np.float16) if dtype == "fp16" else oracle.f32_to_bf16_rne(g)
    # exact ties: gamma 1 on channels 0..3, row max 7, values n + 1/2
    one = np.float16(1.0) if dtype == "fp16" else np.uint16(0x3F80)
    g[:4] = one
    tie = np.array([7.0, 2.5, -3.5, 0.5], dtype=np.float32)
    for r in range(8):
        row = np.zeros(d, dtype=np.float32)
        row[:4] = tie
        row[4:] = rng.uniform(-1, 1, d - 4)
        x[r] = row.astype(np.float16) if dtype == "fp16" else oracle.f32_to_bf16_rne(row)
    fused, _ = oracle.rmsnorm_quant(x, g, 1e-5, dtype, clip)
    fused = oracle.unpack_int4(fused)
    plain, q = plain_codes_exact(x, g, dtype, clip)
    if clip == 1.0:
        assert np.array_equal(plain[:8, :4], np.array([[7, 2, -4, 0]] * 8))   # ties to even
    diff = fused != plain
    near = np.abs(q - (np.floor(q) + 0.5)) <= 2.0 ** -20
    assert not np.any(diff & ~near), "a code differs away from a near-tie"
    print(f"{dtype} clip {clip}: {int(diff.sum())} of {diff.size} codes differ from the plain "
          f"definition, {int(near.sum())} quotients within 2^-20 of a half-integer")
    assert int(diff.sum()) <= int(near.sum())


def test_plain_definition_pin_detects_planted_mistakes():
    """The exact-definition codes are not a copy of the fused path: fused
    codes computed with gamma dropped, or applied twice, differ from them on
    ordinary (non-tie) values, so the pin above would catch either mistake."""
    rng = np.random.default_rng(9)
    x = random_features(7, 64, 1024, "fp16")
    g = (1.0 + 0.1 * rng.standard_normal(1024)).astype(np.float16)
    plain, q = plain_codes_exact(x, g, "fp16", 1.0)
    near = np.abs(q - (np.floor(q) + 0.5)) <= 2.0 ** -20
    ones = np.ones(1024, dtype=np.float16)
    for wrong_g in (ones, (g.astype(np.float32) ** 2).astype(np.float16)):
        wrong = oracle.unpack_int4(oracle.rmsnorm_quant(x, wrong_g, 1e-5, "fp16", 1.0)[0])
        assert np.any((wrong != plain) & ~near)
