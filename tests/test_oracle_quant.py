"""Pins for the oracle's quantizer (O1) and nibble packing (O2).

Nothing here re-types the oracle's formula: the checks are a hand-computed
worked example (tests/golden), an exact-rational implementation of IEEE
binary32 rounding written from the standard's definition, and invariants that
the per-token symmetric RTN quantizer of the paper's W4A4 setting (Appendix A,
Appendix B.3) must satisfy.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from workload import random_features, f32_to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "quant_worked_example.txt")


# ---------------------------------------------------------------- exact fp32
def fl32(q: Fraction) -> Fraction:
    """Round an exact rational to the nearest binary32 value, ties to even
    (IEEE 754 roundTiesToEven; normals and subnormals; no overflow here)."""
    if q == 0:
        return Fraction(0)
    sign = -1 if q < 0 else 1
    a = abs(q)
    e = math.floor(math.log2(a.numerator) - math.log2(a.denominator))
    # fix the floor(log2) estimate exactly
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)                       # subnormal spacing floor
    ulp = Fraction(2) ** (e - 23)
    n = a / ulp
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return sign * fl * ulp


def rne(q: Fraction) -> int:
    fl = q.numerator // q.denominator
    rem = q - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return fl


def exact_quant_row(x_f32: np.ndarray, clip: float):
    xs = [Fraction(float(v)) for v in x_f32]
    a = max(abs(v) for v in xs)
    s = fl32(fl32(Fraction(float(np.float32(clip))) * a) / 7)
    if s == 0:
        return [0] * len(xs), s
    return [min(7, max(-8, rne(fl32(v / s)))) for v in xs], s


# ---------------------------------------------------------------- golden
def load_golden():
    cases, cur = [], {}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, *vals = line.split()
        if key == "dtype" and cur:
            cases.append(cur)
            cur = {}
        cur[key] = vals
    cases.append(cur)
    return cases


@pytest.mark.parametrize("case", load_golden(), ids=lambda c: "clip" + c["clip"][0])
def test_worked_example(case):
    x = np.array([float(v) for v in case["x"]], dtype=np.float16)[None]
    codes, scales = oracle.quantize_rows(x, "fp16", float(case["clip"][0]))
    assert codes[0].tolist() == [int(v) for v in case["codes"]]
    assert scales[0] == np.float32(float(case["scale"][0]))
    packed = oracle.pack_int4(codes)
    assert packed[0].tolist() == [int(v, 16) for v in case["packed"]]
    assert oracle.unpack_int4(packed)[0].tolist() == codes[0].tolist()


RECIP_TRAPS = [(61.4375, 30.71875), (1.6630859375, -0.83154296875), (95.8125, 20.53125),
               (91.375, -45.6875)]


@pytest.mark.parametrize("a,x", RECIP_TRAPS)
def test_division_not_reciprocal_multiply(a, x):
    """Rows where x * fl32(1/s) rounds to a different code than the correctly
    rounded x / s; the exact-rational reference decides."""
    row = np.array([[a, x]], dtype=np.float16)
    codes, scales = oracle.quantize_rows(row)
    ec, es = exact_quant_row(row[0].astype(np.float32), 1.0)
    assert codes[0].tolist() == ec
    r = np.float32(1) / scales[0]
    assert np.rint(np.float32(x) * r) != ec[1]


# ---------------------------------------------------------------- vs exact
@pytest.mark.parametrize("dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("clip", [1.0, 0.9, 0.37])
def test_quantizer_matches_exact_rationals(dtype, clip):
    x = random_features(7, 24, 64, dtype)
    codes, scales = oracle.quantize_rows(x, dtype, clip)
    xf = oracle.as_f32(x, dtype)
    for r in range(x.shape[0]):
        ec, es = exact_quant_row(xf[r], clip)
        assert Fraction(float(scales[r])) == es
        assert codes[r].tolist() == ec


def test_quantizer_near_half_quotients():
    """Rows built so that many quotients x/s land within a few ulps of a
    half-integer, where any rounding-order shortcut shows."""
    rng = np.random.default_rng(3)
    rows = []
    for t in range(40):
        a = np.float16(rng.uniform(0.5, 60.0))
        s = np.float32(np.float32(a) / np.float32(7))
        k = rng.integers(-6, 6, size=31) + 0.5
        vals = (k * s).astype(np.float16)
        rows.append(np.concatenate([[a], vals]).astype(np.float16))
    x = np.stack(rows)
    codes, scales = oracle.quantize_rows(x, "fp16", 1.0)
    for r in range(x.shape[0]):
        ec, es = exact_quant_row(x[r].astype(np.float32), 1.0)
        assert Fraction(float(scales[r])) == es
        assert codes[r].tolist() == ec


# ---------------------------------------------------------------- invariants
def test_code_range_and_extreme_code_clip1():
    x = random_features(11, 200, 256)
    codes, scales = oracle.quantize_rows(x, "fp16", 1.0)
    assert codes.min() >= -7 and codes.max() <= 7       # -8 never at clip 1
    assert np.all(np.max(np.abs(codes), axis=1) == 7)    # absmax element -> +-7


def test_minus8_appears_only_with_clipping():
    x = random_features(12, 64, 128)
    codes, _ = oracle.quantize_rows(x, "fp16", 0.5)
    assert codes.min() == -8 and codes.max() == 7


def test_roundtrip_error_bound():
    x = random_features(13, 64, 512)
    xf = x.astype(np.float64)
    codes, scales = oracle.quantize_rows(x, "fp16", 1.0)
    deq = oracle.dequantize_rows(codes, scales)
    err = np.abs(xf - deq)
    bound = scales.astype(np.float64)[:, None] * 0.5 * (1 + 2.0 ** -20)
    assert np.all(err <= bound)


def test_power_of_two_scale_invariance():
    x = random_features(14, 32, 128, std=0.5).astype(np.float32)
    base, s0 = oracle.quantize_rows(x.astype(np.float16), "fp16")
    for k in (-3, -1, 1, 2):
        xs = (x.astype(np.float16).astype(np.float32) * np.float32(2.0 ** k)).astype(np.float16)
        c, s = oracle.quantize_rows(xs, "fp16")
        assert np.array_equal(c, base)
        assert np.array_equal(s, s0 * np.float32(2.0 ** k))


def test_sign_symmetry_clip1():
    x = random_features(15, 32, 128)
    c1, s1 = oracle.quantize_rows(x, "fp16")
    c2, s2 = oracle.quantize_rows(-x, "fp16")
    assert np.array_equal(c1, -c2) and np.array_equal(s1, s2)


def test_zero_row():
    x = np.zeros((3, 16), dtype=np.float16)
    x[1, 3] = np.float16(-2.0)
    codes, scales = oracle.quantize_rows(x, "fp16")
    assert scales[0] == 0 and scales[2] == 0 and not codes[0].any() and not codes[2].any()
    assert codes[1, 3] == -7 and scales[1] == np.float32(np.float32(2) / np.float32(7))


def test_nonfinite_rejected():
    x = np.array([[1.0, np.inf]], dtype=np.float16)
    with pytest.raises(ValueError):
        oracle.quantize_rows(x, "fp16")


def test_bf16_decoding():
    v = np.array([1.0, -2.5, 3.1415926, 1e-30, -65504.0, 0.0], dtype=np.float32)
    bits = f32_to_bf16_bits(v)
    back = oracle.as_f32(bits, "bf16")
    import torch
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(back, ref)


# ---------------------------------------------------------------- packing
def test_pack_nibble_order():
    c = np.array([[1, -1, 7, -8]], dtype=np.int8)
    assert oracle.pack_int4(c).tolist() == [[0xF1, 0x87]]


def test_pack_roundtrip_all_codes():
    c = np.arange(-8, 8, dtype=np.int8)
    grid = np.stack(np.meshgrid(c, c, indexing="ij"), -1).reshape(1, -1)
    assert np.array_equal(oracle.unpack_int4(oracle.pack_int4(grid)), grid)


def test_high_nibble_unpack_identity():
    """The GPU unpacks nibbles into the high half of an int8 (value 16*code);
    pin that masking a packed byte that way yields exactly 16*code."""
    rng = np.random.default_rng(5)
    c = rng.integers(-8, 8, size=(1, 64)).astype(np.int8)
    p = oracle.pack_int4(c)[0]
    hi = (p & 0xF0).astype(np.uint8).view(np.int8).astype(np.int32)
    lo = ((p.astype(np.uint32) << 4) & 0xF0).astype(np.uint8).view(np.int8).astype(np.int32)
    assert np.array_equal(hi, 16 * c[0, 1::2]) and np.array_equal(lo, 16 * c[0, 0::2])
