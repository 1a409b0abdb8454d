"""Pins of the oracle's block-wise absmax 8-bit quantizer (paper Sec. 3.5: block-wise
8-bit AdamW states with block-wise scale handling; the linear absmax code map is
this implementation's reading).

Pins: the round trip is within half a code step; codes are idempotent; +-A map
to +-127 and A to 255; zero and non-representable scales give a zero block;
odd symmetry and monotonicity; exact ties round to even; the code step is the
once-rounded quotient A/127 (A/255); and the codes equal the exactly rounded
rational q = round_half_even(x * 127 / A) except near ties of the rational
value, where the fp32 product may land on the other side.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from exact_fp import round_half_even, round_to_f32


def _blocks(rng, n, scale):
    x = rng.standard_t(3, size=n).astype(np.float32) * np.float32(scale)
    return x


@pytest.mark.parametrize("scale", [1e-30, 1e-8, 1e-3, 1.0, 1e6])
@pytest.mark.parametrize("n", [1, 7, 256, 2048, 4096])
def test_signed_round_trip_within_half_step(scale, n):
    rng = np.random.default_rng(n + int(np.log10(scale) + 40))
    x = _blocks(rng, n, scale)
    q, A = oracle.quantize_signed(x)
    assert A == np.max(np.abs(x))
    xr = oracle.dequantize_signed(q, A)
    step = float(A) / 127.0
    err = np.abs(xr.astype(np.float64) - x.astype(np.float64))
    assert np.all(err <= 0.5 * step * (1 + 2.0 ** -20) + 2.0 ** -22 * np.abs(x))
    assert q.min() >= -127 and q.max() <= 127


@pytest.mark.parametrize("scale", [1e-30, 1e-12, 1e-6, 1.0, 1e6])
@pytest.mark.parametrize("n", [1, 7, 256, 2048])
def test_unsigned_round_trip_within_half_step(scale, n):
    rng = np.random.default_rng(7 * n + 3)
    x = (rng.standard_t(3, size=n).astype(np.float32) ** 2) * np.float32(scale)
    q, A = oracle.quantize_unsigned(x)
    assert A == np.max(x)
    xr = oracle.dequantize_unsigned(q, A)
    step = float(A) / 255.0
    err = np.abs(xr.astype(np.float64) - x.astype(np.float64))
    assert np.all(err <= 0.5 * step * (1 + 2.0 ** -20) + 2.0 ** -22 * np.abs(x))


def test_extremes_map_to_full_scale():
    x = np.array([0.3, -1.25, 1.25, 0.0], dtype=np.float32)
    q, A = oracle.quantize_signed(x)
    assert A == np.float32(1.25) and q[1] == -127 and q[2] == 127 and q[3] == 0
    v = np.array([0.0, 2.5, 1.0], dtype=np.float32)
    qv, Av = oracle.quantize_unsigned(v)
    assert Av == np.float32(2.5) and qv[1] == 255 and qv[0] == 0


def test_codes_are_idempotent():
    rng = np.random.default_rng(5)
    for _ in range(200):
        n = int(rng.integers(1, 300))
        q = rng.integers(-127, 128, size=n).astype(np.int8)
        q[rng.integers(0, n)] = 127 * (1 if rng.random() < 0.5 else -1)  # block max present
        A = np.float32(10.0 ** rng.uniform(-20, 20))
        q2, A2 = oracle.quantize_signed(oracle.dequantize_signed(q, A))
        assert np.array_equal(q, q2)
        qu = rng.integers(0, 256, size=n).astype(np.uint8)
        qu[rng.integers(0, n)] = 255
        qu2, _ = oracle.quantize_unsigned(oracle.dequantize_unsigned(qu, A))
        assert np.array_equal(qu, qu2)


def test_zero_and_unrepresentable_scales_give_zero_block():
    q, A = oracle.quantize_signed(np.zeros(5, np.float32))
    assert A == 0 and not q.any()
    q, A = oracle.quantize_unsigned(np.zeros(5, np.float32))
    assert A == 0 and not q.any()
    tiny = np.array([1e-40, -2e-40], dtype=np.float32)  # 127 / 2e-40 overflows fp32
    q, A = oracle.quantize_signed(tiny)
    assert A == 0 and not q.any()
    q, A = oracle.quantize_unsigned(np.array([1.0, np.inf], np.float32))
    assert A == 0 and not q.any()


def test_odd_symmetry_and_monotone():
    rng = np.random.default_rng(9)
    x = np.sort(rng.standard_normal(2048).astype(np.float32))
    q, A = oracle.quantize_signed(x)
    qn, An = oracle.quantize_signed(-x)
    assert A == An and np.array_equal(qn, -q)
    assert np.all(np.diff(q.astype(np.int32)) >= 0)
    v = np.sort(np.abs(x))
    qv, _ = oracle.quantize_unsigned(v)
    assert np.all(np.diff(qv.astype(np.int32)) >= 0)


def test_exact_ties_round_to_even():
    """With A = 127 (A = 255) the code scale is exactly 1, so x * inv = x and a
    half-integer x is an exact tie of the rational code value: round half to even."""
    x = np.array([127.0, 2.5, 0.5, -1.5, 3.5, -0.5, 126.5, -125.5], dtype=np.float32)
    q, A = oracle.quantize_signed(x)
    assert A == 127.0
    assert q.tolist() == [127, 2, 0, -2, 4, 0, 126, -126]
    v = np.array([255.0, 2.5, 0.5, 1.5, 254.5, 127.5], dtype=np.float32)
    qv, Av = oracle.quantize_unsigned(v)
    assert Av == 255.0
    assert qv.tolist() == [255, 2, 0, 2, 254, 128]


def test_code_step_is_the_correctly_rounded_quotient():
    """Code 1 dequantizes to fp32(A / 127) (fp32(A / 255)), the quotient rounded once,
    and code q to fp32(q * that step): checked with exact rationals over scales
    from subnormal to near the top of the fp32 range."""
    rng = np.random.default_rng(31)
    scales = np.concatenate([
        (rng.uniform(1, 2, 400) * 2.0 ** rng.integers(-149, 127, 400)).astype(np.float32),
        np.array([1.0, 127.0, 255.0, 1e-45, 3.4e38, 1.1754944e-38], np.float32)])
    one = np.array([1], np.int8)
    qs = np.array([1, -7, 64, 127], np.int8)
    for A in scales.tolist():
        FA = Fraction(A)
        step_m = round_to_f32(FA / 127)
        assert float(oracle.dequantize_signed(one, A)[0]) == step_m, A
        got = oracle.dequantize_signed(qs, A).tolist()
        assert got == [round_to_f32(int(q) * Fraction(step_m)) for q in qs.tolist()], A
        step_v = round_to_f32(FA / 255)
        assert float(oracle.dequantize_unsigned(one.view(np.uint8), A)[0]) == step_v, A


_round_half_even = round_half_even


def test_codes_match_exact_rational_rounding_except_at_ties():
    rng = np.random.default_rng(21)
    mismatches, total = 0, 0
    for _ in range(60):
        x = rng.standard_t(3, size=256).astype(np.float32) * np.float32(1e-3)
        q, A = oracle.quantize_signed(x)
        FA = Fraction(float(A))
        for xi, qi in zip(x.tolist(), q.tolist()):
            exact = Fraction(xi) * 127 / FA
            ref = _round_half_even(exact)
            total += 1
            if ref != qi:
                mismatches += 1
                # only allowed where the rational value sits at a .5 tie to ~fp32 precision
                frac = exact - (exact.numerator // exact.denominator)
                assert abs(frac - Fraction(1, 2)) <= Fraction(1, 2 ** 16), (xi, qi, ref)
                assert abs(ref - qi) == 1
    assert mismatches <= max(1, total // 1000)
