"""Pins of the oracle's dynamic (non-linear) code map and its quantizer.

The map: a code's magnitude bits are leading zeros (the decade 10^-zeros), an
indicator one, and p linear fraction bits spanning (0.1, 1] of the decade.
Checked here through properties that a slip in the construction breaks: the
decade tops are the powers of ten, each decade holds 2^p codes at a constant
spacing 0.9 * 10^-zeros / 2^p starting one spacing above 0.1 * 10^-zeros, the
magnitudes rise strictly, and the top code is exactly 1.  The quantizer is
checked against exact rational nearest-code search, the round trip of code
values, the half-gap error bound, exact ties, the zero-block rule and sign handling."""
import bisect
from fractions import Fraction

import numpy as np
import pytest

import oracle
from exact_fp import round_to_f32


def _decades(bits):
    """(decade index E, first code, number of codes) for a map of `bits` magnitude bits."""
    out = []
    for p in range(bits):
        out.append((bits - 1 - p, 1 << p, 1 << p))
    return out


@pytest.mark.parametrize("signed,bits", [(True, 7), (False, 8)])
def test_map_structure(signed, bits):
    t = oracle.dynamic_map(signed).astype(np.float64)
    assert t.size == 1 << bits
    assert t[0] == 0.0 and t[-1] == 1.0
    assert np.all(np.diff(t) > 0)
    for E, first, count in _decades(bits):
        codes = t[first:first + count]
        top = np.float32(10.0 ** -E)
        assert codes[-1] == top, (E, codes[-1])
        step = 0.9 * 10.0 ** -E / count
        # one spacing above the decade's floor, then constant spacing (fp32 rounding)
        assert abs(codes[0] - (0.1 * 10.0 ** -E + step)) <= 2 * np.spacing(np.float32(codes[0]))
        if count > 1:
            d = np.diff(codes)
            assert np.all(np.abs(d - step) <= 2 * np.spacing(np.float32(top)))
    # smallest nonzero magnitude: 1e-6 (signed), 1e-7 (unsigned)
    assert t[1] == np.float32(1e-6 if signed else 1e-7)


def _exact_nearest(table, a):
    """Index of the nearest table value to a in exact arithmetic (ties: lower)."""
    fa = Fraction(float(a))
    best, bd = 0, None
    for c, v in enumerate(table):
        d = abs(fa - Fraction(float(v)))
        if bd is None or d < bd:
            best, bd = c, d
    return best, bd


@pytest.mark.parametrize("signed", [True, False])
def test_quantizer_against_exact_nearest(signed):
    rng = np.random.default_rng(3)
    t = oracle.dynamic_map(signed)
    n = 2048
    # magnitudes spread over all decades, and values right at codes and midpoints
    x = (10.0 ** rng.uniform(-8, 0, size=n)).astype(np.float32)
    x[:200] = t[rng.integers(0, t.size, size=200)]
    mid = ((t[1:].astype(np.float64) + t[:-1]) / 2).astype(np.float32)
    x[200:400] = mid[rng.integers(0, mid.size, size=200)]
    x[0] = 1.0  # absmax 1: the normalized value is the value itself
    if signed:
        x *= np.where(rng.random(n) < 0.5, -1, 1).astype(np.float32)
        q, A = oracle.quantize_dynamic_signed(x)
        c = q.view(np.uint8) & 0x7F
        neg = (q.view(np.uint8) & 0x80) != 0
        assert np.array_equal(neg, x < 0)
    else:
        q, A = oracle.quantize_dynamic_unsigned(x)
        c = q
    assert A == 1.0
    a = np.abs(x)
    for i in range(n):
        want, _ = _exact_nearest(t, a[i])
        if c[i] != want:
            # allowed only where fp32 distances tie or round across an exact near-tie
            d_got = abs(Fraction(float(a[i])) - Fraction(float(t[c[i]])))
            d_want = abs(Fraction(float(a[i])) - Fraction(float(t[want])))
            assert abs(int(c[i]) - want) == 1
            assert d_got - d_want <= Fraction(float(np.spacing(np.float32(a[i])))), i


@pytest.mark.parametrize("signed", [True, False])
def test_exact_midpoints_take_the_smaller_code(signed):
    """Where the midpoint of two neighbouring magnitudes is itself an fp32 value,
    its two distances are the same real number, so they round alike: an exact
    tie, resolved to the smaller code (the smaller magnitude)."""
    t = oracle.dynamic_map(signed)
    mids, lower = [], []
    for c in range(t.size - 1):
        mid = (Fraction(float(t[c])) + Fraction(float(t[c + 1]))) / 2
        if Fraction(round_to_f32(mid)) == mid:
            mids.append(float(mid))
            lower.append(c)
    assert len(mids) >= 20
    x = np.array([1.0] + mids, dtype=np.float32)  # absmax 1: normalized value = value
    if signed:
        q, A = oracle.quantize_dynamic_signed(-x)
        assert np.all(q.view(np.uint8)[1:] & 0x80)
        c = (q.view(np.uint8) & 0x7F)[1:]
    else:
        q, A = oracle.quantize_dynamic_unsigned(x)
        c = q[1:]
    assert A == 1.0
    assert c.tolist() == lower


def _reading_code(t_exact, A, x):
    """The code of x in a block of absmax A under the fp32 reading, in exact
    arithmetic: a = fp32(|x| * fp32(1 / A)), distances fp32(|a - t_c|), the
    smallest code among the least distances."""
    inv = Fraction(round_to_f32(1 / Fraction(A)))
    a = Fraction(round_to_f32(abs(Fraction(x)) * inv))
    # Rounding is monotone, so a code beyond a's neighbours on either side never
    # has a smaller rounded distance than the neighbour on that side; the code
    # gaps exceed an ulp of any distance, so it cannot tie with it either.
    k = bisect.bisect_left(t_exact, a)
    lo, hi = max(0, k - 2), min(len(t_exact), k + 2)
    d = [round_to_f32(abs(a - tc)) for tc in t_exact[lo:hi]]
    return lo + d.index(min(d))


@pytest.mark.parametrize("signed", [True, False])
def test_codes_follow_the_fp32_reading_exactly(signed):
    """Blocks whose scale has an inexact reciprocal, with values placed within a
    few ulps of the midpoints between codes, where the normalization's rounding
    decides the code: every code equals the exact evaluation of the reading."""
    rng = np.random.default_rng(41 + signed)
    t = oracle.dynamic_map(signed)
    t_exact = [Fraction(float(v)) for v in t]
    for A in (np.float32(0.7), np.float32(3.0e-3), np.float32(1.9e-7)):
        FA = Fraction(float(A))
        c = rng.integers(1, t.size - 1, size=150)
        mids = [(t_exact[i] + t_exact[i + 1]) / 2 * FA for i in c.tolist()]
        x = np.array([round_to_f32(m) for m in mids], dtype=np.float32)
        ulps = rng.integers(-3, 4, size=x.size).astype(np.int32)
        x = (x.view(np.int32) + ulps).view(np.float32)
        x = np.concatenate([[A], x, (rng.uniform(0, 1, 100) * A).astype(np.float32)])
        x = np.minimum(x, A).astype(np.float32)
        if signed:
            q, got_A = oracle.quantize_dynamic_signed(-x)
            codes = (q.view(np.uint8) & 0x7F).tolist()
        else:
            q, got_A = oracle.quantize_dynamic_unsigned(x)
            codes = q.tolist()
        assert got_A == A
        want = [_reading_code(t_exact, float(A), float(v)) for v in x.tolist()]
        assert codes == want, A


@pytest.mark.parametrize("signed", [True, False])
def test_round_trip_and_error_bound(signed):
    t = oracle.dynamic_map(signed)
    rng = np.random.default_rng(4)
    A = np.float32(3.0e-3)
    codes = np.arange(t.size)
    x = (t.astype(np.float64) * A).astype(np.float32)
    x[-1] = A
    if signed:
        q, absmax = oracle.quantize_dynamic_signed(x)
        back = oracle.dequantize_dynamic_signed(q, absmax)
        assert np.array_equal(q.view(np.uint8) & 0x7F, codes)
    else:
        q, absmax = oracle.quantize_dynamic_unsigned(x)
        back = oracle.dequantize_dynamic_unsigned(q, absmax)
        assert np.array_equal(q, codes)
    assert absmax == A
    assert np.array_equal(back, x)  # t * A rounds the same way on both sides
    # random block: error within half the local gap (plus fp32 rounding)
    y = (rng.standard_t(3, size=4096) * 1e-3).astype(np.float32)
    if not signed:
        y = y * y
    q, absmax = (oracle.quantize_dynamic_signed if signed else oracle.quantize_dynamic_unsigned)(y)
    back = (oracle.dequantize_dynamic_signed if signed else oracle.dequantize_dynamic_unsigned)(
        q, absmax)
    a = np.abs(y.astype(np.float64)) / absmax
    hi = np.searchsorted(t.astype(np.float64), a).clip(1, t.size - 1)
    gap = (t[hi].astype(np.float64) - t[hi - 1]) * absmax
    err = np.abs(back.astype(np.float64) - y)
    assert np.all(err <= 0.5 * gap + 4 * np.spacing(np.abs(y)) + 1e-45)


def test_zero_block_nan_and_signs():
    q, A = oracle.quantize_dynamic_signed(np.zeros(64, np.float32))
    assert A == 0 and not q.any()
    x = np.full(64, 1.0, np.float32)
    x[3] = np.inf
    q, A = oracle.quantize_dynamic_signed(x)
    assert A == 0 and not q.any()
    x = np.array([1e-39, 2e-39], np.float32)  # 1/A overflows: zero block
    q, A = oracle.quantize_dynamic_unsigned(x)
    assert A == 0 and not q.any()
    x = np.array([0.5, np.nan, -0.0, -0.25, 1e-9, -1.0, -1e-9], np.float32)
    q, A = oracle.quantize_dynamic_signed(x)
    b = q.view(np.uint8)
    assert A == 1.0 and b[1] == 0 and b[2] == 0 and b[4] == 0
    assert b[5] == 0x80 | 127 and b[3] & 0x80 and not b[0] & 0x80
    assert b[6] == 0x80  # a negative value below the smallest magnitude keeps its sign
    back = oracle.dequantize_dynamic_signed(q, A)
    assert back[6] == 0 and np.signbit(back[6]) and not np.signbit(back[4])
    # odd symmetry
    y = np.linspace(-1, 1, 1001).astype(np.float32)
    q, _ = oracle.quantize_dynamic_signed(y)
    qn, _ = oracle.quantize_dynamic_signed(-y)
    nz = (q.view(np.uint8) & 0x7F) != 0
    assert np.array_equal(q.view(np.uint8)[nz] ^ 0x80, qn.view(np.uint8)[nz])


def test_dynamic_first_step_weights_equal_linear():
    """From zero state the moments decode to 0 under either map, so the weights of
    the first step do not depend on the map (only the stored codes do)."""
    rng = np.random.default_rng(5)
    n, block = 5000, 256
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g = (rng.standard_t(3, size=n) * 1e-3).astype(np.float32)
    out = []
    for cm in (oracle.MAP_LINEAR, oracle.MAP_DYNAMIC):
        ww = w.copy()
        qm, qv = np.zeros(n, np.int8), np.zeros(n, np.uint8)
        am, av = np.zeros(-(-n // block), np.float32), np.zeros(-(-n // block), np.float32)
        oracle.hybrid8bit_adamw_step([ww], [g], [qm], [am], [qv], [av], block, lr=1e-3,
                                     beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, step=1,
                                     code_map=cm)
        out.append((ww, am, av))
    assert out[0][0].tobytes() == out[1][0].tobytes()
    assert out[0][1].tobytes() == out[1][1].tobytes()  # the absmax is the same
    assert out[0][2].tobytes() == out[1][2].tobytes()


def test_dynamic_map_removes_the_small_v_hazard():
    """Three 8-bit steps against fp64 AdamW, as the linear-map drift test: with the
    dynamic map a second moment down to 5e-8 of its block's absmax keeps a nonzero
    code, so the v = 0 / m != 0 case falls from about half of the elements (linear
    map) to a fraction of a percent, where m is tiny too, and every element stays
    within one lr of fp64 AdamW (the linear map drifts by up to ~1400 lr)."""
    rng = np.random.default_rng(10)
    n, block = 2048 * 8, 2048
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    w8, qm, qv = w.copy(), np.zeros(n, np.int8), np.zeros(n, np.uint8)
    am, av = np.zeros(8, np.float32), np.zeros(8, np.float32)
    w64, m64, v64 = w.astype(np.float64), np.zeros(n), np.zeros(n)
    lr, b1, b2, eps, wd = 1e-4, 0.9, 0.999, 1e-8, 0.01
    hazard = np.zeros(n, bool)
    for t in (1, 2, 3):
        g = (rng.standard_t(3, size=n) * 1e-3).astype(np.float32)
        hazard |= (qv == 0) & ((qm.view(np.uint8) & 0x7F) != 0)
        oracle.hybrid8bit_adamw_step([w8], [g], [qm], [am], [qv], [av], block, lr=lr, beta1=b1,
                                     beta2=b2, eps=eps, weight_decay=wd, step=t,
                                     code_map=oracle.MAP_DYNAMIC)
        g64 = g.astype(np.float64)
        m64 = b1 * m64 + (1 - b1) * g64
        v64 = b2 * v64 + (1 - b2) * g64 ** 2
        w64 = w64 * (1 - lr * wd) - lr / (1 - b1 ** t) * m64 / (
            np.sqrt(v64) / np.sqrt(1 - b2 ** t) + eps)
        drift = np.abs(w8 - w64) / lr
        print(f"step {t}: drift/lr max {drift.max():.3g}, hazard fraction {hazard.mean():.4f}")
        assert hazard.mean() < 0.01
        assert drift.max() < 1.0


@pytest.mark.parametrize("as_bf16", [False, True])
def test_hand_worked_dynamic_examples(as_bf16):
    from golden_io import adamw_examples, f32_to_bf16_bits
    n = 0
    for ex in adamw_examples("dynamic_map_worked_examples.txt"):
        g = f32_to_bf16_bits(ex["grad"]) if as_bf16 else ex["grad"]
        w, qm, qv = ex["w"].copy(), ex["m_codes"].copy(), ex["v_codes"].copy()
        am, av = ex["m_absmax"].copy(), ex["v_absmax"].copy()
        oracle.hybrid8bit_adamw_step([w], [g], [qm], [am], [qv], [av], ex["block_size"],
                                     lr=ex["lr"], beta1=ex["beta1"], beta2=ex["beta2"],
                                     eps=ex["eps"], weight_decay=ex["weight_decay"],
                                     step=ex["t"], coef=ex["coef"],
                                     code_map=oracle.MAP_DYNAMIC)
        name = ex["name"]
        assert np.array_equal(w, ex["expect_w"]), (name, w)
        assert np.array_equal(qm, ex["expect_m_codes"]), (name, qm)
        assert np.array_equal(am, ex["expect_m_absmax"]), (name, am)
        assert np.array_equal(qv, ex["expect_v_codes"]), (name, qv)
        assert np.array_equal(av, ex["expect_v_absmax"]), (name, av)
        n += 1
    assert n == 2
