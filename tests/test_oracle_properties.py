"""Property-based pins of the oracle (hypothesis): arbitrary finite fp32 blocks,
including subnormals, signed zeros and values near the fp32 maximum, for the two
linear block quantizers, and arbitrary bf16 gradient lists for the sum of squares.
Each property follows from the definition, not from the oracle's code:

* quantizer: codes stay in range; the stored scale is the block's largest
  magnitude, or 0 exactly when 127/A (255/A) is not finite; a decoded value lies
  within half a code step of the input (plus the rounding of the step and of the
  product), with one exception this search found: a scale of exactly the largest
  fp32 value decodes the signed code +-127 to +-inf, because A/127 rounds up and
  127 times it overflows; negating the block negates the signed codes; codes are
  monotone in the input;
* sum of squares: equal to the exactly rounded sum of the squares within the
  bound of its fixed tree, exactly 0 for an all-zero list, and independent of
  the thread count."""
from fractions import Fraction

import numpy as np
from hypothesis import given, settings, strategies as st

import oracle
from golden_io import bf16_bits_to_f32

F32 = st.floats(width=32, allow_nan=False, allow_infinity=False)
BLOCKS = st.lists(F32, min_size=1, max_size=64).map(lambda xs: np.array(xs, dtype=np.float32))


def _half_step_bound(A, levels, x):
    step = np.float32(A) / np.float32(levels)
    return 0.5 * float(step) * (1 + 2.0 ** -20) + 2.0 ** -22 * abs(float(x))


@settings(max_examples=300, deadline=None)
@given(BLOCKS)
def test_signed_quantizer_properties(x):
    q, A = oracle.quantize_signed(x)
    amax = np.float32(np.max(np.abs(x)))
    inv = np.float32(127.0) / amax if amax > 0 else np.float32(np.inf)
    ok = np.isfinite(amax) and np.isfinite(inv)
    assert q.min() >= -127 and q.max() <= 127
    if not ok:
        assert A == 0 and not q.any()
        return
    assert A == amax
    d = oracle.dequantize_signed(q, A)
    for xi, qi, di in zip(x, q, d):
        if not np.isfinite(di):  # the one overflowing decode: A = FLT_MAX, code +-127
            assert A == np.finfo(np.float32).max and abs(int(qi)) == 127
            continue
        assert abs(float(di) - float(xi)) <= _half_step_bound(A, 127, xi)
    qn, An = oracle.quantize_signed(-x)
    assert An == A and np.array_equal(qn, -q)
    order = np.argsort(x, kind="stable")
    assert np.all(np.diff(q[order].astype(np.int32)) >= 0)


@settings(max_examples=300, deadline=None)
@given(BLOCKS)
def test_unsigned_quantizer_properties(x):
    x = np.abs(x)
    q, A = oracle.quantize_unsigned(x)
    amax = np.float32(np.max(x))
    inv = np.float32(255.0) / amax if amax > 0 else np.float32(np.inf)
    if not (np.isfinite(amax) and np.isfinite(inv)):
        assert A == 0 and not q.any()
        return
    assert A == amax
    d = oracle.dequantize_unsigned(q, A)
    for xi, di in zip(x, d):
        assert abs(float(di) - float(xi)) <= _half_step_bound(A, 255, xi)
    order = np.argsort(x, kind="stable")
    assert np.all(np.diff(q[order].astype(np.int32)) >= 0)


BF16_BITS = st.integers(min_value=0, max_value=0xFFFF).filter(
    lambda b: (b & 0x7F80) != 0x7F80)  # finite bf16 patterns only
GRAD_LISTS = st.lists(st.lists(BF16_BITS, min_size=0, max_size=300), min_size=0, max_size=4)


@settings(max_examples=200, deadline=None)
@given(GRAD_LISTS)
def test_sum_of_squares_properties(lists):
    grads = [np.array(v, dtype=np.uint16) for v in lists]
    _, S, status = oracle.grad_sqnorm(grads)
    assert status == oracle.STATUS_OK
    exact = sum((Fraction(float(x)) ** 2 for g in grads for x in bf16_bits_to_f32(g)),
                Fraction(0))
    if exact == 0:
        assert S == 0.0
        return
    # tree depth: 32 lane adds + 6 + 2 in the chunk + 8 over 256 accumulators + the list
    depth = 32 + 8 + 8 + len(grads)
    assert abs(Fraction(S) - exact) <= exact * Fraction(depth) * Fraction(2) ** -53
    _, S8, _ = oracle.grad_sqnorm(grads, n_threads=8)
    assert S8 == S
