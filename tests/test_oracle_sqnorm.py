"""Pins of the oracle's gradient sum of squares (paper Sec. 3.5: per-tensor norms,
then one global aggregate; the reduction order is this implementation's reading).

Pins, none of which reuse the oracle's own code:
* exact inputs (small integers times 2^-10): every partial sum is exact, so the
  result must equal the integer sum bitwise in any order -- catches a dropped,
  duplicated or misplaced element anywhere in the chunk/lane/tail indexing;
* hand-derived order cases (tests/golden/sqnorm_order.txt) that give different
  bits under any other grouping of lanes, granules, waves, chunks or tensors;
* random inputs against an exactly rounded sum (math.fsum of exact squares) within
  the tree's error bound;
* thread-count invariance and non-finite detection.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from golden_io import bf16_bits_to_f32, dense, f32_to_bf16_bits, sqnorm_cases

SIZES = [1, 7, 8, 255, 257, 2047, 2049, 5120, 8191, 8192, 8193, 3 * 8192 + 17, 300001]


def _exact_inputs(n, rng):
    k = rng.integers(-256, 257, size=n)
    return k, (k.astype(np.float64) * 2.0 ** -10).astype(np.float32)


@pytest.mark.parametrize("as_bf16", [False, True])
def test_exact_integer_inputs_match_integer_sum(as_bf16):
    rng = np.random.default_rng(11)
    arrays, exact_sk = [], []
    for n in SIZES:
        k, x = _exact_inputs(n, rng)
        arrays.append(f32_to_bf16_bits(x) if as_bf16 else x)
        exact_sk.append(float(int(np.sum(k.astype(np.int64) ** 2))) * 2.0 ** -20)
    sk, s, status = oracle.grad_sqnorm(arrays)
    assert status == oracle.STATUS_OK
    assert [v.hex() for v in sk.tolist()] == [v.hex() for v in exact_sk]
    total = float(sum(int(round(v * 2 ** 20)) for v in exact_sk)) * 2.0 ** -20
    assert s == total


def test_exact_inputs_any_permutation():
    rng = np.random.default_rng(12)
    _, x = _exact_inputs(70001, rng)
    _, s0, _ = oracle.grad_sqnorm([x])
    for _ in range(3):
        _, s1, _ = oracle.grad_sqnorm([rng.permutation(x)])
        assert s1 == s0


@pytest.mark.parametrize("as_bf16", [False, True])
def test_hand_derived_reduction_order(as_bf16):
    n_cases = 0
    for name, tensors, expect_sk, expect_s in sqnorm_cases():
        arrays = [dense(n, vals) for n, vals in tensors]
        if as_bf16:
            arrays = [f32_to_bf16_bits(a) for a in arrays]
        sk, s, status = oracle.grad_sqnorm(arrays)
        assert status == oracle.STATUS_OK, name
        assert [v.hex() for v in sk.tolist()] == [v.hex() for v in expect_sk], name
        assert s.hex() == expect_s.hex(), name
        n_cases += 1
    assert n_cases >= 6


def _fsum_sq(arrays):
    terms = []
    for a in arrays:
        f = bf16_bits_to_f32(a) if a.dtype == np.uint16 else a
        terms.append(f.astype(np.float64) ** 2)  # exact squares
    return math.fsum(np.concatenate(terms).tolist())


@pytest.mark.parametrize("workload", [0, 1])
def test_random_inputs_within_tree_error_bound(workload):
    w = synth.WORKLOADS[workload]()
    # the layer's FFN matrices are left out to keep math.fsum's exact sum quick
    arrays = [w.grads(k, synth.grad_stream(w.step)) for k in range(len(w.shapes))
              if w.numels[k] <= 5_000_000]
    sk, s, status = oracle.grad_sqnorm(arrays, n_threads=8)
    assert status == oracle.STATUS_OK
    exact = _fsum_sq(arrays)
    # ~600 additions of non-negative terms at most: relative error < 600 * 2^-53.
    assert abs(s - exact) <= 1e-12 * exact
    for a, v in zip(arrays, sk):
        e = _fsum_sq([a])
        assert abs(v - e) <= 1e-12 * e
    naive = oracle.grad_sqnorm_naive(arrays)
    assert abs(naive - exact) <= 1e-9 * exact  # plain index order: looser bound


def test_thread_count_does_not_change_bits():
    w = synth.layer_3b()
    arrays = [w.grads(k, 3) for k in range(len(w.shapes))]
    r1 = oracle.grad_sqnorm(arrays, n_threads=1)
    r8 = oracle.grad_sqnorm(arrays, n_threads=8)
    assert r1[1] == r8[1]
    assert r1[0].tobytes() == r8[0].tobytes()


@pytest.mark.parametrize("bad", [np.inf, -np.inf, np.nan])
@pytest.mark.parametrize("as_bf16", [False, True])
def test_nonfinite_gradient_sets_status(bad, as_bf16):
    x = np.full(10000, 1e-3, dtype=np.float32)
    x[7777] = bad
    a = f32_to_bf16_bits(x) if as_bf16 else x
    _, s, status = oracle.grad_sqnorm([np.ones(5, np.float32) if not as_bf16 else
                                       f32_to_bf16_bits(np.ones(5, np.float32)), a])
    assert status == oracle.STATUS_NONFINITE
    assert not math.isfinite(s)


def test_largest_finite_inputs_do_not_overflow():
    x = np.full(1 << 16, np.finfo(np.float32).max, dtype=np.float32)
    _, s, status = oracle.grad_sqnorm([x])
    assert status == oracle.STATUS_OK
    assert s == float(np.finfo(np.float32).max) ** 2 * (1 << 16)


def test_subnormal_inputs_are_not_flushed():
    tiny = np.float32(2.0 ** -140)  # an fp32 subnormal; its square is normal in fp64
    x = np.full(3, tiny, dtype=np.float32)
    _, s, _ = oracle.grad_sqnorm([x])
    assert s == 3 * 2.0 ** -280


def test_all_zero_gradients():
    sk, s, status = oracle.grad_sqnorm([np.zeros(n, np.float32) for n in (1, 8193)])
    assert s == 0.0 and status == oracle.STATUS_OK and sk.tolist() == [0.0, 0.0]


def test_empty_list_and_empty_tensors():
    # an empty sum is 0; an empty tensor adds +0.0 to the list-order total, which is
    # exact, so S equals that of the list without it (checked against the naive sum)
    sk, s, status = oracle.grad_sqnorm([])
    assert s == 0.0 and status == oracle.STATUS_OK and sk.size == 0
    rng = np.random.default_rng(5)
    a = f32_to_bf16_bits((rng.standard_normal(9000) * 1e-2).astype(np.float32))
    b = f32_to_bf16_bits((rng.standard_normal(20000) * 1e-2).astype(np.float32))
    e = np.zeros(0, np.uint16)
    sk, s, status = oracle.grad_sqnorm([e, a, e, e, b, e])
    _, s_ab, _ = oracle.grad_sqnorm([a, b])
    assert s == s_ab and status == oracle.STATUS_OK
    assert sk[[0, 2, 3, 5]].tolist() == [0.0] * 4
    assert abs(s - oracle.grad_sqnorm_naive([a, b])) <= 1e-12 * s
    assert oracle.grad_sqnorm([e, e])[1] == 0.0
