"""Pins of the oracle's clip coefficient (paper Sec. 3.5: the global norm scales
the gradients with one multiplication; App. C: max grad norm 1.0).

Pinned against PyTorch's own clip_grad_norm_ (a different implementation with a
different reduction order: agreement within 1e-6 relative), and against closed
forms: max_norm = inf gives exactly 1, a norm below the threshold gives exactly 1.
"""
import math

import numpy as np
import pytest
import torch

import oracle


@pytest.mark.parametrize("scale", [1e-4, 1e-2, 1.0, 30.0, 1e4])
def test_matches_torch_clip_grad_norm(scale):
    g = torch.Generator().manual_seed(int(scale * 1000) % 9973)
    shapes = [(257, 33), (1000,), (64, 64, 3), (1,)]
    grads = [torch.randn(s, generator=g, dtype=torch.float32) * scale for s in shapes]
    params = [torch.nn.Parameter(torch.zeros(s)) for s in shapes]
    for p, gr in zip(params, grads):
        p.grad = gr.clone()
    total = torch.nn.utils.clip_grad_norm_(params, max_norm=1.0, foreach=False)
    # coefficient torch applied, read back from one nonzero element
    ratio = float(params[0].grad.flatten()[0] / grads[0].flatten()[0])

    _, s, status = oracle.grad_sqnorm([x.numpy().ravel() for x in grads])
    norm, coef = oracle.clip_coef(s, 1.0)
    assert status == oracle.STATUS_OK
    assert abs(float(norm) - float(total)) <= 1e-6 * float(total)
    assert abs(float(coef) - ratio) <= 1e-6 * ratio


def test_infinite_max_norm_means_no_clipping():
    for s in (0.0, 1e-30, 0.5, 1.0, 3.7e3, 1e300):
        norm, coef = oracle.clip_coef(s, math.inf)
        assert coef == np.float32(1.0)
        with np.errstate(over="ignore"):  # sqrt(1e300) = 1e150 rounds to fp32 infinity
            assert norm == np.float32(math.sqrt(s))


def test_below_threshold_is_exactly_one():
    for s in (0.0, 1e-12, 0.25, 0.9801):
        _, coef = oracle.clip_coef(s, 1.0)
        assert coef == np.float32(1.0)


def test_above_threshold_scales_to_max_norm():
    # S = 16 -> norm 4 -> coef ~ 1/4 (the 1e-6 guard makes it a hair smaller)
    norm, coef = oracle.clip_coef(16.0, 1.0)
    assert norm == np.float32(4.0)
    assert 0.25 * (1 - 1e-6) <= float(coef) < 0.25
    norm, coef = oracle.clip_coef(16.0, 2.0)
    assert 0.5 * (1 - 1e-6) <= float(coef) < 0.5


def test_threshold_itself_is_slightly_clipped():
    # norm == max_norm: coef = 1 / (1 + 1e-6) < 1, as in the PyTorch convention
    _, coef = oracle.clip_coef(1.0, 1.0)
    assert float(coef) < 1.0 and abs(float(coef) - 1 / (1 + 1e-6)) < 1e-7


def test_norm_is_fp64_sqrt_rounded_once():
    # 2^-149 squared is far below fp32 range but the norm is exact after the fp64 sqrt
    norm, _ = oracle.clip_coef(2.0 ** -298, 1.0)
    assert norm == np.float32(2.0 ** -149)
    norm, _ = oracle.clip_coef(2.0 ** 200, 1.0)
    assert norm == np.float32(2.0 ** 100)


def test_nonfinite_sum_of_squares():
    norm, coef = oracle.clip_coef(math.inf, 1.0)
    assert math.isinf(norm) and coef == np.float32(0.0)
    norm, coef = oracle.clip_coef(math.nan, 1.0)
    assert math.isnan(norm) and coef == np.float32(1.0)  # fminf ignores the NaN
