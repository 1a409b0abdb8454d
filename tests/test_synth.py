"""The seeded input generator: determinism, slicing, thread invariance, and the
value distributions of the synthetic workloads."""
import math

import numpy as np
import pytest
from scipy import stats

import synth
from golden_io import bf16_bits_to_f32


def test_workload_sizes():
    assert synth.tiny().n_params == 2_622_464
    assert synth.layer_3b().n_params == 77_074_432
    assert synth.full_3b().n_params == 3_085_844_480
    assert len(synth.full_3b().shapes) == 325
    assert synth.streamed_27b().n_params == 21_139_947_520
    assert len(synth.streamed_27b().shapes) == 576
    assert synth.clip_stress().n_params == 3_085_844_480


def test_slices_and_threads_are_bitwise_stable():
    w = synth.layer_3b()
    full = w.grads(1, 5, n_threads=1)
    assert np.array_equal(full, w.grads(1, 5, n_threads=8))
    part = w.grads(1, 5, offset=12345, n=1000)
    assert np.array_equal(part, full[12345:13345])
    wf = w.weights(7)
    assert np.array_equal(wf[1:9], w.weights(7, offset=1, n=8))  # odd offset of a normal pair


def test_streams_and_tensors_are_independent():
    w = synth.layer_3b()
    a = bf16_bits_to_f32(w.grads(1, 3)).astype(np.float64)
    b = bf16_bits_to_f32(w.grads(1, 4)).astype(np.float64)
    c = bf16_bits_to_f32(w.grads(2, 3)).astype(np.float64)
    assert abs(np.corrcoef(a, b)[0, 1]) < 0.01 and abs(np.corrcoef(a, c)[0, 1]) < 0.01


def test_distributions():
    w = synth.layer_3b()
    x = w.weights(4, n=400_000)
    assert abs(x.std() - 0.02) < 2e-4
    assert stats.kstest(x / 0.02, "norm").pvalue > 1e-3
    g = bf16_bits_to_f32(w.grads(4, 4, n=400_000))
    assert stats.kstest(g / 1e-3, "t", args=(3,)).pvalue > 1e-3
    t = synth.tiny()
    g0 = t.grads(1, 4)
    big = np.abs(g0) > 2e-2  # outliers are x100 of a 1e-3 normal
    assert 0.005 < big.mean() < 0.015


def test_clip_stress_outliers_and_zero_blocks():
    w = synth.clip_stress()
    k = 1
    g = bf16_bits_to_f32(w.grads(k, synth.grad_stream(1)))
    block = 2048
    nb = g.size // block
    zero = np.array([synth.block_is_zero(w.seed, k, b, 64) for b in range(nb)])
    gb = g.reshape(nb, block)
    assert not np.any(gb[zero])
    assert 0.005 < zero.mean() < 0.03
    out = np.abs(g) == np.float32(9984.0)  # +-1e4 rounds to +-9984 in bf16
    assert 0.0005 < out.mean() < 0.0015
    sigma = 1e3 / math.sqrt(w.n_params)
    body = g[(~out) & np.repeat(~zero, block)]
    assert abs(body.std() / sigma - 1) < 0.02
    # same zero blocks at every step
    g2 = bf16_bits_to_f32(w.grads(k, synth.grad_stream(2)))
    assert not np.any(g2.reshape(nb, block)[zero])
