"""Norm accumulation as gradients arrive: chunk partials written part by part
(in reverse layer order, on two streams) and finished once give S_k, S and the
status bitwise equal to the one-call sum of squares and to the oracle; the
layer-streamed step fed the finished norm (norm_ready) skips its first pass and
gives bitwise the same step."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, assert_state_equal, gpu_norm_and_coef, oracle_step, \
    to_dev, to_host

pytestmark = pytest.mark.gpu

SIZES = [1, 8192, 8193, 7, 100003, 65536, 2049, 300001, 16384, 5]
LAYERS = [0, 3, 4, 7, 10]


def _grads(rng, as_bf16):
    g = [(rng.standard_t(3, size=n) * 1e-3).astype(np.float32) for n in SIZES]
    return [f32_to_bf16_bits(x) for x in g] if as_bf16 else g


def _arrival(gdev, order, streams):
    acc = lt.GradNormAccumulator(SIZES, DEV)
    for i, layer in enumerate(order):
        a, b = LAYERS[layer], LAYERS[layer + 1]
        s = streams[i % len(streams)]
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            acc.add(a, gdev[a:b], stream=s)
    for s in streams:
        torch.cuda.current_stream().wait_stream(s)
    sk = torch.empty(len(SIZES), dtype=torch.float64, device=DEV)
    S = torch.empty(1, dtype=torch.float64, device=DEV)
    status = torch.empty(1, dtype=torch.int32, device=DEV)
    acc.finish(S, status, sq_per_tensor=sk)
    torch.cuda.synchronize()
    return to_host(sk), to_host(S)[0], int(to_host(status)[0])


@pytest.mark.parametrize("as_bf16", [False, True])
def test_partials_in_reverse_order_equal_one_call_and_oracle(as_bf16):
    rng = np.random.default_rng(70 + as_bf16)
    g = _grads(rng, as_bf16)
    gdev = [to_dev(x) for x in g]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    sk, S, st = _arrival(gdev, list(reversed(range(len(LAYERS) - 1))), streams)
    sk1, S1, st1, _, _ = gpu_norm_and_coef(gdev, 1.0)
    torch.cuda.synchronize()
    assert st == st1 == lt.LT_STATUS_OK
    assert S.hex() == to_host(S1)[0].hex()
    assert sk.tobytes() == to_host(sk1).tobytes()
    sk_o, S_o, st_o = oracle.grad_sqnorm(g, n_threads=8)
    assert S.hex() == float(S_o).hex() and st_o == lt.LT_STATUS_OK
    assert sk.tobytes() == np.asarray(sk_o, np.float64).tobytes()


def test_nonfinite_part_sets_status():
    rng = np.random.default_rng(72)
    g = _grads(rng, True)
    g[4][777] = 0x7FC0  # NaN in one layer
    gdev = [to_dev(x) for x in g]
    _, _, st = _arrival(gdev, [3, 1, 2, 0], [torch.cuda.current_stream()])
    assert st == lt.LT_STATUS_NONFINITE


@pytest.mark.parametrize("keep", [False, True])
def test_streamed_step_with_norm_ready(keep):
    """norm_ready against the two-pass streamed step and the oracle; with keep_grads
    pass 2 copies the gradients into their resident regions instead of the slots."""
    rng = np.random.default_rng(73)
    block = 2048
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in SIZES]
    base = State.zero_host(w, block)
    for k, n in enumerate(SIZES):
        base.mq[k][:] = rng.integers(-127, 128, size=n)
        base.vq[k][:] = rng.integers(0, 256, size=n)
        base.ma[k][:] = rng.uniform(0.1, 5.0, size=base.ma[k].size) * 1e-3
        base.va[k][:] = rng.uniform(0.1, 5.0, size=base.va[k].size) * 1e-6
    g = _grads(rng, True)
    pin = lambda a: torch.from_numpy(a).pin_memory()

    def host_state():
        return State(*[[pin(a.copy()) for a in lst] for lst in (base.w, base.mq, base.ma,
                                                                base.vq, base.va)])
    g_pin = [torch.from_numpy(x.view(np.int16)).pin_memory().view(torch.bfloat16) for x in g]
    results = []
    for ready in (False, True):
        host = host_state()
        S = torch.zeros(1, dtype=torch.float64, device=DEV)
        status = torch.zeros(1, dtype=torch.int32, device=DEV)
        coef = torch.zeros(1, dtype=torch.float32, device=DEV)
        if ready:
            # the gradients as they arrived on the device during backward
            acc = lt.GradNormAccumulator(SIZES, DEV)
            gdev = [to_dev(x) for x in g]
            for layer in reversed(range(len(LAYERS) - 1)):
                a, b = LAYERS[layer], LAYERS[layer + 1]
                acc.add(a, gdev[a:b])
            acc.finish(S, status)
        lt.lt_streamed_hybrid8bit_adamw_step(host.w, g_pin, host.mq, host.ma, host.vq, host.va,
                                             LAYERS, block, step=2, max_norm=1.0, ring_slots=3,
                                             sq_total=S, coef=coef, status=status,
                                             norm_ready=ready, keep_grads=keep, **HYPER)
        torch.cuda.synchronize()
        results.append((host, to_host(S)[0], to_host(coef)[0]))
    (h0, S0, c0), (h1, S1, c1) = results
    assert S0.hex() == S1.hex() and c0 == c1
    as_np = lambda h: State(*[[t.numpy() for t in lst] for lst in (h.w, h.mq, h.ma, h.vq, h.va)])
    assert_state_equal(as_np(h1), as_np(h0), "norm_ready vs two-pass streamed")
    ref = base.copy()
    _, S_o, st_o = oracle.grad_sqnorm(g, n_threads=8)
    _, c_o = oracle.clip_coef(S_o, 1.0)
    oracle_step(ref, g, block, 2, coef=float(c_o), status=st_o)
    assert_state_equal(as_np(h1), ref, "norm_ready streamed vs oracle")


def test_accumulator_rejects_mismatched_parts():
    acc = lt.GradNormAccumulator(SIZES, DEV)
    with pytest.raises(ValueError):
        acc.add(1, [torch.zeros(5, dtype=torch.bfloat16, device=DEV)])
    with pytest.raises(ValueError):
        acc.add(len(SIZES) - 1, [torch.zeros(5, dtype=torch.bfloat16, device=DEV)] * 2)
