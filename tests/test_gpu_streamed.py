"""The layer-streamed step (host-resident state passing through a ring of device
slots) against the resident HIP path and the oracle on the same data: norm,
coefficient, weights, codes and scales bitwise, for 2 and 3 slots, separate and
shared streams, gradients kept in HBM between the passes or copied in twice, two
consecutive steps, ragged layers and the non-finite skip."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
import synth
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, assert_state_equal, gpu_norm_and_coef, gpu_step, \
    oracle_step, to_dev, to_host

pytestmark = pytest.mark.gpu


def _model(seed):
    """Six small decoder layers plus one ragged layer, bf16 gradients, random states."""
    rng = np.random.default_rng(seed)
    layer = [int(np.prod(s)) for s in synth.layer_shapes(256, 704, 4, 2, 64)]
    numels = 6 * layer + [1, 7, 2049, 100003]
    first = list(range(0, 6 * len(layer) + 1, len(layer))) + [6 * len(layer) + 4]
    return rng, numels, first


def _random_state(rng, numels, block):
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in numels]
    st = State.zero_host(w, block)
    for k, n in enumerate(numels):
        st.mq[k][:] = rng.integers(-127, 128, size=n)
        st.vq[k][:] = rng.integers(0, 256, size=n)
        st.ma[k][:] = rng.uniform(0.1, 5.0, size=st.ma[k].size) * 1e-3
        st.va[k][:] = rng.uniform(0.1, 5.0, size=st.va[k].size) * 1e-6
    return st


def _pinned(st: State):
    pin = lambda a: torch.from_numpy(a).pin_memory()
    return State(*[[pin(a) for a in lst] for lst in (st.w, st.mq, st.ma, st.vq, st.va)])


def _host_np(st: State):
    return State(*[[t.numpy().copy() for t in lst] for lst in (st.w, st.mq, st.ma, st.vq, st.va)])


def _streamed(host: State, grads_pinned, first, block, t, slots, streams, max_norm=1.0,
              keep_grads=False):
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    norm = torch.zeros(1, dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    cs, hs, ds = streams
    if cs is not None:
        cs.wait_stream(torch.cuda.current_stream())  # the outputs above are zeroed there
    lt.lt_streamed_hybrid8bit_adamw_step(host.w, grads_pinned, host.mq, host.ma, host.vq, host.va,
                                         first, block, step=t, max_norm=max_norm,
                                         ring_slots=slots, sq_total=S, coef=coef, status=status,
                                         total_norm=norm, compute_stream=cs, h2d_stream=hs,
                                         d2h_stream=ds, keep_grads=keep_grads, **HYPER)
    (cs or torch.cuda.current_stream()).synchronize()
    return to_host(S)[0], to_host(coef)[0], int(to_host(status)[0])


@pytest.mark.parametrize("slots,separate,keep", [(3, True, False), (2, True, False),
                                                  (3, False, False), (3, True, True),
                                                  (2, False, True)])
@pytest.mark.parametrize("block", [2048, 256])
def test_streamed_equals_resident_and_oracle(slots, separate, keep, block):
    rng, numels, first = _model(slots * 10 + block + keep)
    base = _random_state(rng, numels, block)
    streams = (torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()) if separate else \
        (None, None, None)
    host = _pinned(base)
    ref = base.copy()
    dev = base.to_dev()
    for t in (3, 4):  # two consecutive calls reuse the slots and events
        g = [f32_to_bf16_bits((rng.standard_t(3, size=n) * 1e-3).astype(np.float32))
             for n in numels]
        g_pin = [torch.from_numpy(x.view(np.int16)).pin_memory().view(torch.bfloat16) for x in g]
        S_s, coef_s, st_s = _streamed(host, g_pin, first, block, t, slots, streams,
                                      keep_grads=keep)
        # resident path on the same data
        gdev = [to_dev(x) for x in g]
        _, S_r, status_r, _, coef_r = gpu_norm_and_coef(gdev, 1.0)
        gpu_step(dev, gdev, block, t, coef=coef_r, status=status_r)
        torch.cuda.synchronize()
        assert st_s == lt.LT_STATUS_OK
        assert S_s.hex() == to_host(S_r)[0].hex() and coef_s == to_host(coef_r)[0]
        # oracle
        _, S_o, st_o = oracle.grad_sqnorm(g, n_threads=8)
        _, c_o = oracle.clip_coef(S_o, 1.0)
        oracle_step(ref, g, block, t, coef=float(c_o), status=st_o)
        assert S_s.hex() == S_o.hex() and coef_s == c_o
        got = _host_np(host)
        assert_state_equal(got, dev.to_host(), f"streamed vs resident, t={t}")
        assert_state_equal(got, ref, f"streamed vs oracle, t={t}")


@pytest.mark.parametrize("keep", [False, True])
def test_streamed_skips_nonfinite_and_no_clip(keep):
    rng, numels, first = _model(5)
    base = _random_state(rng, numels, 2048)
    host = _pinned(base)
    g = [f32_to_bf16_bits((rng.standard_normal(n) * 1e-3).astype(np.float32)) for n in numels]
    g[20][3] = 0x7FC0  # NaN in bf16
    g_pin = [torch.from_numpy(x.view(np.int16)).pin_memory().view(torch.bfloat16) for x in g]
    _, _, st = _streamed(host, g_pin, first, 2048, 2, 3, (None, None, None), keep_grads=keep)
    assert st == lt.LT_STATUS_NONFINITE
    assert_state_equal(_host_np(host), base, "skipped streamed step")
    # max_norm = inf: no clipping, equal to the oracle step without a coefficient
    g[20][3] = 0
    g_pin = [torch.from_numpy(x.view(np.int16)).pin_memory().view(torch.bfloat16) for x in g]
    _, coef, st = _streamed(host, g_pin, first, 2048, 2, 3, (None, None, None), max_norm=math.inf,
                            keep_grads=keep)
    assert st == lt.LT_STATUS_OK and coef == np.float32(1.0)
    ref = base.copy()
    oracle_step(ref, g, 2048, 2)
    assert_state_equal(_host_np(host), ref, "streamed without clipping")


def test_streamed_rejects_bad_layers():
    w = torch.zeros(10).pin_memory()
    g = torch.zeros(10, dtype=torch.bfloat16).pin_memory()
    q = torch.zeros(10, dtype=torch.int8).pin_memory()
    u = torch.zeros(10, dtype=torch.uint8).pin_memory()
    a = torch.zeros(1).pin_memory()
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    c = torch.zeros(1, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    with pytest.raises(ValueError):
        lt.lt_streamed_hybrid8bit_adamw_step([w], [g], [q], [a], [u], [a], [0, 2], 2048,
                                             step=1, max_norm=1.0, ring_slots=3, sq_total=S,
                                             coef=c, status=st, **HYPER)
    with pytest.raises(ValueError):
        lt.lt_streamed_hybrid8bit_adamw_step([w], [g], [q], [a], [u], [a], [0, 1], 2048,
                                             step=1, max_norm=1.0, ring_slots=1, sq_total=S,
                                             coef=c, status=st, **HYPER)
