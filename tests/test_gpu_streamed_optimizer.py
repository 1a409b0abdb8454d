"""StreamedHybrid8bitAdamW, the optimizer object of the layer-streamed step, against the
oracle: host weights and 8-bit states bitwise after each of several steps from zero
state (gradients kept in HBM between the passes, and copied in twice), a skipped
non-finite step that changes nothing and does not advance the step count, the abort
after three consecutive skips, and a checkpoint that resumes bitwise."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
import synth
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, assert_state_equal, oracle_step

pytestmark = pytest.mark.gpu

BLOCK = 2048


def _model(seed):
    rng = np.random.default_rng(seed)
    layer = [int(np.prod(s)) for s in synth.layer_shapes(256, 704, 4, 2, 64)]
    numels = 3 * layer + [7, 2049, 100003]
    first = list(range(0, 3 * len(layer) + 1, len(layer))) + [3 * len(layer) + 3]
    w0 = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in numels]
    return rng, numels, first, w0


def _grads(rng, numels, bad=False):
    g = [f32_to_bf16_bits((rng.standard_t(3, size=n) * 1e-3).astype(np.float32)) for n in numels]
    if bad:
        g[len(g) // 2][5] = 0x7FC0  # NaN
    return g, [torch.from_numpy(x.view(np.int16)).pin_memory().view(torch.bfloat16) for x in g]


def _host_state(params, opt):
    as_np = lambda ts: [t.numpy() for t in ts]
    return State(as_np(params), as_np(opt.m_codes), as_np(opt.m_absmax), as_np(opt.v_codes),
                 as_np(opt.v_absmax))


@pytest.mark.parametrize("keep", [True, False])
def test_steps_and_skip_against_oracle(keep):
    rng, numels, first, w0 = _model(81)
    params = [torch.from_numpy(x.copy()).pin_memory() for x in w0]
    opt = lt.StreamedHybrid8bitAdamW(params, first, DEV, lr=HYPER["lr"], betas=(0.9, 0.999),
                                     eps=HYPER["eps"], weight_decay=HYPER["weight_decay"],
                                     block_size=BLOCK, keep_grads=keep,
                                     code_map=lt.LT_MAP_LINEAR)
    ref = State.zero_host(w0, BLOCK)
    t = 0
    for call, bad in enumerate((False, True, False, False)):
        g, g_pin = _grads(rng, numels, bad)
        st = opt.step(g_pin)
        _, S, st_o = oracle.grad_sqnorm(g, n_threads=8)
        assert st == st_o, f"call {call}"
        if st_o == lt.LT_STATUS_OK:
            t += 1
            _, c = oracle.clip_coef(S, 1.0)
            oracle_step(ref, g, BLOCK, t, coef=float(c), status=st_o)
        assert opt.step_count == t
        assert_state_equal(_host_state(params, opt), ref, f"call {call}, keep {keep}")


def test_abort_after_three_consecutive_skips_and_checkpoint():
    rng, numels, first, w0 = _model(82)
    params = [torch.from_numpy(x.copy()).pin_memory() for x in w0]
    opt = lt.StreamedHybrid8bitAdamW(params, first, DEV, lr=1e-4, block_size=BLOCK)
    assert opt.step(_grads(rng, numels)[1]) == lt.LT_STATUS_OK
    # checkpoint after one step, then two more steps here
    saved = opt.state_dict()
    saved_w = [p.clone() for p in params]
    later = [_grads(rng, numels)[1] for _ in range(2)]
    for g in later:
        assert opt.step(g) == lt.LT_STATUS_OK
    # a fresh optimizer restored from the checkpoint continues bitwise
    params2 = [w.pin_memory() for w in saved_w]
    opt2 = lt.StreamedHybrid8bitAdamW(params2, first, DEV, lr=1e-4, block_size=BLOCK)
    opt2.load_state_dict(saved)
    for g in later:
        assert opt2.step(g) == lt.LT_STATUS_OK
    assert opt2.step_count == opt.step_count == 3
    assert_state_equal(_host_state(params2, opt2), _host_state(params, opt), "resumed")
    # three non-finite steps in a row: the third raises, nothing changes
    before = _host_state(params, opt).copy()
    assert opt.step(_grads(rng, numels, bad=True)[1]) == lt.LT_STATUS_NONFINITE
    assert opt.step(_grads(rng, numels, bad=True)[1]) == lt.LT_STATUS_NONFINITE
    with pytest.raises(lt.NonFiniteAbort):
        opt.step(_grads(rng, numels, bad=True)[1])
    with pytest.raises(lt.NonFiniteAbort):
        opt.step(_grads(rng, numels)[1])
    assert opt.step_count == 3
    assert_state_equal(_host_state(params, opt), before, "after skipped steps")
