"""The device step state: the step index and bias corrections come from the device,
so Hybrid8bitAdamW enqueues steps without waiting for earlier ones.

* The step entry points with a step state give bitwise the results of the same steps
  with explicit step indices (8-bit at block 2048 and 3072, fp32 states), skips
  included (a skipped step does not count).
* Twenty optimizer steps, some with non-finite gradients, enqueue behind a busy GPU
  without the host waiting, and equal the oracle bitwise (8-bit slice with the
  decade-tree map, fp32 states for the rest).
* The step table grows on the device, and the learning rate may change every step.
* After three skips in a row the device stops: finite steps enqueued behind the
  stop write nothing, and the host raises NonFiniteAbort when it reads the state."""
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, assert_state_equal, to_dev, to_host

pytestmark = pytest.mark.gpu

SIZES = [40000, 300001, 5000, 123457, 2048, 7]


def _grads(rng, sizes, bad=False):
    g = [f32_to_bf16_bits((rng.standard_t(3, size=n) * 1e-2).astype(np.float32)) for n in sizes]
    if bad:
        g[1][11] = 0x7FC0  # NaN
    return g


@pytest.mark.parametrize("block,code_map", [(2048, lt.LT_MAP_LINEAR), (2048, lt.LT_MAP_DYNAMIC),
                                            (3072, lt.LT_MAP_LINEAR)])
def test_step_state_equals_explicit_steps(block, code_map):
    rng = np.random.default_rng(block + code_map)
    w0 = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in SIZES]
    a, b = State.zero_host(w0, block).to_dev(), State.zero_host(w0, block).to_dev()
    m32 = [torch.zeros(n, device=DEV) for n in SIZES]
    v32 = [torch.zeros(n, device=DEV) for n in SIZES]
    wa32 = [to_dev(x) for x in w0]
    wb32, mb32, vb32 = [to_dev(x) for x in w0], [x.clone() for x in m32], [x.clone() for x in v32]
    state = torch.empty(lt.lt_step_state_bytes(16), dtype=torch.uint8, device=DEV)
    lt.lt_step_state_init(state, 16, 0.9, 0.999)
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    t = 0
    for call, bad in enumerate((False, False, True, False, False)):
        g = [to_dev(x) for x in _grads(rng, SIZES, bad)]
        lt.lt_grad_sqnorm(g, S, st)
        lt.lt_clip_coef(S, 1.0, coef)
        lr = 1e-4 * (1 + call)  # a learning rate that changes every step
        h = dict(HYPER, lr=lr)
        lt.lt_hybrid8bit_adamw_step(a.w, g, a.mq, a.ma, a.vq, a.va, block, step=0, coef=coef,
                                    status=st, step_state=state, code_map=code_map, **h)
        lt.lt_adamw_fp32_step(wa32, g, m32, v32, step=0, coef=coef, status=st, step_state=state,
                              **h)
        lt.lt_step_state_advance(state, st)
        if not bad:
            t += 1
        lt.lt_hybrid8bit_adamw_step(b.w, g, b.mq, b.ma, b.vq, b.va, block, step=max(t, 1),
                                    coef=coef, status=st, code_map=code_map, **h)
        lt.lt_adamw_fp32_step(wb32, g, mb32, vb32, step=max(t, 1), coef=coef, status=st, **h)
        torch.cuda.synchronize()
        assert_state_equal(a.to_host(), b.to_host(), f"call {call}")
        for x, y in zip(wa32 + m32 + v32, wb32 + mb32 + vb32):
            assert to_host(x).tobytes() == to_host(y).tobytes(), f"fp32 states, call {call}"
    hdr = state[:28].cpu().numpy()
    assert int(hdr[:8].view(np.int64)[0]) == 4  # applied
    assert int(hdr[16:20].view(np.int32)[0]) == 0 and int(hdr[24:28].view(np.int32)[0]) == 0


def _oracle_opt(ref8, ref32, idx8, idx32, g, t, lr, omap):
    _, S, st = oracle.grad_sqnorm(g, n_threads=8)
    if st != oracle.STATUS_OK:
        return False
    _, c = oracle.clip_coef(S, 1.0)
    h = dict(HYPER, lr=lr)
    oracle.hybrid8bit_adamw_step(ref8.w, [g[i] for i in idx8], ref8.mq, ref8.ma, ref8.vq, ref8.va,
                                 2048, step=t, coef=float(c), status=st, n_threads=8,
                                 code_map=omap, **h)
    for (wr, mr, vr), i in zip(ref32, idx32):
        oracle.adamw_fp32_step(wr, g[i], mr, vr, step=t, coef=float(c), **h)
    return True


def _check_opt(opt, params, ref8, ref32, what):
    got8 = State([to_host(params[i]) for i in opt.idx8], [to_host(x) for x in opt.m_codes],
                 [to_host(x) for x in opt.m_absmax], [to_host(x) for x in opt.v_codes],
                 [to_host(x) for x in opt.v_absmax])
    assert_state_equal(got8, ref8, what)
    for (wr, mr, vr), i, m, v in zip(ref32, opt.idx32, opt.exp_avg, opt.exp_avg_sq):
        assert to_host(params[i]).tobytes() == wr.tobytes(), what
        assert to_host(m).tobytes() == mr.tobytes() and to_host(v).tobytes() == vr.tobytes(), what


def _sleep_cycles_for(ms):
    probe = 10_000_000
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    torch.cuda._sleep(probe)
    b.record()
    b.synchronize()
    return int(min(probe / max(a.elapsed_time(b), 1e-3) * ms, 300 * probe))


def test_twenty_optimizer_steps_run_ahead_of_the_gpu(monkeypatch):
    monkeypatch.setattr(lt.Hybrid8bitAdamW, "TABLE", 8)  # the table grows twice on the way
    rng = np.random.default_rng(61)
    w0 = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in SIZES]
    params = [to_dev(x) for x in w0]
    opt = lt.Hybrid8bitAdamW(params, lr=1e-4, block_size=2048, slice_fraction=0.3)
    assert opt.idx8 and opt.idx32
    ref8 = State.zero_host([w0[i] for i in opt.idx8], 2048)
    ref32 = [(w0[i].copy(), np.zeros_like(w0[i]), np.zeros_like(w0[i])) for i in opt.idx32]
    bad_at = {4, 9, 10, 15}
    gs = [_grads(rng, SIZES, i in bad_at) for i in range(20)]
    gd = [[to_dev(x) for x in g] for g in gs]
    lrs = [1e-4 * (1 + 0.1 * i) for i in range(20)]
    torch.cuda.synchronize()
    done = torch.cuda.Event()
    t0 = time.perf_counter()
    torch.cuda._sleep(_sleep_cycles_for(3000.0))  # the GPU is busy for about three seconds
    for i in range(20):
        opt.lr = lrs[i]
        opt.step(gd[i])
    done.record()
    enqueue_s = time.perf_counter() - t0
    busy = not done.query()
    st = opt.last_status()
    total_s = time.perf_counter() - t0
    print(f"20 steps enqueued in {enqueue_s * 1e3:.1f} ms; done after {total_s * 1e3:.0f} ms",
          flush=True)
    assert busy, "the GPU finished before the host had enqueued the steps"
    assert enqueue_s < 0.5 * total_s
    t = 0
    for i in range(20):
        if _oracle_opt(ref8, ref32, opt.idx8, opt.idx32, gs[i], t + 1, lrs[i], oracle.MAP_DYNAMIC):
            t += 1
    assert st == lt.LT_STATUS_OK and opt.step_count == t == 16 and opt.consecutive_skips == 0
    _check_opt(opt, params, ref8, ref32, "after 20 steps")


def test_device_stop_after_three_skips_without_reading():
    rng = np.random.default_rng(62)
    w0 = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in SIZES]
    params = [to_dev(x) for x in w0]
    opt = lt.Hybrid8bitAdamW(params, lr=1e-4, block_size=2048, code_map=lt.LT_MAP_LINEAR)
    ref8 = State.zero_host(w0, 2048)
    seq = (False, True, True, True, False, False)  # three skips, then two finite steps
    gs = [_grads(rng, SIZES, bad) for bad in seq]
    gd = [[to_dev(x) for x in g] for g in gs]  # (copies from pageable memory wait for the GPU)
    torch.cuda.synchronize()
    torch.cuda._sleep(_sleep_cycles_for(2000.0))  # all six are enqueued before any runs
    for g in gd:
        opt.step(g)
    # only the first step applies: the device stops at the third skip
    _oracle_opt(ref8, [], list(range(len(SIZES))), [], gs[0], 1, 1e-4, oracle.MAP_LINEAR)
    with pytest.raises(lt.NonFiniteAbort) as e:
        opt.last_status()
    assert e.value.skips == 3 and opt.step_count == 1
    _check_opt(opt, params, ref8, [], "stopped")
    with pytest.raises(lt.NonFiniteAbort):
        opt.step([to_dev(x) for x in _grads(rng, SIZES)])
    opt.consecutive_skips = 0  # the caller goes on explicitly
    g = _grads(rng, SIZES)
    opt.step([to_dev(x) for x in g])
    _oracle_opt(ref8, [], list(range(len(SIZES))), [], g, 2, 1e-4, oracle.MAP_LINEAR)
    assert opt.last_status() == lt.LT_STATUS_OK and opt.step_count == 2
    _check_opt(opt, params, ref8, [], "after going on")
