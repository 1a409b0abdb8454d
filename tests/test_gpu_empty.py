"""Empty inputs through the C ABI: an empty tensor list and zero-element tensors
inside lists.  An empty tensor contributes a zero sum of squares and is not
stepped; every other result is bitwise what the oracle computes on the same
list (which, by the same definition, is the list without the empty tensors)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, assert_state_equal, gpu_norm_and_coef, to_dev, to_host

pytestmark = pytest.mark.gpu


def _grads(rng, sizes):
    return [f32_to_bf16_bits((rng.standard_normal(n) * 1e-2).astype(np.float32)) for n in sizes]


def _random_state(rng, sizes, block):
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    st = State.zero_host(w, block)
    for k, n in enumerate(sizes):
        st.mq[k][:] = rng.integers(-127, 128, size=n)
        st.vq[k][:] = rng.integers(0, 256, size=n)
        st.ma[k][:] = rng.uniform(0.1, 5.0, size=st.ma[k].size) * 1e-3
        st.va[k][:] = rng.uniform(0.1, 5.0, size=st.va[k].size) * 1e-6
    return st


def test_sqnorm_of_an_empty_list_is_zero():
    S = torch.full((1,), 7.0, dtype=torch.float64, device=DEV)
    status = torch.full((1,), 9, dtype=torch.int32, device=DEV)
    lt.lt_grad_sqnorm([], S, status)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    norm = torch.full((1,), 3.0, dtype=torch.float32, device=DEV)
    lt.lt_clip_coef(S, 1.0, coef, total_norm=norm)
    torch.cuda.synchronize()
    assert S.item() == 0.0 and status.item() == lt.LT_STATUS_OK
    assert norm.item() == 0.0 and coef.item() == 1.0


@pytest.mark.parametrize("sizes", [[0], [0, 0, 0], [5000, 0, 8193], [0, 1, 0, 100003, 0]])
def test_sqnorm_with_empty_tensors(sizes):
    rng = np.random.default_rng(sum(sizes) + len(sizes))
    grads = _grads(rng, sizes)
    sk_o, S_o, st_o = oracle.grad_sqnorm(grads)
    sk, S, status, _, _ = gpu_norm_and_coef([to_dev(g) for g in grads], 1.0)
    torch.cuda.synchronize()
    assert to_host(sk).tobytes() == sk_o.tobytes()
    assert S.item() == S_o and status.item() == st_o
    for k, n in enumerate(sizes):
        if n == 0:
            assert to_host(sk)[k] == 0.0
    # dropping the empty tensors changes nothing: adding +0.0 is exact
    _, S_ne, _ = oracle.grad_sqnorm([g for g in grads if g.size])
    assert S.item() == S_ne


def test_norm_accumulated_by_parts_with_empty_tensors():
    rng = np.random.default_rng(3)
    sizes = [0, 9000, 0, 0, 20000, 0]
    grads = [to_dev(g) for g in _grads(rng, sizes)]
    _, S_ref, st_ref = oracle.grad_sqnorm([to_host(g) for g in grads])
    acc = lt.GradNormAccumulator(sizes, DEV)
    acc.add(4, grads[4:])          # parts in any order, some of them all-empty
    acc.add(2, grads[2:4])
    acc.add(0, grads[0:2])
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    status = torch.full((1,), 5, dtype=torch.int32, device=DEV)
    acc.finish(S, status)
    torch.cuda.synchronize()
    assert S.item() == S_ref and status.item() == st_ref
    # a model whose every tensor is empty has no chunks at all
    empty = lt.GradNormAccumulator([0, 0], DEV)
    empty.add(0, grads[0:1])
    empty.finish(S, status)
    torch.cuda.synchronize()
    assert S.item() == 0.0 and status.item() == lt.LT_STATUS_OK


@pytest.mark.parametrize("block", [256, 2048])
def test_step_with_empty_tensors(block):
    rng = np.random.default_rng(block)
    sizes = [0, 3 * block + 5, 0, 1, 70001, 0]
    grads = _grads(rng, sizes)
    ref = _random_state(rng, sizes, block)
    dev = ref.to_dev()
    wb = [torch.full((n,), 0x7FC0, dtype=torch.int16, device=DEV).view(torch.bfloat16)
          for n in sizes]
    _, S, st = oracle.grad_sqnorm(grads)
    _, c = oracle.clip_coef(S, 1.0)
    oracle.hybrid8bit_adamw_step(ref.w, grads, ref.mq, ref.ma, ref.vq, ref.va, block, step=3,
                                 coef=float(c), status=st, **HYPER)
    _, _, status, _, coef = gpu_norm_and_coef([to_dev(g) for g in grads], 1.0)
    lt.lt_hybrid8bit_adamw_step(dev.w, [to_dev(g) for g in grads], dev.mq, dev.ma, dev.vq,
                                dev.va, block, step=3, coef=coef, status=status, params_bf16=wb,
                                **HYPER)
    torch.cuda.synchronize()
    assert_state_equal(dev.to_host(), ref, f"empty tensors, block {block}")
    for k, n in enumerate(sizes):
        if n:
            assert to_host(wb[k]).tobytes() == oracle.round_bf16(ref.w[k]).tobytes()


def test_step_of_an_empty_list_does_nothing():
    lt.lt_hybrid8bit_adamw_step([], [], [], [], [], [], 2048, step=1, **HYPER)
    lt.lt_adamw_fp32_step([], [], [], [], step=1, **HYPER)
    e = torch.zeros(0, dtype=torch.float32, device=DEV)
    lt.lt_hybrid8bit_adamw_step([e], [e], [torch.zeros(0, dtype=torch.int8, device=DEV)],
                                [e], [torch.zeros(0, dtype=torch.uint8, device=DEV)], [e],
                                2048, step=1, **HYPER)
    torch.cuda.synchronize()


def test_fp32_state_step_with_empty_tensors():
    rng = np.random.default_rng(11)
    sizes = [0, 4097, 0, 33]
    grads = [(rng.standard_normal(n) * 1e-2).astype(np.float32) for n in sizes]
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    m = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in sizes]
    v = [(rng.uniform(0, 1, n) * 1e-6).astype(np.float32) for n in sizes]
    dw, dm, dv = [to_dev(x) for x in w], [to_dev(x) for x in m], [to_dev(x) for x in v]
    lt.lt_adamw_fp32_step(dw, [to_dev(g) for g in grads], dm, dv, step=4, **HYPER)
    torch.cuda.synchronize()
    for k in range(len(sizes)):
        oracle.adamw_fp32_step(w[k], grads[k], m[k], v[k], step=4, coef=1.0, **HYPER)
        for a, b in ((dw[k], w[k]), (dm[k], m[k]), (dv[k], v[k])):
            assert to_host(a).tobytes() == b.tobytes()


def test_optimizer_object_with_an_empty_parameter():
    rng = np.random.default_rng(21)
    sizes = [5000, 0, 4096 * 2 + 3]
    w0 = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    params = [to_dev(x) for x in w0]
    opt = lt.Hybrid8bitAdamW(params, lr=1e-5, block_size=4096, code_map=lt.LT_MAP_LINEAR)
    ref = State.zero_host(w0, 4096)
    for t in (1, 2):
        g = _grads(rng, sizes)
        opt.step([to_dev(x) for x in g])
        assert opt.last_status() == lt.LT_STATUS_OK
        _, S, st = oracle.grad_sqnorm(g)
        _, c = oracle.clip_coef(S, 1.0)
        oracle.hybrid8bit_adamw_step(ref.w, g, ref.mq, ref.ma, ref.vq, ref.va, 4096, step=t,
                                     coef=float(c), status=st, **dict(HYPER, lr=1e-5))
    got = State([to_host(p) for p in params], [to_host(x) for x in opt.m_codes],
                [to_host(x) for x in opt.m_absmax], [to_host(x) for x in opt.v_codes],
                [to_host(x) for x in opt.v_absmax])
    assert_state_equal(got, ref, "Hybrid8bitAdamW with an empty parameter")


def test_streamed_layer_with_empty_tensors():
    rng = np.random.default_rng(31)
    block = 2048
    sizes = [0, 9000, 0, 12345, 0, 0, 4096]   # layers: [0, 9000, 0] [12345, 0] [0] [4096]
    first = [0, 3, 5, 6, 7]
    grads = _grads(rng, sizes)
    ref = _random_state(rng, sizes, block)
    # empty host arrays stay unpinned: the library never touches them
    pin = lambda a: torch.from_numpy(a).pin_memory() if a.size else torch.from_numpy(a)
    host = State(*[[pin(a.copy()) for a in lst] for lst in (ref.w, ref.mq, ref.ma, ref.vq, ref.va)])
    _, S_o, st_o = oracle.grad_sqnorm(grads)
    _, c = oracle.clip_coef(S_o, 1.0)
    oracle.hybrid8bit_adamw_step(ref.w, grads, ref.mq, ref.ma, ref.vq, ref.va, block, step=2,
                                 coef=float(c), status=st_o, **HYPER)
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    lt.lt_streamed_hybrid8bit_adamw_step(host.w, [pin(g.view(np.int16)) for g in grads], host.mq,
                                         host.ma, host.vq, host.va, first, block, step=2,
                                         max_norm=1.0, ring_slots=2, sq_total=S, coef=coef,
                                         status=status, **HYPER)
    torch.cuda.synchronize()
    assert S.item() == S_o and coef.item() == c and status.item() == st_o
    got = State(*[[t.numpy() for t in lst] for lst in (host.w, host.mq, host.ma, host.vq, host.va)])
    assert_state_equal(got, ref, "streamed, empty tensors")


def test_optimizer_rejects_mismatched_gradients_before_any_work():
    params = [torch.zeros(300, dtype=torch.float32, device=DEV),
              torch.zeros(0, dtype=torch.float32, device=DEV)]
    opt = lt.Hybrid8bitAdamW(params, block_size=256)
    g = torch.zeros(300, dtype=torch.bfloat16, device=DEV)
    e = torch.zeros(0, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(ValueError, match="one gradient per parameter"):
        opt.step([g])
    with pytest.raises(ValueError, match="is None"):
        opt.step([g, None])
    with pytest.raises(ValueError, match="elements"):
        opt.step([g[:299], e])
    assert opt.step_count == 0
    opt.step([g, e])
    assert opt.last_status() == lt.LT_STATUS_OK and opt.step_count == 1


def test_overlapping_tensors_are_rejected_before_launch():
    buf = torch.zeros(3 * 4096, dtype=torch.float32, device=DEV)
    g = torch.zeros(4096, dtype=torch.bfloat16, device=DEV)
    mq = torch.zeros(2 * 4096, dtype=torch.int8, device=DEV)
    vq = torch.zeros(4096, dtype=torch.uint8, device=DEV)
    ma = torch.zeros(4, dtype=torch.float32, device=DEV)
    va = torch.zeros(4, dtype=torch.float32, device=DEV)
    # two parameters sharing 4 KB
    with pytest.raises(lt.LazyTrainError, match="overlap") as e:
        lt.lt_hybrid8bit_adamw_step([buf[:4096], buf[3072:3072 + 4096]], [g, g],
                                    [mq[:4096], mq[4096:]], [ma[:2], ma[2:]],
                                    [vq, torch.zeros(4096, dtype=torch.uint8, device=DEV)],
                                    [va[:2], va[2:]], 2048, step=1, **HYPER)
    assert e.value.code == 1  # LT_ERR_INVALID_ARG
    # a written array inside a gradient
    with pytest.raises(lt.LazyTrainError, match="overlap"):
        lt.lt_hybrid8bit_adamw_step([buf[:4096]], [buf[4096:8192]], [mq[:4096]], [ma[:2]], [vq],
                                    [buf[4096:4098]], 2048, step=1, **HYPER)
    # the same gradient for two tensors is fine (only read)
    lt.lt_hybrid8bit_adamw_step([buf[:4096], buf[4096:8192]], [g, g], [mq[:4096], mq[4096:]],
                                [ma[:2], ma[2:]],
                                [vq, torch.zeros(4096, dtype=torch.uint8, device=DEV)],
                                [va[:2], va[2:]], 2048, step=1, **HYPER)
    # fp32-state step: exp_avg sharing bytes with exp_avg_sq
    m = torch.zeros(8192, dtype=torch.float32, device=DEV)
    with pytest.raises(lt.LazyTrainError, match="overlap"):
        lt.lt_adamw_fp32_step([buf[:4096]], [g], [m[:4096]], [m[2048:6144]], step=1, **HYPER)
    torch.cuda.synchronize()
