"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the same
seeded inputs.  The bar is bitwise equality for the norm, the coefficient, the
weights, the codes and the scales; the stated tolerances (weights 1e-6 relative,
codes +-1 at ties with rate <= 1e-6) are checked as well."""
import ctypes
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
import synth
from golden_io import adamw_examples, dense, f32_to_bf16_bits, sqnorm_cases
from gpu_helpers import (DEV, HYPER, State, assert_state_equal, check_stated_tolerance,
                         golden_eps, gpu_norm_and_coef, gpu_step, oracle_step, to_dev, to_host)

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


@pytest.fixture(autouse=True)
def _reset_grid():
    lt.lt_set_max_workgroups(0)
    yield
    lt.lt_set_max_workgroups(0)
    torch.cuda.synchronize()


# ------------------------------------------------------------ a1-a3: norm, clip

def _sq_parity(host_grads, max_norm=1.0):
    dev = [to_dev(g) for g in host_grads]
    sk, S, status, norm, coef = gpu_norm_and_coef(dev, max_norm)
    rsk, rS, rst = oracle.grad_sqnorm(host_grads, n_threads=8)
    rnorm, rcoef = oracle.clip_coef(rS, max_norm)
    assert to_host(sk).tobytes() == rsk.tobytes()
    assert to_host(S)[0].hex() == rS.hex()
    assert int(to_host(status)[0]) == rst
    assert to_host(norm)[0].tobytes() == rnorm.tobytes()
    assert to_host(coef)[0].tobytes() == rcoef.tobytes()
    return rS


@pytest.mark.parametrize("wid", [0, 1])
def test_sqnorm_and_clip_workloads(wid):
    w = synth.WORKLOADS[wid]()
    _say(f"sqnorm parity on {w.name}")
    grads = [w.grads(k, synth.grad_stream(w.step)) for k in range(len(w.shapes))]
    S = _sq_parity(grads, w.max_norm)
    assert S > 0


@pytest.mark.parametrize("as_bf16", [False, True])
def test_sqnorm_ragged_lists(as_bf16):
    rng = np.random.default_rng(31)
    sizes = [1, 7, 8, 9, 255, 2047, 2049, 8191, 8192, 8193, 5120, 3 * 8192 + 17, 300001, 65536]
    grads = []
    for n in sizes:
        x = (rng.standard_t(3, size=n) * 1e-3).astype(np.float32)
        grads.append(f32_to_bf16_bits(x) if as_bf16 else x)
    _sq_parity(grads)


@pytest.mark.parametrize("as_bf16", [False, True])
def test_sqnorm_hand_derived_order_cases(as_bf16):
    for name, tensors, expect_sk, expect_s in sqnorm_cases():
        arrays = [dense(n, vals) for n, vals in tensors]
        if as_bf16:
            arrays = [f32_to_bf16_bits(a) for a in arrays]
        dev = [to_dev(a) for a in arrays]
        sk, S, status, _, _ = gpu_norm_and_coef(dev, 1.0)
        assert to_host(sk).tolist() == expect_sk, name
        assert to_host(S)[0].hex() == expect_s.hex(), name


def test_sqnorm_grid_size_does_not_change_bits():
    w = synth.layer_3b()
    dev = [to_dev(w.grads(k, 4)) for k in range(len(w.shapes))]
    results = []
    for cap in (0, 1, 7, 300):
        lt.lt_set_max_workgroups(cap)
        sk, S, _, _, coef = gpu_norm_and_coef(dev, 1.0)
        results.append((to_host(sk).tobytes(), to_host(S).tobytes(), to_host(coef).tobytes()))
    assert all(r == results[0] for r in results)


@pytest.mark.parametrize("bad", [math.inf, -math.inf, math.nan])
def test_sqnorm_nonfinite_status(bad):
    x = np.full(20000, 1e-3, np.float32)
    x[12345] = bad
    dev = [to_dev(np.ones(10, np.float32)), to_dev(x)]
    _, S, status, _, _ = gpu_norm_and_coef(dev, 1.0)
    assert lt.lt_read_status(status) == lt.LT_STATUS_NONFINITE
    assert not math.isfinite(to_host(S)[0])


def test_sqnorm_repeated_calls_on_one_workspace():
    """Forty calls on one workspace alternate between a list of 1500 tensors (the
    total reads S_k in two batches of at most 1024) and one of 2 tensors: repeats of
    a list reuse the descriptors already in the workspace, each switch uploads new
    ones.  Every S_k and S stays bitwise the oracle's."""
    rng = np.random.default_rng(77)
    lists = [[(rng.standard_normal(int(n)) * 1e-2).astype(np.float32)
              for n in rng.integers(1, 3000, size=1500)],
             [(rng.standard_normal(n) * 1e-2).astype(np.float32) for n in (70000, 9)]]
    refs = [oracle.grad_sqnorm(h, n_threads=8) for h in lists]
    devs = [[to_dev(a) for a in h] for h in lists]
    ws = torch.empty(max(lt.lt_grad_sqnorm_workspace_bytes([a.size for a in h]) for h in lists),
                     dtype=torch.uint8, device=DEV)
    try:
        for i in range(40):
            j = (i // 3) % 2  # three calls per list, then switch
            K = len(devs[j])
            sk = torch.empty(K, dtype=torch.float64, device=DEV)
            S = torch.empty(1, dtype=torch.float64, device=DEV)
            status = torch.empty(1, dtype=torch.int32, device=DEV)
            lt.lt_grad_sqnorm(devs[j], S, status, sq_per_tensor=sk, workspace=ws)
            rsk, rS, rst = refs[j]
            assert to_host(sk).tobytes() == rsk.tobytes(), f"call {i}"
            assert to_host(S)[0].hex() == rS.hex(), f"call {i}"
            assert int(to_host(status)[0]) == rst, f"call {i}"
    finally:
        torch.cuda.synchronize()
        lt.lt_workspace_release(ws)


def test_sqnorm_subnormal_gradients():
    x = np.full(4097, np.float32(2.0 ** -140), np.float32)
    _sq_parity([x])


def test_clip_coef_many_values():
    rng = np.random.default_rng(5)
    values = list(10.0 ** rng.uniform(-300, 300, size=400)) + list(rng.uniform(0, 4, size=200))
    values += [0.0, 1.0, 4.0, 0.25, 2.0 ** -298, 2.0 ** -300, 1e-320, 1.0 + 2.0 ** -52,
               1.3407807929942596e154 ** 2 / 4, 1.1579208923731620e77, 1.157920892373162e77 * 2,
               math.inf, math.nan]
    # exact squares of fp32 midpoints and their neighbours (ties of the rounding)
    for f in rng.uniform(1e-3, 1e3, size=50).astype(np.float32):
        mid = float(f) + 0.5 * float(np.spacing(f))
        values += [mid * mid, np.nextafter(mid * mid, 0.0), np.nextafter(mid * mid, np.inf)]
    S = torch.empty(1, dtype=torch.float64, device=DEV)
    norm = torch.empty(1, dtype=torch.float32, device=DEV)
    coef = torch.empty(1, dtype=torch.float32, device=DEV)
    for max_norm in (1.0, 0.37, math.inf):
        for v in values:
            S.fill_(v)
            lt.lt_clip_coef(S, max_norm, coef, total_norm=norm)
            rn, rc = oracle.clip_coef(v, max_norm)
            gn, gc = to_host(norm)[0], to_host(coef)[0]
            assert gn.tobytes() == rn.tobytes(), (v, gn, rn)
            assert gc.tobytes() == rc.tobytes(), (v, max_norm, gc, rc)


# ------------------------------------------------------------- a4-a10: the step

def _prior_step_state(weights, prior, block):
    """Both sides' initial states: one step from zero state at t = 1 with lr = 0."""
    ref = State.zero_host(weights, block)
    oracle_step(ref, prior, block, 1, lr=0.0)
    dev = State.zero_host(weights, block).to_dev()
    gpu_step(dev, [to_dev(g) for g in prior], block, 1, lr=0.0)
    assert_state_equal(dev.to_host(), ref, "prior-step initial state")
    return ref, dev


@pytest.mark.parametrize("wid", [0, 1])
def test_workload_step_parity(wid):
    w = synth.WORKLOADS[wid]()
    K, B = len(w.shapes), w.block_size
    _say(f"step parity on {w.name}: {w.n_params} params, block {B}")
    weights = [w.weights(k) for k in range(K)]
    prior = [w.prior_grads(k) for k in range(K)]
    grads = [w.grads(k, synth.grad_stream(w.step)) for k in range(K)]
    ref, dev = _prior_step_state(weights, prior, B)

    rsk, rS, rst = oracle.grad_sqnorm(grads, n_threads=8)
    _, rcoef = oracle.clip_coef(rS, w.max_norm)
    assert rcoef < 1.0 or wid == 1  # clipping is active on the tiny workload
    oracle_step(ref, grads, B, w.step, coef=float(rcoef), status=rst)

    gdev = [to_dev(g) for g in grads]
    sk, S, status, norm, coef = gpu_norm_and_coef(gdev, w.max_norm)
    gpu_step(dev, gdev, B, w.step, coef=coef, status=status)
    got = dev.to_host()
    assert to_host(S)[0].hex() == rS.hex()
    assert to_host(coef)[0].tobytes() == rcoef.tobytes()
    assert_state_equal(got, ref, w.name)
    check_stated_tolerance(got, ref, HYPER["lr"])


def _random_state(sizes, block, rng, zero_frac=0.1):
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    st = State.zero_host(w, block)
    for k, n in enumerate(sizes):
        st.mq[k][:] = rng.integers(-127, 128, size=n)
        st.vq[k][:] = rng.integers(0, 256, size=n)
        nb = st.ma[k].size
        st.ma[k][:] = rng.uniform(0.1, 5.0, size=nb) * 1e-3
        st.va[k][:] = rng.uniform(0.1, 5.0, size=nb) * 1e-6
        z = rng.random(nb) < zero_frac
        st.ma[k][z] = 0
        st.va[k][z] = 0
    return st


SIZES = [1, 7, 8, 63, 64, 65, 200, 2047, 2048, 2049, 4095, 5120, 8193, 20000, 100003]


@pytest.mark.parametrize("block", [64, 128, 256, 512, 1024, 2048, 4096, 8192])
@pytest.mark.parametrize("as_bf16", [False, True])
def test_step_every_block_size_ragged(block, as_bf16):
    rng = np.random.default_rng(block + (7 if as_bf16 else 0))
    ref = _random_state(SIZES, block, rng)
    dev = ref.to_dev()
    g32 = [(rng.standard_t(3, size=n) * 1e-3).astype(np.float32) for n in SIZES]
    grads = [f32_to_bf16_bits(g) for g in g32] if as_bf16 else g32
    oracle_step(ref, grads, block, 3, coef=0.625)
    c = torch.tensor([0.625], dtype=torch.float32, device=DEV)
    gpu_step(dev, [to_dev(g) for g in grads], block, 3, coef=c)
    assert_state_equal(dev.to_host(), ref, f"block {block}")


def test_step_hand_worked_examples():
    """The exact blocks of tests/golden (block size 4 there): each 4-element block is a
    tensor of its own, which is one partial block at the GPU's block size 64.  Examples
    worked with eps = 0 run with the smallest positive eps (golden_eps); eps = 0 itself
    is rejected by the library."""
    for ex in adamw_examples():
        eps = golden_eps(ex)
        n, b = ex["w"].size, ex["block_size"]
        for lo in range(0, n, b):
            hi = min(n, lo + b)
            blk = lo // b
            st = State([ex["w"][lo:hi].copy()], [ex["m_codes"][lo:hi].copy()],
                       [ex["m_absmax"][blk:blk + 1].copy()], [ex["v_codes"][lo:hi].copy()],
                       [ex["v_absmax"][blk:blk + 1].copy()]).to_dev()
            c = torch.tensor([ex["coef"]], dtype=torch.float32, device=DEV)
            if ex["eps"] == 0:
                with pytest.raises(lt.LazyTrainError) as e:
                    gpu_step(st, [to_dev(ex["grad"][lo:hi].copy())], 64, ex["t"], coef=c,
                             lr=ex["lr"], beta1=ex["beta1"], beta2=ex["beta2"], eps=0.0,
                             weight_decay=ex["weight_decay"])
                assert e.value.code == lt.LT_ERR_INVALID_ARG
            gpu_step(st, [to_dev(ex["grad"][lo:hi].copy())], 64, ex["t"], coef=c, lr=ex["lr"],
                     beta1=ex["beta1"], beta2=ex["beta2"], eps=eps,
                     weight_decay=ex["weight_decay"])
            got = st.to_host()
            assert np.array_equal(got.w[0], ex["expect_w"][lo:hi]), ex["name"]
            assert np.array_equal(got.mq[0], ex["expect_m_codes"][lo:hi]), ex["name"]
            assert np.array_equal(got.vq[0], ex["expect_v_codes"][lo:hi]), ex["name"]
            assert got.ma[0][0] == ex["expect_m_absmax"][blk], ex["name"]
            assert got.va[0][0] == ex["expect_v_absmax"][blk], ex["name"]


def test_step_skip_on_nonfinite_and_no_clip_paths():
    rng = np.random.default_rng(8)
    sizes = [3000, 70001]
    ref = _random_state(sizes, 2048, rng)
    g = [f32_to_bf16_bits((rng.standard_normal(n) * 1e-3).astype(np.float32)) for n in sizes]
    g[1][5] = 0x7F80  # +inf in bf16
    gdev = [to_dev(x) for x in g]
    dev = ref.to_dev()
    sk, S, status, norm, coef = gpu_norm_and_coef(gdev, 1.0)
    gpu_step(dev, gdev, 2048, 2, coef=coef, status=status)
    assert lt.lt_read_status(status) == lt.LT_STATUS_NONFINITE
    assert_state_equal(dev.to_host(), ref, "skipped step must not write")

    # max_norm = inf gives coef == 1, identical to passing no coefficient at all
    g[1][5] = 0
    gdev = [to_dev(x) for x in g]
    a, b = ref.to_dev(), ref.to_dev()
    _, _, status, _, coef = gpu_norm_and_coef(gdev, math.inf)
    assert to_host(coef)[0] == np.float32(1.0)
    gpu_step(a, gdev, 2048, 2, coef=coef, status=status)
    gpu_step(b, gdev, 2048, 2)
    ha, hb = a.to_host(), b.to_host()
    assert_state_equal(ha, hb, "coef 1 vs no coef")
    oracle_step(ref, g, 2048, 2)
    assert_state_equal(ha, ref, "no-clip step")


def test_step_grid_size_does_not_change_bits():
    rng = np.random.default_rng(9)
    sizes = [300000, 2049, 77777]
    base = _random_state(sizes, 2048, rng)
    g = [to_dev(f32_to_bf16_bits((rng.standard_t(3, size=n) * 1e-3).astype(np.float32)))
         for n in sizes]
    outs = []
    for cap in (0, 1, 3, 64):
        lt.lt_set_max_workgroups(cap)
        d = base.to_dev()
        gpu_step(d, g, 2048, 5)
        outs.append(d.to_host())
    for o in outs[1:]:
        assert_state_equal(o, outs[0], "grid cap")


def test_validation_errors_are_reported_before_launch():
    w = torch.zeros(4096 + 4, dtype=torch.float32, device=DEV)
    g = torch.zeros(4096, dtype=torch.bfloat16, device=DEV)
    mq = torch.zeros(4096, dtype=torch.int8, device=DEV)
    vq = torch.zeros(4096, dtype=torch.uint8, device=DEV)
    ma = torch.zeros(128, dtype=torch.float32, device=DEV)  # enough for any block size tried
    va = torch.zeros(128, dtype=torch.float32, device=DEV)
    args = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, step=1)
    with pytest.raises(lt.LazyTrainError) as e:
        lt.lt_hybrid8bit_adamw_step([w[1:4097]], [g], [mq], [ma], [vq], [va], 2048, **args)
    assert e.value.code == 2  # LT_ERR_ALIGNMENT: 4-byte offset view
    with pytest.raises(lt.LazyTrainError) as e:
        lt.lt_hybrid8bit_adamw_step([w[:4096]], [g], [mq], [ma], [vq], [va], 1000, **args)
    assert e.value.code == 1  # block size not a multiple of 64
    for bad_block in (0, 32, 96, 65536 + 64):
        with pytest.raises(lt.LazyTrainError) as e:
            lt.lt_hybrid8bit_adamw_step([w[:4096]], [g], [mq], [ma], [vq], [va], bad_block,
                                        **args)
        assert e.value.code == 1
    # eps must be positive, also once rounded to fp32 (eps = 0 divides 0 by 0 on a
    # zero gradient over a zero second moment)
    for bad_eps in (0.0, -1e-8, 1e-50, float("inf"), float("nan")):
        with pytest.raises(lt.LazyTrainError) as e:
            lt.lt_hybrid8bit_adamw_step([w[:4096]], [g], [mq], [ma], [vq], [va], 2048,
                                        **dict(args, eps=bad_eps))
        assert e.value.code == 1
        m32 = torch.zeros(4096, dtype=torch.float32, device=DEV)
        with pytest.raises(lt.LazyTrainError) as e:
            lt.lt_adamw_fp32_step([w[:4096]], [g], [m32], [m32.clone()],
                                  **dict(args, eps=bad_eps))
        assert e.value.code == 1
    with pytest.raises(lt.LazyTrainError) as e:
        lt.lt_hybrid8bit_adamw_step([w[:4096]], [g], [mq], [ma], [vq], [va], 2048,
                                    **dict(args, beta1=1.0))
    assert e.value.code == 1
    with pytest.raises(lt.LazyTrainError) as e:
        lt.lt_hybrid8bit_adamw_step([w[:4096]], [g], [mq], [ma], [vq], [va], 2048,
                                    **dict(args, step=0))
    assert e.value.code == 1
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    with pytest.raises(lt.LazyTrainError) as e:
        lt.lt_clip_coef(S, 0.0, torch.zeros(1, device=DEV))
    assert e.value.code == 1
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    small = torch.zeros(256, dtype=torch.uint8, device=DEV)
    with pytest.raises(ValueError):  # the binding checks the size first
        lt.lt_grad_sqnorm([g], S, st, workspace=small)
    # the C ABI checks it too
    ptrs = (ctypes.c_void_p * 1)(g.data_ptr())
    numels = (ctypes.c_int64 * 1)(g.numel())
    rc = lt.lib().lt_grad_sqnorm(ptrs, numels, 1, lt.LT_DTYPE_BF16, small.data_ptr(), 256, None,
                                 S.data_ptr(), st.data_ptr(), None)
    assert rc == 4  # LT_ERR_WORKSPACE
    assert b"workspace" in lt.lib().lt_last_error()
    rc = lt.lib().lt_grad_sqnorm(ptrs, numels, 1, 7, small.data_ptr(), 256, None, S.data_ptr(),
                                 st.data_ptr(), None)
    assert rc == 1  # unknown dtype


def test_optimizer_object_two_steps_against_oracle():
    """The optimizer object with its defaults (the decade-tree code map)."""
    rng = np.random.default_rng(12)
    sizes = [5000, 4096 * 3]
    w0 = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    params = [to_dev(x) for x in w0]
    opt = lt.Hybrid8bitAdamW(params, lr=1e-5, block_size=4096)
    assert opt.code_map == lt.LT_MAP_DYNAMIC
    ref = State.zero_host(w0, 4096)
    for t in (1, 2):
        g = [f32_to_bf16_bits((rng.standard_t(3, size=n) * 1e-2).astype(np.float32))
             for n in sizes]
        opt.step([to_dev(x) for x in g])
        assert opt.last_status() == lt.LT_STATUS_OK
        _, S, st = oracle.grad_sqnorm(g)
        _, c = oracle.clip_coef(S, 1.0)
        oracle_step(ref, g, 4096, t, coef=float(c), status=st, lr=1e-5,
                    code_map=oracle.MAP_DYNAMIC)
    got = State([to_host(p) for p in params], [to_host(x) for x in opt.m_codes],
                [to_host(x) for x in opt.m_absmax], [to_host(x) for x in opt.v_codes],
                [to_host(x) for x in opt.v_absmax])
    assert_state_equal(got, ref, "Hybrid8bitAdamW")
