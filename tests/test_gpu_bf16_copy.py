"""The optional bf16 weight copy written by the steps (8-bit, fp32-state and
layer-streamed): bitwise the oracle's round-to-nearest-even of the oracle's
updated weights; asking for the copy leaves weights, codes and scales bitwise
unchanged; after a skipped step the copy holds the unchanged weights; tensors
without a copy (None entries) are not touched."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, assert_state_equal, gpu_norm_and_coef, oracle_step, \
    to_dev, to_host

pytestmark = pytest.mark.gpu

SIZES = [1, 7, 8, 9, 1023, 2048, 2049, 4097, 65537, 300001]
SENTINEL = 0xBEEF


def _bf16_out(sizes, device=DEV):
    """bf16 outputs prefilled with a sentinel pattern."""
    return [torch.full((n,), SENTINEL - (1 << 16), dtype=torch.int16, device=device)
            .view(torch.bfloat16) for n in sizes]


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _is_nan(b):
    return ((b & 0x7F80) == 0x7F80) & ((b & 0x007F) != 0)


def _assert_bf16_equal(got, want, what):
    """Bitwise, except that a NaN only has to be a quiet NaN (fp32 NaN payloads are
    not fixed by IEEE arithmetic, so neither are the bits the copy keeps)."""
    nan_w, nan_g = _is_nan(want), _is_nan(got)
    assert np.array_equal(nan_g, nan_w), f"{what}: NaN positions differ"
    assert np.all((got[nan_g] & 0x0040) != 0), f"{what}: a NaN copy is not quiet"
    ok = ~nan_w
    if not np.array_equal(got[ok], want[ok]):
        i = np.flatnonzero(got[ok] != want[ok])[0]
        raise AssertionError(f"{what}: {np.count_nonzero(got[ok] != want[ok])} values differ, "
                             f"first {hex(got[ok][i])} vs {hex(want[ok][i])}")


def _random_state(rng, sizes, block):
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    st = State.zero_host(w, block)
    for k, n in enumerate(sizes):
        st.mq[k][:] = rng.integers(-127, 128, size=n)
        st.vq[k][:] = rng.integers(0, 256, size=n)
        st.ma[k][:] = rng.uniform(0.1, 5.0, size=st.ma[k].size) * 1e-3
        st.va[k][:] = rng.uniform(0.1, 5.0, size=st.va[k].size) * 1e-6
    return st


def _grads(rng, sizes, as_bf16):
    g = [(rng.standard_t(3, size=n) * 1e-3).astype(np.float32) for n in sizes]
    return [f32_to_bf16_bits(x) for x in g] if as_bf16 else g


@pytest.mark.parametrize("block", [64, 128, 256, 512, 1024, 2048, 4096, 8192])
@pytest.mark.parametrize("as_bf16", [False, True])
@pytest.mark.parametrize("code_map", [lt.LT_MAP_LINEAR, lt.LT_MAP_DYNAMIC])
def test_8bit_step_bf16_copy_matches_oracle(block, as_bf16, code_map):
    rng = np.random.default_rng(block + as_bf16 + 10 * code_map)
    base = _random_state(rng, SIZES, block)
    if code_map == lt.LT_MAP_DYNAMIC:  # every byte is a valid sign-magnitude code
        for k, n in enumerate(SIZES):
            base.mq[k][:] = rng.integers(-128, 128, size=n)
    g = _grads(rng, SIZES, as_bf16)
    gdev = [to_dev(x) for x in g]
    _, _, status, _, coef = gpu_norm_and_coef(gdev, 1.0)
    with_copy, without = base.to_dev(), base.to_dev()
    out = _bf16_out(SIZES)
    lt.lt_hybrid8bit_adamw_step(with_copy.w, gdev, with_copy.mq, with_copy.ma, with_copy.vq,
                                with_copy.va, block, step=3, coef=coef, status=status,
                                params_bf16=out, code_map=code_map, **HYPER)
    lt.lt_hybrid8bit_adamw_step(without.w, gdev, without.mq, without.ma, without.vq, without.va,
                                block, step=3, coef=coef, status=status, code_map=code_map,
                                **HYPER)
    torch.cuda.synchronize()
    assert_state_equal(with_copy.to_host(), without.to_host(), "state with vs without copy")
    ref = base.copy()
    _, S, st = oracle.grad_sqnorm(g, n_threads=8)
    _, c = oracle.clip_coef(S, 1.0)
    oracle_step(ref, g, block, 3, coef=float(c), status=st, code_map=code_map)
    assert_state_equal(with_copy.to_host(), ref, "state vs oracle")
    for k in range(len(SIZES)):
        _assert_bf16_equal(_bits(out[k]), oracle.round_bf16(ref.w[k]), f"copy of tensor {k}")


def _rounding_patterns():
    """Every upper half of the fp32 pattern with the lower halves that decide
    rounding: ties, near-ties, subnormals, infinities, NaN."""
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x1234, 0xC000], np.uint32)
    return (hi[:, None] | lows[None, :]).ravel().view(np.float32)


def test_bf16_copy_rounding_of_every_exponent():
    # lr = 0 and weight_decay = 0: w1 = fma(-0, m1/d, w * 1) = w, so the copy is the
    # rounding of the drawn patterns themselves
    w = _rounding_patterns()
    n = w.size
    block = 2048
    st = State.zero_host([w], block)
    g = [np.zeros(n, np.float32)]
    dev = st.to_dev()
    out = _bf16_out([n])
    hyper = dict(HYPER, lr=0.0, weight_decay=0.0)
    lt.lt_hybrid8bit_adamw_step(dev.w, [to_dev(g[0])], dev.mq, dev.ma, dev.vq, dev.va, block,
                                step=1, params_bf16=out, **hyper)
    ref = st.copy()
    oracle_step(ref, g, block, 1, **hyper)
    got_w = to_host(dev.w[0])
    finite = ~np.isnan(ref.w[0])
    assert np.array_equal(got_w[finite].view(np.uint32), ref.w[0][finite].view(np.uint32))
    assert np.array_equal(np.isnan(got_w), ~finite)
    _assert_bf16_equal(_bits(out[0]), oracle.round_bf16(ref.w[0]), "rounding patterns")


def test_bf16_copy_after_skipped_step_and_partial_lists():
    rng = np.random.default_rng(7)
    base = _random_state(rng, SIZES, 2048)
    g = _grads(rng, SIZES, True)
    g[3][0] = 0x7F80  # +inf in bf16: the step is skipped
    gdev = [to_dev(x) for x in g]
    _, _, status, _, coef = gpu_norm_and_coef(gdev, 1.0)
    dev = base.to_dev()
    out = _bf16_out(SIZES)
    partial = [o if k % 2 == 0 else None for k, o in enumerate(out)]
    lt.lt_hybrid8bit_adamw_step(dev.w, gdev, dev.mq, dev.ma, dev.vq, dev.va, 2048, step=2,
                                coef=coef, status=status, params_bf16=partial, **HYPER)
    torch.cuda.synchronize()
    assert lt.lt_read_status(status) == lt.LT_STATUS_NONFINITE
    assert_state_equal(dev.to_host(), base, "skipped step")
    for k in range(len(SIZES)):
        if k % 2 == 0:
            _assert_bf16_equal(_bits(out[k]), oracle.round_bf16(base.w[k]), f"skipped, {k}")
        else:
            assert np.all(_bits(out[k]) == SENTINEL), f"tensor {k} without a copy was written"


@pytest.mark.parametrize("as_bf16", [False, True])
def test_fp32_state_step_bf16_copy(as_bf16):
    rng = np.random.default_rng(50 + as_bf16)
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in SIZES]
    m = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in SIZES]
    v = [(rng.random(n) * 1e-6).astype(np.float32) for n in SIZES]
    g = _grads(rng, SIZES, as_bf16)
    gdev = [to_dev(x) for x in g]
    dw, dm, dv = [to_dev(x) for x in w], [to_dev(x) for x in m], [to_dev(x) for x in v]
    _, _, status, _, coef = gpu_norm_and_coef(gdev, 1.0)
    out = _bf16_out(SIZES)
    partial = [o if k != 2 else None for k, o in enumerate(out)]
    lt.lt_adamw_fp32_step(dw, gdev, dm, dv, step=4, coef=coef, status=status,
                          params_bf16=partial, **HYPER)
    torch.cuda.synchronize()
    _, S, _ = oracle.grad_sqnorm(g, n_threads=8)
    _, c = oracle.clip_coef(S, 1.0)
    for k in range(len(SIZES)):
        oracle.adamw_fp32_step(w[k], g[k], m[k], v[k], step=4, coef=float(c), **HYPER)
        assert to_host(dw[k]).tobytes() == w[k].tobytes()
        if k == 2:
            assert np.all(_bits(out[k]) == SENTINEL)
        else:
            _assert_bf16_equal(_bits(out[k]), oracle.round_bf16(w[k]), f"fp32-state copy {k}")


def test_streamed_bf16_copy_equals_resident():
    rng = np.random.default_rng(11)
    sizes = [4097, 65537, 9, 300001, 2048, 1]
    first = [0, 2, 4, 6]
    base = _random_state(rng, sizes, 2048)
    g = _grads(rng, sizes, True)
    pin = lambda a: torch.from_numpy(a).pin_memory()
    host = State(*[[pin(a.copy()) for a in lst] for lst in (base.w, base.mq, base.ma, base.vq,
                                                            base.va)])
    g_pin = [torch.from_numpy(x.view(np.int16)).pin_memory().view(torch.bfloat16) for x in g]
    host_out = [t.pin_memory() for t in _bf16_out(sizes, torch.device("cpu"))]
    host_out[4] = None
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    lt.lt_streamed_hybrid8bit_adamw_step(host.w, g_pin, host.mq, host.ma, host.vq, host.va,
                                         first, 2048, step=2, max_norm=1.0, ring_slots=2,
                                         sq_total=S, coef=coef, status=status,
                                         params_bf16=host_out, **HYPER)
    torch.cuda.synchronize()
    ref = base.copy()
    _, S_o, st_o = oracle.grad_sqnorm(g, n_threads=8)
    _, c_o = oracle.clip_coef(S_o, 1.0)
    oracle_step(ref, g, 2048, 2, coef=float(c_o), status=st_o)
    got = State(*[[t.numpy() for t in lst] for lst in (host.w, host.mq, host.ma, host.vq,
                                                        host.va)])
    assert_state_equal(got, ref, "streamed with copy vs oracle")
    for k in range(len(sizes)):
        if host_out[k] is None:
            continue
        _assert_bf16_equal(host_out[k].view(torch.int16).numpy().view(np.uint16),
                           oracle.round_bf16(ref.w[k]), f"streamed copy {k}")


def test_bf16_copy_rejects_bad_lists():
    w = [torch.zeros(16, device=DEV)]
    g = [torch.zeros(16, dtype=torch.bfloat16, device=DEV)]
    q = [torch.zeros(16, dtype=torch.int8, device=DEV)]
    u = [torch.zeros(16, dtype=torch.uint8, device=DEV)]
    a = [torch.zeros(1, device=DEV)]
    with pytest.raises(ValueError):
        lt.lt_hybrid8bit_adamw_step(w, g, q, a, u, a, 2048, step=1,
                                    params_bf16=[torch.zeros(15, dtype=torch.bfloat16,
                                                             device=DEV)], **HYPER)
    with pytest.raises(TypeError):
        lt.lt_hybrid8bit_adamw_step(w, g, q, a, u, a, 2048, step=1,
                                    params_bf16=[torch.zeros(16, device=DEV)], **HYPER)
    with pytest.raises(ValueError):
        lt.lt_hybrid8bit_adamw_step(w, g, q, a, u, a, 2048, step=1, params_bf16=[], **HYPER)
