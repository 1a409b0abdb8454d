"""Pins of the oracle's Hybrid 8-bit AdamW step (paper Sec. 3.5: block-wise 8-bit
AdamW states on fp32 master weights, clipped gradients; App. C training-config
table: beta1 0.9, beta2 0.999, eps 1e-8, lr 1e-5, weight decay 0.01, max grad norm
1.0, non-finite gradients skip the step).

Pins that do not reuse the oracle's code:
* hand-worked blocks with exact dyadic values (tests/golden/adamw8_worked_examples.txt);
* torch.optim.AdamW (fp32, single-tensor path) with the 8-bit states decoded onto
  its fp32 state: the weight update, the decoupled decay and the new moments;
* closed forms: the first step from zero state is -lr*g/(|g|+eps) plus decay;
  lr = 0 leaves the weights unchanged; beta1 = 0 makes the new first-moment absmax
  max|g|; an all-zero block on zero state stays a zero block;
* the skip rule for non-finite gradients.
"""
import numpy as np
import pytest
import torch

import oracle
from golden_io import adamw_examples, bf16_bits_to_f32, f32_to_bf16_bits


def _state(n, block, rng, scale_m=1e-3, scale_v=1e-6, zero_frac=0.0):
    nb = -(-n // block)
    qm = rng.integers(-127, 128, size=n).astype(np.int8)
    qv = rng.integers(0, 256, size=n).astype(np.uint8)
    am = (rng.uniform(0.2, 5.0, size=nb) * scale_m).astype(np.float32)
    av = (rng.uniform(0.2, 5.0, size=nb) * scale_v).astype(np.float32)
    if zero_frac:
        z = rng.random(nb) < zero_frac
        am[z] = 0
        av[z] = 0
    return qm, am, qv, av


def _decode(qm, am, qv, av, block):
    """The 8-bit states as fp32 tensors: q * (A / 127) and q * (A / 255)."""
    n = qm.size
    bi = np.arange(n) // block
    sm = (am / np.float32(127.0)).astype(np.float32)
    sv = (av / np.float32(255.0)).astype(np.float32)
    return (qm.astype(np.float32) * sm[bi]).astype(np.float32), \
        (qv.astype(np.float32) * sv[bi]).astype(np.float32)


def _torch_adamw(w, g32, m0, v0, t, lr, b1, b2, eps, wd):
    p = torch.nn.Parameter(torch.from_numpy(w.copy()))
    opt = torch.optim.AdamW([p], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd,
                            foreach=False, fused=False)
    opt.state[p] = {"step": torch.tensor(float(t - 1)),
                    "exp_avg": torch.from_numpy(m0.copy()),
                    "exp_avg_sq": torch.from_numpy(v0.copy())}
    p.grad = torch.from_numpy(g32.copy())
    opt.step()
    st = opt.state[p]
    return p.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()


def _run(w, g, qm, am, qv, av, block, **kw):
    w, qm, am, qv, av = (a.copy() for a in (w, qm, am, qv, av))
    oracle.hybrid8bit_adamw_step([w], [g], [qm], [am], [qv], [av], block, **kw)
    return w, qm, am, qv, av


# ------------------------------------------------------------ hand-worked blocks

@pytest.mark.parametrize("as_bf16", [False, True])
def test_hand_worked_examples(as_bf16):
    n = 0
    for ex in adamw_examples():
        g = ex["grad"]
        if as_bf16:
            g = f32_to_bf16_bits(g)
            assert np.array_equal(bf16_bits_to_f32(g), ex["grad"])  # exact in bf16
        w, qm, am, qv, av = _run(ex["w"], g, ex["m_codes"], ex["m_absmax"], ex["v_codes"],
                                 ex["v_absmax"], ex["block_size"], lr=ex["lr"],
                                 beta1=ex["beta1"], beta2=ex["beta2"], eps=ex["eps"],
                                 weight_decay=ex["weight_decay"], step=ex["t"], coef=ex["coef"])
        name = ex["name"]
        assert np.array_equal(w, ex["expect_w"]), (name, w)
        assert np.array_equal(qm, ex["expect_m_codes"]), (name, qm)
        assert np.array_equal(am, ex["expect_m_absmax"]), (name, am)
        assert np.array_equal(qv, ex["expect_v_codes"]), (name, qv)
        assert np.array_equal(av, ex["expect_v_absmax"]), (name, av)
        n += 1
    assert n >= 5


# ------------------------------------------------------------------ torch AdamW

CASES = [
    # t, lr, beta1, beta2, eps, wd, coef, grad scale
    (2, 1e-4, 0.9, 0.999, 1e-8, 0.01, 1.0, 1e-3),
    (2, 1e-5, 0.9, 0.999, 1e-8, 0.01, 0.06, 1e-3),
    (1, 1e-4, 0.9, 0.999, 1e-8, 0.01, 1.0, 1e-3),
    (10, 3e-4, 0.8, 0.99, 1e-8, 0.1, 0.5, 1e-2),
    (3, 1e-4, 0.9, 0.999, 1e-8, 0.0, 1.0, 1e-8),   # |g| ~ eps: eps placement matters
    (5, 1e-3, 0.5, 0.6, 1e-6, 0.05, 1.0, 1.0),
]


@pytest.mark.parametrize("case", CASES)
def test_update_matches_torch_adamw(case):
    t, lr, b1, b2, eps, wd, coef, gs = case
    rng = np.random.default_rng(hash(case) % (2 ** 32))
    n, block = 3000, 256
    g = (rng.standard_t(3, size=n) * gs).astype(np.float32)
    qm, am, qv, av = _state(n, block, rng, scale_m=gs, scale_v=gs * gs)
    if t == 1:
        qm[:] = 0
        qv[:] = 0
    m0, v0 = _decode(qm, am, qv, av, block)
    gc = (g * np.float32(coef)).astype(np.float32)  # the clipped gradient, one rounding

    # w = 0 isolates the Adam update itself (no decay, no rounding against a large w).
    # Both sides round each operation once but in different orders (torch's lerp for m1),
    # so the bound is a few ulps of the *terms* of m1 and of the result, not of m1 alone
    # (m1 = b1*m0 + (1-b1)*g can cancel).
    w = np.zeros(n, np.float32)
    w1, _, _, _, _ = _run(w, g, qm, am, qv, av, block, lr=lr, beta1=b1, beta2=b2, eps=eps,
                          weight_decay=wd, step=t, coef=coef)
    wt, _, vt = _torch_adamw(w, gc, m0, v0, t, lr, b1, b2, eps, wd)
    step_size = lr / (1 - b1 ** t)
    denom = np.sqrt(vt.astype(np.float64)) / np.sqrt(1 - b2 ** t) + eps
    terms = step_size * (b1 * np.abs(m0.astype(np.float64)) + (1 - b1) * np.abs(gc)) / denom
    d = np.abs(w1.astype(np.float64) - wt)
    assert np.all(d <= 5e-7 * (terms + np.abs(wt)) + 1e-37), (d / (terms + np.abs(wt))).max()

    # decoupled decay on realistic weights: the same bound plus an ulp of w*decay
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    w1, qm1, am1, qv1, av1 = _run(w, g, qm, am, qv, av, block, lr=lr, beta1=b1, beta2=b2,
                                  eps=eps, weight_decay=wd, step=t, coef=coef)
    wt, mt, vt = _torch_adamw(w, gc, m0, v0, t, lr, b1, b2, eps, wd)
    d = np.abs(w1.astype(np.float64) - wt)
    wd_term = np.abs(w.astype(np.float64)) * (1 - lr * wd)
    assert np.all(d <= 5e-7 * (terms + wd_term + np.abs(wt)) + 1e-37), d.max()
    # a missing decay would be off by lr*wd*|w|, far outside that bound when wd > 0

    # the stored codes decode to torch's new moments within half a code step
    m1, v1 = _decode(qm1, am1, qv1, av1, block)
    bi = np.arange(n) // block
    assert np.all(np.abs(m1 - mt) <= 0.5 * am1[bi] / 127 * (1 + 1e-5) + 1e-6 * np.abs(mt) + 1e-38)
    assert np.all(np.abs(v1 - vt) <= 0.5 * av1[bi] / 255 * (1 + 1e-5) + 1e-6 * np.abs(vt) + 1e-38)
    # and the new scales are the block maxima of torch's moments (to rounding)
    for b in range(len(am1)):
        sl = slice(b * block, (b + 1) * block)
        assert abs(am1[b] - np.abs(mt[sl]).max()) <= 2e-7 * am1[b] + 1e-38
        assert abs(av1[b] - vt[sl].max()) <= 2e-7 * av1[b] + 1e-38


def test_eight_bit_step_is_fp32_adamw_when_states_are_on_the_grid():
    rng = np.random.default_rng(3)
    n, block = 4096 + 100, 512
    g = (rng.standard_t(3, size=n) * 1e-3).astype(np.float32)
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    qm, am, qv, av = _state(n, block, rng)
    m0, v0 = _decode(qm, am, qv, av, block)
    kw = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, step=4)
    w8, qm1, am1, qv1, av1 = _run(w, g, qm, am, qv, av, block, coef=0.7, **kw)
    wf, mf, vf = w.copy(), m0.copy(), v0.copy()
    oracle.adamw_fp32_step(wf, g, mf, vf, coef=0.7, **kw)
    assert w8.tobytes() == wf.tobytes()
    for b in range(-(-n // block)):
        sl = slice(b * block, min(n, (b + 1) * block))
        q, a = oracle.quantize_signed(mf[sl])
        assert np.array_equal(q, qm1[sl]) and a == am1[b]
        q, a = oracle.quantize_unsigned(vf[sl])
        assert np.array_equal(q, qv1[sl]) and a == av1[b]


# ----------------------------------------------------------------- closed forms

def test_first_step_from_zero_state_closed_form():
    rng = np.random.default_rng(4)
    n, block = 5000, 2048
    g = (rng.standard_t(3, size=n) * 1e-3).astype(np.float32)
    g[::97] = np.float32(3e-9)  # comparable to eps
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    z8 = np.zeros(n, np.int8)
    zu = np.zeros(n, np.uint8)
    za = np.zeros(-(-n // block), np.float32)
    lr, wd, eps = 1e-4, 0.01, 1e-8
    w1, *_ = _run(w, g, z8, za, zu, za, block, lr=lr, beta1=0.9, beta2=0.999, eps=eps,
                  weight_decay=wd, step=1)
    g64 = g.astype(np.float64)
    expect = w.astype(np.float64) * (1 - lr * wd) - lr * g64 / (np.abs(g64) + eps)
    assert np.all(np.abs(w1 - expect) <= 1e-5 * lr + 2 * np.spacing(np.abs(w)))


def test_zero_learning_rate_leaves_weights_unchanged():
    rng = np.random.default_rng(5)
    n, block = 3333, 256
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    w[w == 0] = 1.0
    qm, am, qv, av = _state(n, block, rng)
    w1, *_ = _run(w, g, qm, am, qv, av, block, lr=0.0, beta1=0.9, beta2=0.999, eps=1e-8,
                  weight_decay=0.5, step=3)
    assert w1.tobytes() == w.tobytes()


def test_host_scalars():
    s = oracle.step_scalars(1e-5, 0.9, 0.999, 1e-8, 0.0, 1)
    assert s["decay"] == np.float32(1.0)
    assert s["step_size"] == np.float32(1e-5 / (1 - 0.9))
    assert s["rbc2"] == np.float32(1 / np.sqrt(1 - 0.999))
    assert s["c1"] == np.float32(1 - 0.9) and s["c2"] == np.float32(1 - 0.999)
    assert s["beta2"] == np.float32(0.999) and s["eps"] == np.float32(1e-8)
    s = oracle.step_scalars(1e-4, 0.9, 0.999, 1e-8, 0.01, 2)
    assert s["decay"] == np.float32(1 - 1e-6)
    assert s["step_size"] == np.float32(1e-4 / (1 - 0.9 ** 2))
    assert s["rbc2"] == np.float32(1 / np.sqrt(1 - 0.999 ** 2))


def test_beta1_zero_first_moment_is_the_gradient():
    rng = np.random.default_rng(6)
    n, block = 2048 * 3, 2048
    g = (rng.standard_t(3, size=n) * 1e-3).astype(np.float32)
    qm, am, qv, av = _state(n, block, rng)
    _, qm1, am1, _, _ = _run(np.zeros(n, np.float32), g, qm, am, qv, av, block, lr=1e-4,
                             beta1=0.0, beta2=0.999, eps=1e-8, weight_decay=0.0, step=2,
                             coef=0.25)
    gc = (g * np.float32(0.25)).astype(np.float32)
    for b in range(3):
        assert am1[b] == np.abs(gc[b * block:(b + 1) * block]).max()


def test_zero_gradient_block_on_zero_state_stays_zero():
    n, block = 4096 + 17, 2048
    w = np.linspace(-1, 1, n).astype(np.float32)
    w1, qm1, am1, qv1, av1 = _run(w, np.zeros(n, np.float32), np.zeros(n, np.int8),
                                  np.zeros(3, np.float32), np.zeros(n, np.uint8),
                                  np.zeros(3, np.float32), block, lr=1e-4, beta1=0.9,
                                  beta2=0.999, eps=1e-8, weight_decay=0.01, step=1)
    decay = oracle.step_scalars(1e-4, 0.9, 0.999, 1e-8, 0.01, 1)["decay"]
    assert w1.tobytes() == (w * decay).astype(np.float32).tobytes()
    assert not qm1.any() and not qv1.any() and not am1.any() and not av1.any()


# ------------------------------------------------------------- skip and wiring

def _random_problem(seed, n=5000, block=256, bf16=True):
    rng = np.random.default_rng(seed)
    g32 = (rng.standard_t(3, size=n) * 1e-3).astype(np.float32)
    g = f32_to_bf16_bits(g32) if bf16 else g32
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    return w, g, _state(n, block, rng, zero_frac=0.05)


KW = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, step=2)


def test_nonfinite_status_skips_the_step():
    w, g, (qm, am, qv, av) = _random_problem(7)
    out = _run(w, g, qm, am, qv, av, 256, coef=0.5, status=oracle.STATUS_NONFINITE, **KW)
    for a, b in zip(out, (w, qm, am, qv, av)):
        assert a.tobytes() == b.tobytes()
    out_ok = _run(w, g, qm, am, qv, av, 256, coef=0.5, status=oracle.STATUS_OK, **KW)
    out_none = _run(w, g, qm, am, qv, av, 256, coef=0.5, **KW)
    assert out_ok[0].tobytes() != w.tobytes()
    for a, b in zip(out_ok, out_none):
        assert a.tobytes() == b.tobytes()


def test_no_coef_is_coef_one_and_coef_scales_the_gradient():
    w, g, (qm, am, qv, av) = _random_problem(8, bf16=False)
    a = _run(w, g, qm, am, qv, av, 256, **KW)
    b = _run(w, g, qm, am, qv, av, 256, coef=1.0, **KW)
    for x, y in zip(a, b):
        assert x.tobytes() == y.tobytes()
    c = _run(w, g, qm, am, qv, av, 256, coef=0.37, **KW)
    d = _run(w, (g * np.float32(0.37)).astype(np.float32), qm, am, qv, av, 256, **KW)
    for x, y in zip(c, d):
        assert x.tobytes() == y.tobytes()


def test_list_call_equals_per_tensor_and_per_block_calls():
    block = 256
    probs = [_random_problem(20 + i, n) for i, n in enumerate((1, 255, 256, 2049, 4096))]
    lists = [[p[0].copy() for p in probs], [p[1] for p in probs]] + \
        [[p[2][j].copy() for p in probs] for j in range(4)]
    w, g, qm, am, qv, av = lists
    oracle.hybrid8bit_adamw_step(w, g, qm, am, qv, av, block, coef=0.8, **KW)
    for i, (w0, g0, (qm0, am0, qv0, av0)) in enumerate(probs):
        n = w0.size
        for b in range(-(-n // block)):
            sl = slice(b * block, min(n, (b + 1) * block))
            r = _run(w0[sl], g0[sl], qm0[sl], am0[b:b + 1], qv0[sl], av0[b:b + 1], block,
                     coef=0.8, **KW)
            assert r[0].tobytes() == w[i][sl].tobytes()
            assert r[1].tobytes() == qm[i][sl].tobytes() and r[2][0] == am[i][b]
            assert r[3].tobytes() == qv[i][sl].tobytes() and r[4][0] == av[i][b]


def test_thread_count_does_not_change_bits():
    w, g, (qm, am, qv, av) = _random_problem(9, n=300000, block=2048)
    a = _run(w, g, qm, am, qv, av, 2048, coef=0.3, n_threads=1, **KW)
    b = _run(w, g, qm, am, qv, av, 2048, coef=0.3, n_threads=8, **KW)
    for x, y in zip(a, b):
        assert x.tobytes() == y.tobytes()


def test_three_step_drift_against_unquantized_fp64_adamw():
    """Informative (not a parity pin): three 8-bit steps against fp64 AdamW with fp64
    states.  With the linear absmax code map, a second moment far below its block's
    absmax rounds to code 0 while the first moment may not; the next step then
    divides m1 by a tiny denominator.  The test measures that hazard separately:
    elements that never met it stay within about one lr of fp64 AdamW, the others
    are reported."""
    rng = np.random.default_rng(10)
    n, block = 2048 * 8, 2048
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    w8, qm, qv = w.copy(), np.zeros(n, np.int8), np.zeros(n, np.uint8)
    am, av = np.zeros(8, np.float32), np.zeros(8, np.float32)
    w64, m64, v64 = w.astype(np.float64), np.zeros(n), np.zeros(n)
    lr, b1, b2, eps, wd = 1e-4, 0.9, 0.999, 1e-8, 0.01
    hazard = np.zeros(n, bool)
    for t in (1, 2, 3):
        g = (rng.standard_t(3, size=n) * 1e-3).astype(np.float32)
        hazard |= (qv == 0) & (qm != 0)
        oracle.hybrid8bit_adamw_step([w8], [g], [qm], [am], [qv], [av], block, lr=lr, beta1=b1,
                                     beta2=b2, eps=eps, weight_decay=wd, step=t)
        g64 = g.astype(np.float64)
        m64 = b1 * m64 + (1 - b1) * g64
        v64 = b2 * v64 + (1 - b2) * g64 ** 2
        w64 = w64 * (1 - lr * wd) - lr / (1 - b1 ** t) * m64 / (
            np.sqrt(v64) / np.sqrt(1 - b2 ** t) + eps)
        drift = np.abs(w8 - w64) / lr
        print(f"step {t}: drift/lr max {drift.max():.3g}, outside hazard max "
              f"{drift[~hazard].max():.3g}, hazard fraction {hazard.mean():.3f}")
        assert drift[~hazard].max() < 2.0


@pytest.mark.parametrize("case", CASES[:4])
def test_fp32_state_adamw_matches_torch(case):
    """The fp32-state step (the non-8-bit part of the hybrid operator) against
    torch.optim.AdamW with the same fp32 states, to the rounding-error bound."""
    t, lr, b1, b2, eps, wd, coef, gs = case
    rng = np.random.default_rng(abs(hash(case)) % (2 ** 32) + 1)
    n = 5000
    g = (rng.standard_t(3, size=n) * gs).astype(np.float32)
    m0 = (rng.standard_normal(n) * gs).astype(np.float32)
    v0 = (rng.random(n) * gs * gs).astype(np.float32)
    if t == 1:
        m0[:] = 0
        v0[:] = 0
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    wo, mo, vo = w.copy(), m0.copy(), v0.copy()
    oracle.adamw_fp32_step(wo, g, mo, vo, lr=lr, beta1=b1, beta2=b2, eps=eps, weight_decay=wd,
                           step=t, coef=coef)
    gc = (g * np.float32(coef)).astype(np.float32)
    wt, mt, vt = _torch_adamw(w, gc, m0, v0, t, lr, b1, b2, eps, wd)
    assert np.all(np.abs(mo - mt) <= 4e-7 * (b1 * np.abs(m0) + (1 - b1) * np.abs(gc)) + 1e-38)
    assert np.all(np.abs(vo - vt) <= 4e-7 * np.abs(vt) + 1e-38)
    step_size = lr / (1 - b1 ** t)
    denom = np.sqrt(vt.astype(np.float64)) / np.sqrt(1 - b2 ** t) + eps
    terms = step_size * (b1 * np.abs(m0.astype(np.float64)) + (1 - b1) * np.abs(gc)) / denom
    d = np.abs(wo.astype(np.float64) - wt)
    assert np.all(d <= 5e-7 * (terms + np.abs(w) + np.abs(wt)) + 1e-37)


def test_empty_tensors_are_not_stepped():
    # a zero-element tensor has no blocks: the others step exactly as without it
    block = 256
    probs = [_random_problem(40 + i, n) for i, n in enumerate((300, 4096))]
    full = [[p[0].copy() for p in probs], [p[1] for p in probs]] + \
        [[p[2][j].copy() for p in probs] for j in range(4)]
    oracle.hybrid8bit_adamw_step(*full, block, coef=0.7, **KW)
    e32, e8, eu8 = np.zeros(0, np.float32), np.zeros(0, np.int8), np.zeros(0, np.uint8)
    eg = np.zeros(0, probs[0][1].dtype)
    mixed = [[e32, probs[0][0].copy(), e32, probs[1][0].copy()],
             [eg, probs[0][1], eg, probs[1][1]]] + \
        [[{0: e8, 1: e32, 2: eu8, 3: e32}[j], probs[0][2][j].copy(),
          {0: e8, 1: e32, 2: eu8, 3: e32}[j], probs[1][2][j].copy()] for j in range(4)]
    oracle.hybrid8bit_adamw_step(*mixed, block, coef=0.7, **KW)
    for got, want in zip(mixed, full):
        assert got[0].size == 0 and got[2].size == 0
        assert got[1].tobytes() == want[0].tobytes() and got[3].tobytes() == want[1].tobytes()
    oracle.hybrid8bit_adamw_step([], [], [], [], [], [], block, coef=0.7, **KW)
