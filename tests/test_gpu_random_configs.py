"""Seeded sweep of random configurations against the oracle: tensor counts and
ragged sizes, block size, gradient dtype, code map, every hyperparameter (beta1
down to 0, beta2 from 0.5 to 0.9999, eps, lr including 0, weight decay, the step
index), max_norm (clipping on and off), random 8-bit states with zero blocks, and
the bf16 weight copy.  S, the clip coefficient, weights, codes, scales and the
copy must be bitwise the oracle's in every case."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, State, assert_state_equal, to_dev, to_host

pytestmark = pytest.mark.gpu

BLOCKS = [64, 128, 256, 512, 1024, 2048, 4096, 8192]


def _config(seed):
    rng = np.random.default_rng(seed)
    K = int(rng.integers(1, 7))
    sizes = []
    for _ in range(K):
        kind = rng.integers(0, 4)
        sizes.append(int(rng.integers(1, 64)) if kind == 0 else
                     int(rng.integers(64, 9000)) if kind == 1 else
                     int(rng.integers(9000, 300000)) if kind == 2 else
                     int(rng.choice([2048, 4096, 8192, 65536])) + int(rng.integers(-1, 2)))
    return dict(
        rng=rng, sizes=sizes, block=int(rng.choice(BLOCKS)), bf16=bool(rng.integers(0, 2)),
        code_map=int(rng.integers(0, 2)), copy=bool(rng.integers(0, 2)),
        hyper=dict(lr=float(rng.choice([0.0, 1e-5, 1e-3, 0.1])),
                   beta1=float(rng.choice([0.0, 0.5, 0.9, 0.99])),
                   beta2=float(rng.choice([0.5, 0.9, 0.999, 0.9999])),
                   eps=float(rng.choice([1e-8, 1e-6, 1e-3])),
                   weight_decay=float(rng.choice([0.0, 0.01, 0.1]))),
        step=int(rng.choice([1, 2, 10, 1000])),
        max_norm=float(rng.choice([0.1, 1.0, math.inf])),
        grad_scale=float(rng.choice([1e-6, 1e-3, 1.0])))


@pytest.mark.parametrize("seed", range(80))
def test_random_configuration_matches_oracle(seed):
    c = _config(seed)
    rng, sizes, B = c["rng"], c["sizes"], c["block"]
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    g32 = [(rng.standard_t(3, size=n) * c["grad_scale"]).astype(np.float32) for n in sizes]
    g = [f32_to_bf16_bits(x) for x in g32] if c["bf16"] else g32
    base = State.zero_host(w, B)
    for k, n in enumerate(sizes):
        lo = -128 if c["code_map"] == lt.LT_MAP_DYNAMIC else -127
        base.mq[k][:] = rng.integers(lo, 128, size=n)
        base.vq[k][:] = rng.integers(0, 256, size=n)
        nb = base.ma[k].size
        base.ma[k][:] = rng.uniform(0.1, 5.0, size=nb) * c["grad_scale"]
        base.va[k][:] = rng.uniform(0.1, 5.0, size=nb) * c["grad_scale"] ** 2
        zero = rng.random(nb) < 0.1
        base.ma[k][zero] = 0.0
        base.va[k][zero] = 0.0

    # oracle
    ref = base.copy()
    _, S_o, st_o = oracle.grad_sqnorm(g, n_threads=8)
    _, c_o = oracle.clip_coef(S_o, c["max_norm"])
    oracle.hybrid8bit_adamw_step(ref.w, g, ref.mq, ref.ma, ref.vq, ref.va, B, step=c["step"],
                                 coef=float(c_o), status=st_o, code_map=c["code_map"],
                                 n_threads=8, **c["hyper"])
    # HIP path
    dev = base.to_dev()
    gd = [to_dev(x) for x in g]
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    wb = [torch.zeros(n, dtype=torch.bfloat16, device=DEV) for n in sizes] if c["copy"] else None
    lt.lt_grad_sqnorm(gd, S, status)
    lt.lt_clip_coef(S, c["max_norm"], coef)
    lt.lt_hybrid8bit_adamw_step(dev.w, gd, dev.mq, dev.ma, dev.vq, dev.va, B, step=c["step"],
                                coef=coef, status=status, code_map=c["code_map"],
                                params_bf16=wb, **c["hyper"])
    torch.cuda.synchronize()
    what = (f"seed {seed}: sizes {sizes}, block {B}, bf16 {c['bf16']}, map {c['code_map']}, "
            f"{c['hyper']}, step {c['step']}, max_norm {c['max_norm']}")
    assert to_host(S)[0].hex() == S_o.hex(), what
    assert int(to_host(status)[0]) == st_o, what
    assert to_host(coef)[0] == c_o, what
    got = dev.to_host()
    if wb is not None:
        for k in range(len(sizes)):
            want = oracle.round_bf16(ref.w[k])
            have = to_host(wb[k])
            nan = ((want & 0x7F80) == 0x7F80) & ((want & 0x7F) != 0)
            assert np.array_equal(have[~nan], want[~nan]), what
    # no NaN is expected (finite inputs, eps > 0); one would only have to be NaN on
    # both sides, as NaN payloads are not fixed
    for k in range(len(sizes)):
        a, b = got.w[k], ref.w[k]
        both = np.isnan(a) & np.isnan(b)
        a[both] = b[both] = 0.0
    assert_state_equal(got, ref, what)


@pytest.mark.parametrize("seed", range(100, 115))
def test_random_configuration_fp32_state_step(seed):
    c = _config(seed)
    rng, sizes = c["rng"], c["sizes"]
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    g32 = [(rng.standard_t(3, size=n) * c["grad_scale"]).astype(np.float32) for n in sizes]
    g = [f32_to_bf16_bits(x) for x in g32] if c["bf16"] else g32
    m = [(rng.standard_normal(n) * c["grad_scale"]).astype(np.float32) for n in sizes]
    v = [(rng.uniform(0, 1, n) * c["grad_scale"] ** 2).astype(np.float32) for n in sizes]
    dw, dm, dv = [to_dev(x) for x in w], [to_dev(x) for x in m], [to_dev(x) for x in v]
    coef = torch.tensor([0.37], dtype=torch.float32, device=DEV)
    lt.lt_adamw_fp32_step(dw, [to_dev(x) for x in g], dm, dv, step=c["step"], coef=coef,
                          **c["hyper"])
    torch.cuda.synchronize()
    for k in range(len(sizes)):
        oracle.adamw_fp32_step(w[k], g[k], m[k], v[k], step=c["step"], coef=0.37, **c["hyper"])
        for a, b, name in ((dw[k], w[k], "w"), (dm[k], m[k], "m"), (dv[k], v[k], "v")):
            assert to_host(a).tobytes() == b.tobytes(), f"seed {seed}: {name}[{k}]"


@pytest.mark.parametrize("seed", range(200, 212))
def test_random_configuration_streamed_step(seed):
    c = _config(seed)
    rng, sizes, B = c["rng"], c["sizes"], c["block"]
    # random layer split of the list, ring of 2..4 slots, separate or shared streams
    cuts = sorted(set(rng.choice(np.arange(1, len(sizes)), size=min(len(sizes) - 1, 2),
                                 replace=False).tolist())) if len(sizes) > 1 else []
    first = [0] + cuts + [len(sizes)]
    slots = int(rng.integers(2, 5))
    separate = bool(rng.integers(0, 2))
    keep = bool(rng.integers(0, 2))
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    g32 = [(rng.standard_t(3, size=n) * c["grad_scale"]).astype(np.float32) for n in sizes]
    g = [f32_to_bf16_bits(x) for x in g32] if c["bf16"] else g32
    base = State.zero_host(w, B)
    for k, n in enumerate(sizes):
        lo = -128 if c["code_map"] == lt.LT_MAP_DYNAMIC else -127
        base.mq[k][:] = rng.integers(lo, 128, size=n)
        base.vq[k][:] = rng.integers(0, 256, size=n)
        base.ma[k][:] = rng.uniform(0.1, 5.0, size=base.ma[k].size) * c["grad_scale"]
        base.va[k][:] = rng.uniform(0.1, 5.0, size=base.va[k].size) * c["grad_scale"] ** 2
    ref = base.copy()
    _, S_o, st_o = oracle.grad_sqnorm(g, n_threads=8)
    _, c_o = oracle.clip_coef(S_o, c["max_norm"])
    oracle.hybrid8bit_adamw_step(ref.w, g, ref.mq, ref.ma, ref.vq, ref.va, B, step=c["step"],
                                 coef=float(c_o), status=st_o, code_map=c["code_map"],
                                 n_threads=8, **c["hyper"])
    pin = lambda a: torch.from_numpy(a).pin_memory()
    host = State(*[[pin(a.copy()) for a in lst] for lst in
                   (base.w, base.mq, base.ma, base.vq, base.va)])
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    streams = [torch.cuda.Stream(DEV) for _ in range(3)] if separate else [None] * 3
    if separate:
        streams[0].wait_stream(torch.cuda.current_stream())
    g_host = [pin(x.view(np.int16)).view(torch.bfloat16) if c["bf16"] else pin(x) for x in g]
    lt.lt_streamed_hybrid8bit_adamw_step(host.w, g_host, host.mq,
                                         host.ma, host.vq, host.va, first, B, step=c["step"],
                                         max_norm=c["max_norm"], ring_slots=slots, sq_total=S,
                                         coef=coef, status=status, compute_stream=streams[0],
                                         h2d_stream=streams[1], d2h_stream=streams[2],
                                         code_map=c["code_map"], keep_grads=keep, **c["hyper"])
    (streams[0] or torch.cuda.current_stream()).synchronize()
    what = (f"seed {seed}: sizes {sizes}, layers {first}, block {B}, slots {slots}, "
            f"keep {keep}, bf16 {c['bf16']}")
    assert to_host(S)[0].hex() == S_o.hex() and to_host(coef)[0] == c_o, what
    got = State(*[[t.numpy() for t in lst] for lst in (host.w, host.mq, host.ma, host.vq, host.va)])
    assert_state_equal(got, ref, what)
