"""Parity on extreme and corrupted optimizer states: stored scales that are +-inf,
NaN, negative, zero (with nonzero codes), subnormal or the largest fp32; the
linear map's unused code -128; weights that are NaN, +-inf, -0 or subnormal;
subnormal, -0 and extreme gradients.  The readings define every case (decode
q * (A / 127) for any code and scale, block maxima that skip NaN elements, the
clamp, the zero-block rule), so the GPU must match the oracle bitwise, except
that a NaN weight only has to be NaN on both sides (NaN payloads are not fixed)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, to_dev

pytestmark = pytest.mark.gpu

F32_MAX = np.float32(np.finfo(np.float32).max)
SUB = np.float32(1e-40)  # fp32 subnormal


def _edge_problem(block, code_map, seed):
    rng = np.random.default_rng(seed)
    # at least 10 blocks, and two whole wave spans plus a ragged one at small blocks
    nb = max(10, 2 * 2048 // block + 3)
    n = nb * block - 37  # ragged last block
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g32 = (rng.standard_t(3, size=n) * 1e-3).astype(np.float32)
    mq = rng.integers(-127, 128, size=n).astype(np.int8)
    vq = rng.integers(0, 256, size=n).astype(np.uint8)
    if code_map == lt.LT_MAP_DYNAMIC:
        mq = rng.integers(-128, 128, size=n).astype(np.int8)
    ma = (rng.uniform(0.2, 5.0, size=nb) * 1e-3).astype(np.float32)
    va = (rng.uniform(0.2, 5.0, size=nb) * 1e-6).astype(np.float32)
    blk = lambda b: slice(b * block, min(n, (b + 1) * block))
    ma[0], va[0] = np.inf, np.float32(3e-6)          # infinite first-moment scale
    ma[1], va[1] = np.nan, np.nan                    # NaN scales
    ma[2], va[2] = -np.float32(2e-3), -np.float32(1e-6)  # negative scales
    ma[3], va[3] = 0.0, 0.0                          # zero scales under nonzero codes
    ma[4], va[4] = SUB, SUB                          # subnormal scales
    ma[5], va[5] = F32_MAX, F32_MAX                  # largest finite scales
    mq[blk(6)] = -128                                # the code the linear map never writes
    va[7] = -np.inf
    ma[nb - 1], va[nb - 2] = np.nan, np.inf          # in the last, ragged wave span
    # weights and gradients with special values, spread over the blocks
    idx = rng.choice(n, size=64, replace=False)
    w[idx[:8]] = np.nan
    w[idx[8:16]] = np.inf
    w[idx[16:24]] = -np.inf
    w[idx[24:32]] = -0.0
    w[idx[32:40]] = SUB
    g32[idx[40:48]] = -0.0
    g32[idx[48:56]] = SUB
    g32[idx[56:60]] = np.float32(3e38)
    g32[idx[60:64]] = -np.float32(3e38)
    g = f32_to_bf16_bits(g32)
    return w, g, mq, ma, vq, va


def _assert_equal_nan_aware(got: State, ref: State, what):
    for k, (a, b) in enumerate(zip(got.w, ref.w)):
        both_nan = np.isnan(a) & np.isnan(b)
        same = (a.view(np.uint32) == b.view(np.uint32)) | both_nan
        if not same.all():
            i = np.flatnonzero(~same)[0]
            raise AssertionError(f"{what}: w[{k}] differs at {np.count_nonzero(~same)} "
                                 f"positions, first {i}: gpu {a[i]!r} oracle {b[i]!r}")
    for name in ("mq", "ma", "vq", "va"):
        for k, (a, b) in enumerate(zip(getattr(got, name), getattr(ref, name))):
            if a.tobytes() != b.tobytes():
                bad = np.flatnonzero(a.view(np.uint8 if a.itemsize == 1 else np.uint32) !=
                                     b.view(np.uint8 if b.itemsize == 1 else np.uint32))
                raise AssertionError(f"{what}: {name}[{k}] differs at {bad.size} positions, "
                                     f"first {bad[0]}: gpu {a[bad[0]]!r} oracle {b[bad[0]]!r}")


@pytest.mark.parametrize("block", [64, 128, 256, 512, 2048])
@pytest.mark.parametrize("code_map", [lt.LT_MAP_LINEAR, lt.LT_MAP_DYNAMIC])
@pytest.mark.parametrize("coef", [None, 0.37])
def test_step_on_extreme_and_corrupted_states(block, code_map, coef):
    w, g, mq, ma, vq, va = _edge_problem(block, code_map, seed=block + 7 * code_map)
    ref = State([w.copy()], [mq.copy()], [ma.copy()], [vq.copy()], [va.copy()])
    oracle.hybrid8bit_adamw_step(ref.w, [g], ref.mq, ref.ma, ref.vq, ref.va, block, step=5,
                                 coef=coef, code_map=code_map, **HYPER)
    dev = State([to_dev(w)], [to_dev(mq)], [to_dev(ma)], [to_dev(vq)], [to_dev(va)])
    c = None if coef is None else torch.tensor([coef], dtype=torch.float32, device=DEV)
    lt.lt_hybrid8bit_adamw_step(dev.w, [to_dev(g)], dev.mq, dev.ma, dev.vq, dev.va, block,
                                step=5, coef=c, code_map=code_map, **HYPER)
    torch.cuda.synchronize()
    got = dev.to_host()
    _assert_equal_nan_aware(got, ref, f"block {block}, map {code_map}, coef {coef}")
    # the stored scales are never NaN or infinite, whatever came in
    assert np.all(np.isfinite(got.ma[0])) and np.all(np.isfinite(got.va[0]))


def test_fp32_state_step_on_extreme_values():
    rng = np.random.default_rng(5)
    n = 5000
    w = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    v = (rng.uniform(0, 1, n) * 1e-6).astype(np.float32)
    idx = rng.choice(n, size=60, replace=False)
    w[idx[:6]], w[idx[6:12]], w[idx[12:18]] = np.nan, np.inf, -0.0
    m[idx[18:24]], m[idx[24:30]] = np.nan, -np.inf
    v[idx[30:36]], v[idx[36:42]] = -np.float32(1e-6), np.inf     # negative and infinite v
    v[idx[42:48]] = SUB
    g[idx[48:54]], g[idx[54:60]] = SUB, np.float32(3e38)
    dw, dm, dv = to_dev(w), to_dev(m), to_dev(v)
    lt.lt_adamw_fp32_step([dw], [to_dev(g)], [dm], [dv], step=3, **HYPER)
    torch.cuda.synchronize()
    oracle.adamw_fp32_step(w, g, m, v, step=3, coef=1.0, **HYPER)
    for a, b, name in ((dw, w, "w"), (dm, m, "m"), (dv, v, "v")):
        a = a.cpu().numpy()
        same = (a.view(np.uint32) == b.view(np.uint32)) | (np.isnan(a) & np.isnan(b))
        assert same.all(), f"{name} differs at {np.flatnonzero(~same)[:5]}"
