"""Block sizes outside the fast kernels' powers of two (any multiple of 64 up to
65536; the boundary's domain, which holds the paper's 4096): the generic step
kernel against the oracle, bitwise, with both code maps, bf16 and fp32 gradients,
ragged tensors (shorter than one block, a partial last block, a partial last
granule), clipping, two consecutive steps, the bf16 weight copy, and the
non-finite skip.  Sizes above 8192 take the path that recomputes the moments in
its second pass instead of keeping them in LDS."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, assert_state_equal, gpu_norm_and_coef, to_dev, to_host

pytestmark = pytest.mark.gpu

BLOCKS = [192, 576, 3072, 12288, 16384, 65536]


def _sizes(B):
    return [1, 7, 63, 64, B - 1, B, B + 9, 2 * B + 64, 3 * B - 5, 100003]


def _state(sizes, B, rng):
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    st = State.zero_host(w, B)
    for k, n in enumerate(sizes):
        st.mq[k][:] = rng.integers(-127, 128, size=n)
        st.vq[k][:] = rng.integers(0, 256, size=n)
        nb = st.ma[k].size
        st.ma[k][:] = rng.uniform(0.1, 5.0, size=nb) * 1e-3
        st.va[k][:] = rng.uniform(0.1, 5.0, size=nb) * 1e-6
        z = rng.random(nb) < 0.1
        st.ma[k][z] = 0
        st.va[k][z] = 0
    return st


def _grads(rng, sizes, as_bf16):
    g32 = [(rng.standard_t(3, size=n) * 1e-3).astype(np.float32) for n in sizes]
    return [f32_to_bf16_bits(g) for g in g32] if as_bf16 else g32


@pytest.mark.parametrize("B", BLOCKS)
@pytest.mark.parametrize("code_map", [lt.LT_MAP_LINEAR, lt.LT_MAP_DYNAMIC])
@pytest.mark.parametrize("as_bf16", [False, True])
def test_generic_block_sizes_two_clipped_steps(B, code_map, as_bf16):
    rng = np.random.default_rng(B + 3 * code_map + (1 if as_bf16 else 0))
    sizes = _sizes(B)
    omap = oracle.MAP_DYNAMIC if code_map == lt.LT_MAP_DYNAMIC else oracle.MAP_LINEAR
    ref = _state(sizes, B, rng)
    dev = ref.to_dev()
    for t in (3, 4):
        g = _grads(rng, sizes, as_bf16)
        gd = [to_dev(x) for x in g]
        _, S, status, _, coef = gpu_norm_and_coef(gd, 0.05)
        lt.lt_hybrid8bit_adamw_step(dev.w, gd, dev.mq, dev.ma, dev.vq, dev.va, B, step=t,
                                    coef=coef, status=status, code_map=code_map, **HYPER)
        _, rS, rst = oracle.grad_sqnorm(g, n_threads=8)
        _, rc = oracle.clip_coef(rS, 0.05)
        assert rc < 1.0  # clipping is active
        oracle.hybrid8bit_adamw_step(ref.w, g, ref.mq, ref.ma, ref.vq, ref.va, B, step=t,
                                     coef=float(rc), status=rst, n_threads=8, code_map=omap,
                                     **HYPER)
        assert_state_equal(dev.to_host(), ref, f"block {B}, map {code_map}, t = {t}")


@pytest.mark.parametrize("B", [3072, 16384])
def test_generic_bf16_copy_and_skip(B):
    rng = np.random.default_rng(B)
    sizes = _sizes(B)
    ref = _state(sizes, B, rng)
    dev = ref.to_dev()
    copies = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    g = _grads(rng, sizes, True)
    gd = [to_dev(x) for x in g]
    _, S, status, _, coef = gpu_norm_and_coef(gd, 1.0)
    lt.lt_hybrid8bit_adamw_step(dev.w, gd, dev.mq, dev.ma, dev.vq, dev.va, B, step=2, coef=coef,
                                status=status, params_bf16=copies, **HYPER)
    _, rS, rst = oracle.grad_sqnorm(g, n_threads=8)
    _, rc = oracle.clip_coef(rS, 1.0)
    oracle.hybrid8bit_adamw_step(ref.w, g, ref.mq, ref.ma, ref.vq, ref.va, B, step=2,
                                 coef=float(rc), status=rst, n_threads=8, **HYPER)
    got = dev.to_host()
    assert_state_equal(got, ref, f"block {B}")
    for c, w in zip(copies, ref.w):
        assert to_host(c).tobytes() == oracle.round_bf16(w).tobytes()
    # a non-finite gradient: nothing changes
    g[3][0] = 0x7F80  # +inf (bf16 bits)
    gd = [to_dev(x) for x in g]
    _, S, status, _, coef = gpu_norm_and_coef(gd, 1.0)
    assert lt.lt_read_status(status) == lt.LT_STATUS_NONFINITE
    lt.lt_hybrid8bit_adamw_step(dev.w, gd, dev.mq, dev.ma, dev.vq, dev.va, B, step=3, coef=coef,
                                status=status, params_bf16=copies, **HYPER)
    assert_state_equal(dev.to_host(), got, f"block {B}, skipped")


def test_generic_block_streamed_matches_resident():
    """The layer-streamed step at a generic block size: bitwise the resident step."""
    B = 3072
    rng = np.random.default_rng(5)
    sizes = [B * 5 + 17, 64, 9000, B * 2, 333]
    first = [0, 2, 5]
    ref = _state(sizes, B, rng)
    dev = ref.to_dev()
    g = _grads(rng, sizes, True)
    gd = [to_dev(x) for x in g]
    _, S, status, _, coef = gpu_norm_and_coef(gd, 1.0)
    lt.lt_hybrid8bit_adamw_step(dev.w, gd, dev.mq, dev.ma, dev.vq, dev.va, B, step=2, coef=coef,
                                status=status, **HYPER)
    host = State([torch.from_numpy(x.copy()).pin_memory() for x in ref.w],
                 [torch.from_numpy(x.copy()).pin_memory() for x in ref.mq],
                 [torch.from_numpy(x.copy()).pin_memory() for x in ref.ma],
                 [torch.from_numpy(x.copy()).pin_memory() for x in ref.vq],
                 [torch.from_numpy(x.copy()).pin_memory() for x in ref.va])
    gh = [torch.from_numpy(x.view(np.int16)).pin_memory().view(torch.bfloat16) for x in g]
    S2 = torch.zeros(1, dtype=torch.float64, device=DEV)
    c2 = torch.zeros(1, dtype=torch.float32, device=DEV)
    st2 = torch.zeros(1, dtype=torch.int32, device=DEV)
    cs = torch.cuda.Stream(DEV)
    cs.wait_stream(torch.cuda.current_stream())
    lt.lt_streamed_hybrid8bit_adamw_step(host.w, gh, host.mq, host.ma, host.vq, host.va, first, B,
                                         step=2, max_norm=1.0, ring_slots=2, sq_total=S2,
                                         coef=c2, status=st2, compute_stream=cs, **HYPER)
    cs.synchronize()
    as_np = State(*[[t.numpy() for t in lst] for lst in (host.w, host.mq, host.ma, host.vq,
                                                          host.va)])
    assert_state_equal(as_np, dev.to_host(), "streamed vs resident, block 3072")
