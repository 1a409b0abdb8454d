"""The dynamic code map in the fused step against the oracle, bitwise: random
sign-magnitude and unsigned codes with random scales over ragged tensors at
every block size (fp32 and bf16 gradients, clipped, two consecutive steps); an
encoder sweep in which beta1 = beta2 = 0 and a unit absmax make the normalized
moments the gradients themselves (every bucket edge of the kernel's lookup,
every code value and every midpoint between codes, with fp32 neighbours); and
the layer-streamed step with the dynamic map."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, assert_state_equal, gpu_norm_and_coef, oracle_step, \
    to_dev, to_host

pytestmark = pytest.mark.gpu

SIZES = [1, 7, 8, 9, 63, 64, 65, 1023, 2048, 2049, 4096, 8191, 8193, 65537]
DYN = lt.LT_MAP_DYNAMIC


def _random_state(rng, sizes, block):
    w = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in sizes]
    st = State.zero_host(w, block)
    for k, n in enumerate(sizes):
        st.mq[k][:] = rng.integers(-128, 128, size=n)
        st.vq[k][:] = rng.integers(0, 256, size=n)
        st.ma[k][:] = rng.uniform(0.1, 5.0, size=st.ma[k].size) * 1e-3
        st.va[k][:] = rng.uniform(0.1, 5.0, size=st.va[k].size) * 1e-6
    return st


@pytest.mark.parametrize("block", [64, 128, 256, 512, 1024, 2048, 4096, 8192])
@pytest.mark.parametrize("as_bf16", [False, True])
def test_dynamic_step_matches_oracle(block, as_bf16):
    rng = np.random.default_rng(block * 2 + as_bf16)
    st = _random_state(rng, SIZES, block)
    ref = st.copy()
    dev = st.to_dev()
    for t in (5, 6):
        g = [(rng.standard_t(3, size=n) * 1e-3).astype(np.float32) for n in SIZES]
        if as_bf16:
            g = [f32_to_bf16_bits(x) for x in g]
        gdev = [to_dev(x) for x in g]
        _, _, status, _, coef = gpu_norm_and_coef(gdev, 0.05)
        lt.lt_hybrid8bit_adamw_step(dev.w, gdev, dev.mq, dev.ma, dev.vq, dev.va, block, step=t,
                                    coef=coef, status=status, code_map=DYN, **HYPER)
        _, S, sto = oracle.grad_sqnorm(g, n_threads=8)
        _, c = oracle.clip_coef(S, 0.05)
        oracle.hybrid8bit_adamw_step(ref.w, g, ref.mq, ref.ma, ref.vq, ref.va, block, step=t,
                                     coef=float(c), status=sto, n_threads=8, code_map=DYN,
                                     **HYPER)
        torch.cuda.synchronize()
        assert_state_equal(dev.to_host(), ref, f"dynamic map, block {block}, t={t}")


def _sweep_values():
    """Normalized magnitudes that probe the kernel's encoder."""
    vals = []
    for bits, base_exp in ((7, 21), (8, 25)):
        base = (127 - base_exp) << 7
        top = (127 << 7) - base
        u = ((base + np.arange(top + 2, dtype=np.int64)) << 16).astype(np.uint32)
        for d in (-1, 0, 1):
            vals.append((u.astype(np.int64) + d).astype(np.uint32).view(np.float32))
        t = oracle.dynamic_map(bits == 7).astype(np.float64)
        mids = ((t[1:] + t[:-1]) / 2).astype(np.float32).view(np.uint32).astype(np.int64)
        codes = t.astype(np.float32).view(np.uint32).astype(np.int64)
        for d in range(-2, 3):
            vals.append((mids + d).astype(np.uint32).view(np.float32))
            vals.append(np.clip(codes + d, 0, None).astype(np.uint32).view(np.float32))
    v = np.concatenate(vals)
    v = v[(v >= 0) & (v <= 1)]
    return v


def test_encoder_sweep_matches_oracle():
    block = 2048
    vals = _sweep_values()
    per = block - 1
    nb = -(-vals.size // per)
    g = np.zeros(nb * block, np.float32)
    for b in range(nb):
        chunk = vals[b * per:(b + 1) * per]
        g[b * block] = 1.0  # unit absmax in every block
        sign = np.where(np.arange(chunk.size) % 2 == 0, 1, -1).astype(np.float32)
        g[b * block + 1:b * block + 1 + chunk.size] = chunk * sign
    n = g.size
    hyper = dict(HYPER, beta1=0.0, beta2=0.0)
    st = State.zero_host([np.zeros(n, np.float32)], block)
    ref = st.copy()
    dev = st.to_dev()
    lt.lt_hybrid8bit_adamw_step(dev.w, [to_dev(g)], dev.mq, dev.ma, dev.vq, dev.va, block,
                                step=1, code_map=DYN, **hyper)
    oracle.hybrid8bit_adamw_step(ref.w, [g], ref.mq, ref.ma, ref.vq, ref.va, block, step=1,
                                 n_threads=8, code_map=DYN, **hyper)
    torch.cuda.synchronize()
    got = dev.to_host()
    assert np.all(ref.ma[0] == 1.0)
    assert_state_equal(got, ref, "encoder sweep")


def test_streamed_dynamic_equals_resident():
    rng = np.random.default_rng(91)
    sizes = [4097, 65537, 9, 300001, 2048, 1]
    first = [0, 2, 4, 6]
    block = 2048
    base = _random_state(rng, sizes, block)
    g = [f32_to_bf16_bits((rng.standard_t(3, size=n) * 1e-3).astype(np.float32)) for n in sizes]
    pin = lambda a: torch.from_numpy(a).pin_memory()
    host = State(*[[pin(a.copy()) for a in lst] for lst in (base.w, base.mq, base.ma, base.vq,
                                                            base.va)])
    g_pin = [torch.from_numpy(x.view(np.int16)).pin_memory().view(torch.bfloat16) for x in g]
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    lt.lt_streamed_hybrid8bit_adamw_step(host.w, g_pin, host.mq, host.ma, host.vq, host.va,
                                         first, block, step=2, max_norm=1.0, ring_slots=2,
                                         sq_total=S, coef=coef, status=status, code_map=DYN,
                                         **HYPER)
    torch.cuda.synchronize()
    ref = base.copy()
    _, S_o, st_o = oracle.grad_sqnorm(g, n_threads=8)
    _, c_o = oracle.clip_coef(S_o, 1.0)
    oracle.hybrid8bit_adamw_step(ref.w, g, ref.mq, ref.ma, ref.vq, ref.va, block, step=2,
                                 coef=float(c_o), status=st_o, n_threads=8, code_map=DYN,
                                 **HYPER)
    got = State(*[[t.numpy() for t in lst] for lst in (host.w, host.mq, host.ma, host.vq,
                                                        host.va)])
    assert_state_equal(got, ref, "streamed dynamic vs oracle")


def test_rejects_unknown_code_map():
    w = [torch.zeros(16, device=DEV)]
    g = [torch.zeros(16, dtype=torch.bfloat16, device=DEV)]
    q = [torch.zeros(16, dtype=torch.int8, device=DEV)]
    u = [torch.zeros(16, dtype=torch.uint8, device=DEV)]
    a = [torch.zeros(1, device=DEV)]
    with pytest.raises(lt.LazyTrainError):
        lt.lt_hybrid8bit_adamw_step(w, g, q, a, u, a, 2048, step=1, code_map=2, **HYPER)


def test_hand_worked_dynamic_examples():
    """The exact blocks of tests/golden/dynamic_map_worked_examples.txt through the
    HIP path (each 4-element block is one partial block at the GPU's block size 64; an
    example worked with eps = 0 runs with the smallest positive eps, see golden_eps)."""
    from golden_io import adamw_examples
    from gpu_helpers import golden_eps
    n = 0
    for ex in adamw_examples("dynamic_map_worked_examples.txt"):
        st = State([ex["w"].copy()], [ex["m_codes"].copy()], [ex["m_absmax"].copy()],
                   [ex["v_codes"].copy()], [ex["v_absmax"].copy()]).to_dev()
        c = torch.tensor([ex["coef"]], dtype=torch.float32, device=DEV)
        lt.lt_hybrid8bit_adamw_step(st.w, [to_dev(ex["grad"].copy())], st.mq, st.ma, st.vq,
                                    st.va, 64, step=ex["t"], coef=c, code_map=DYN,
                                    lr=ex["lr"], beta1=ex["beta1"], beta2=ex["beta2"],
                                    eps=golden_eps(ex, oracle.MAP_DYNAMIC),
                                    weight_decay=ex["weight_decay"])
        got = st.to_host()
        assert np.array_equal(got.w[0], ex["expect_w"]), ex["name"]
        assert np.array_equal(got.mq[0], ex["expect_m_codes"]), ex["name"]
        assert np.array_equal(got.vq[0], ex["expect_v_codes"]), ex["name"]
        assert got.ma[0][0] == ex["expect_m_absmax"][0], ex["name"]
        assert got.va[0][0] == ex["expect_v_absmax"][0], ex["name"]
        n += 1
    assert n == 2
