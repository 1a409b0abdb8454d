"""A single tensor of more than 2^31 elements (64-bit indexing through every
kernel): the sum of squares bitwise against the oracle over the whole tensor, and
the step bitwise on sampled blocks on both sides of element 2^31 and at the
ragged end, which the oracle recomputes one by one."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
import synth
from gpu_helpers import DEV, HYPER, to_host

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

N = (1 << 31) + 12345
BLOCK = 2048


def test_tensor_beyond_two_to_the_31_elements():
    seed, stream = 21, synth.grad_stream(1)
    n_threads = synth.default_threads()
    g = synth.draw(synth.BF16, N, seed, stream, 0, synth.Recipe(synth.STUDENT_T3, 1e-3),
                   n_threads=n_threads)
    w = synth.draw(synth.F32, N, seed, synth.STREAM_WEIGHTS, 0, synth.Recipe(synth.NORMAL, 0.02),
                   n_threads=n_threads)
    gd = torch.from_numpy(g.view(np.int16)).to(DEV).view(torch.bfloat16)
    wd = torch.from_numpy(w).to(DEV)
    nb = -(-N // BLOCK)
    mq = torch.zeros(N, dtype=torch.int8, device=DEV)
    vq = torch.zeros(N, dtype=torch.uint8, device=DEV)
    ma = torch.zeros(nb, dtype=torch.float32, device=DEV)
    va = torch.zeros(nb, dtype=torch.float32, device=DEV)
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    lt.lt_grad_sqnorm([gd], S, status)
    lt.lt_clip_coef(S, 1.0, coef)
    lt.lt_hybrid8bit_adamw_step([wd], [gd], [mq], [ma], [vq], [va], BLOCK, step=1, coef=coef,
                                status=status, **HYPER)
    torch.cuda.synchronize()
    _, S_o, st_o = oracle.grad_sqnorm([g], n_threads=n_threads)
    _, c_o = oracle.clip_coef(S_o, 1.0)
    assert to_host(S)[0].hex() == float(S_o).hex() and st_o == 0
    assert to_host(coef)[0] == c_o
    edge = (1 << 31) // BLOCK
    blocks = sorted({0, 1, edge - 2, edge - 1, edge, edge + 1, nb - 2, nb - 1} |
                    set(int(b) for b in np.random.default_rng(3).integers(0, nb, size=40)))
    for b in blocks:
        lo, hi = b * BLOCK, min(N, (b + 1) * BLOCK)
        ww = w[lo:hi].copy()
        qm, qv = np.zeros(hi - lo, np.int8), np.zeros(hi - lo, np.uint8)
        am, av = np.zeros(1, np.float32), np.zeros(1, np.float32)
        oracle.hybrid8bit_adamw_step([ww], [g[lo:hi]], [qm], [am], [qv], [av], BLOCK, step=1,
                                     coef=float(c_o), status=st_o, **HYPER)
        assert to_host(wd[lo:hi]).tobytes() == ww.tobytes(), b
        assert to_host(mq[lo:hi]).tobytes() == qm.tobytes(), b
        assert to_host(vq[lo:hi]).tobytes() == qv.tobytes(), b
        assert to_host(ma[b:b + 1])[0] == am[0] and to_host(va[b:b + 1])[0] == av[0], b
