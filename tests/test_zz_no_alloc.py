"""lt_grad_sqnorm_noalloc, the sum of squares that allocates nothing (its descriptors
and partial sums live in the library's own device scratch), against lt_grad_sqnorm
through the C ABI: S_k, S and the status bitwise, on two calls in a row (the second
with a smaller list, so the scratch holds the first call's larger contents), and
with the oracle as a second reference.  A list too large for the scratch is
rejected before any device work."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
import synth
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, to_dev, to_host

pytestmark = pytest.mark.gpu


def _c_call(fn, grads, gdt, sk, S, st, extra=()):
    K = len(grads)
    ptrs = (ctypes.c_void_p * K)(*[g.data_ptr() for g in grads])
    numels = (ctypes.c_int64 * K)(*[g.numel() for g in grads])
    return fn(ptrs, numels, K, gdt, *extra, sk.data_ptr(), S.data_ptr(), st.data_ptr(),
              torch.cuda.current_stream().cuda_stream)


def _both(host_grads, gdt):
    """(noalloc outputs, workspace-path outputs) for one list."""
    L = lt.lib()
    gd = [to_dev(g) for g in host_grads]
    K = len(gd)
    out = []
    for noalloc in (True, False):
        sk = torch.full((K,), -1.0, dtype=torch.float64, device=DEV)
        S = torch.full((1,), -1.0, dtype=torch.float64, device=DEV)
        st = torch.full((1,), -7, dtype=torch.int32, device=DEV)
        if noalloc:
            rc = _c_call(L.lt_grad_sqnorm_noalloc, gd, gdt, sk, S, st)
        else:
            nbytes = lt.lt_grad_sqnorm_workspace_bytes([g.numel() for g in gd])
            ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
            rc = _c_call(L.lt_grad_sqnorm, gd, gdt, sk, S, st, (ws.data_ptr(), nbytes))
        assert rc == lt.LT_OK, L.lt_last_error()
        torch.cuda.synchronize()
        out.append((to_host(sk), to_host(S), to_host(st)))
    return out


def _check(host_grads, gdt, what):
    (sk, S, st), (rsk, rS, rst) = _both(host_grads, gdt)
    assert sk.tobytes() == rsk.tobytes(), what
    assert S.tobytes() == rS.tobytes(), what
    assert st.tobytes() == rst.tobytes(), what
    osk, oS, ost = oracle.grad_sqnorm(host_grads, n_threads=8)
    assert sk.tobytes() == osk.tobytes() and S[0].hex() == oS.hex() and int(st[0]) == ost, what
    return S[0]


def test_two_calls_in_a_row_the_second_smaller():
    w = synth.layer_3b()  # 9 tensors, 77.1M parameters, bf16
    big = [w.grads(k, synth.grad_stream(2), n_threads=8) for k in range(len(w.numels))]
    _check(big, lt.LT_DTYPE_BF16, "3B-class layer")
    rng = np.random.default_rng(3)
    small = [f32_to_bf16_bits((rng.standard_t(3, size=n) * 1e-3).astype(np.float32))
             for n in (7, 8193, 100003)]
    _check(small, lt.LT_DTYPE_BF16, "three ragged tensors")
    f32 = [(rng.standard_normal(n) * 1e-2).astype(np.float32) for n in (1, 9000, 70001)]
    _check(f32, lt.LT_DTYPE_F32, "fp32 gradients")


def test_nonfinite_empty_and_many_tensors():
    rng = np.random.default_rng(4)
    g = [(rng.standard_normal(n) * 1e-2).astype(np.float32) for n in (5000, 0, 300)]
    g[2][17] = np.inf
    _check(g, lt.LT_DTYPE_F32, "an infinite gradient")
    many = [(rng.standard_normal(n) * 1e-2).astype(np.float32)
            for n in rng.integers(1, 3000, size=1500)]  # several descriptor launches
    _check(many, lt.LT_DTYPE_F32, "1500 tensors")
    (sk, S, st), _ = _both([], lt.LT_DTYPE_F32)
    assert S[0] == 0.0 and int(st[0]) == lt.LT_STATUS_OK


def test_a_list_too_large_for_the_scratch_is_rejected():
    L = lt.lib()
    ptrs = (ctypes.c_void_p * 1)(0x100000)  # never dereferenced: rejected first
    numels = (ctypes.c_int64 * 1)(1 << 36)  # 8.4 million chunks
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    rc = L.lt_grad_sqnorm_noalloc(ptrs, numels, 1, lt.LT_DTYPE_BF16, None, S.data_ptr(),
                                  st.data_ptr(), None)
    assert rc == lt.LT_ERR_INVALID_ARG and b"scratch" in L.lt_last_error()
