"""Helpers shared by the GPU parity tests: host<->device copies and the two sides of
one clipped Hybrid 8-bit step (the HIP path through the C ABI binding, the oracle
on host copies of the same generator output)."""
import numpy as np
import torch

import oracle
import paper_2608_11919_amd as lt

DEV = torch.device("cuda", 0)


def to_dev(a: np.ndarray) -> torch.Tensor:
    """Host array -> device tensor; uint16 arrays are bf16 bits."""
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def to_host(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


class State:
    """Weights and 8-bit states of a tensor list, on host (numpy) or device (torch)."""

    def __init__(self, w, mq, ma, vq, va):
        self.w, self.mq, self.ma, self.vq, self.va = w, mq, ma, vq, va

    @staticmethod
    def zero_host(weights, block):
        nb = [-(-x.size // block) for x in weights]
        return State([x.copy() for x in weights], [np.zeros(x.size, np.int8) for x in weights],
                     [np.zeros(n, np.float32) for n in nb],
                     [np.zeros(x.size, np.uint8) for x in weights],
                     [np.zeros(n, np.float32) for n in nb])

    def to_dev(self):
        return State(*[[to_dev(a) for a in lst] for lst in
                       (self.w, self.mq, self.ma, self.vq, self.va)])

    def to_host(self):
        return State(*[[to_host(a) for a in lst] for lst in
                       (self.w, self.mq, self.ma, self.vq, self.va)])

    def copy(self):
        return State(*[[a.copy() for a in lst] for lst in
                       (self.w, self.mq, self.ma, self.vq, self.va)])


HYPER = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)

# The smallest positive fp32.  Hand-worked golden blocks use eps = 0 to keep their
# arithmetic exact; the library requires eps > 0, and on those blocks the oracle gives
# the same bits with this eps (golden_eps checks it per example).
EPS_MIN = 2.0 ** -149


def golden_eps(ex, code_map=None):
    """The eps to run a golden example with on the GPU: its own, or EPS_MIN in place
    of 0 after checking that the oracle then still gives the example's expected bits."""
    if ex["eps"] != 0:
        return ex["eps"]
    names = ("w", "m_codes", "m_absmax", "v_codes", "v_absmax")
    w, mq, ma, vq, va = ([ex[k].copy()] for k in names)
    kw = {} if code_map is None else {"code_map": code_map}
    oracle.hybrid8bit_adamw_step(w, [ex["grad"].copy()], mq, ma, vq, va, ex["block_size"],
                                 step=ex["t"], coef=ex["coef"], lr=ex["lr"], beta1=ex["beta1"],
                                 beta2=ex["beta2"], eps=EPS_MIN,
                                 weight_decay=ex["weight_decay"], **kw)
    for k, got in zip(names, (w, mq, ma, vq, va)):
        assert got[0].tobytes() == ex["expect_" + k].tobytes(), (ex["name"], k)
    return EPS_MIN


def oracle_step(st: State, grads, block, step, coef=None, status=None, n_threads=8, **hyper):
    h = dict(HYPER, **hyper)
    oracle.hybrid8bit_adamw_step(st.w, grads, st.mq, st.ma, st.vq, st.va, block, step=step,
                                 coef=coef, status=status, n_threads=n_threads, **h)


def gpu_step(st: State, grads, block, step, coef=None, status=None, **hyper):
    h = dict(HYPER, **hyper)
    lt.lt_hybrid8bit_adamw_step(st.w, grads, st.mq, st.ma, st.vq, st.va, block, step=step,
                                coef=coef, status=status, **h)


def gpu_norm_and_coef(grads_dev, max_norm):
    """Returns device tensors (S_k, S, status, norm, coef) after a1-a3."""
    K = len(grads_dev)
    sk = torch.empty(K, dtype=torch.float64, device=DEV)
    S = torch.empty(1, dtype=torch.float64, device=DEV)
    status = torch.empty(1, dtype=torch.int32, device=DEV)
    norm = torch.empty(1, dtype=torch.float32, device=DEV)
    coef = torch.empty(1, dtype=torch.float32, device=DEV)
    lt.lt_grad_sqnorm(grads_dev, S, status, sq_per_tensor=sk)
    lt.lt_clip_coef(S, max_norm, coef, total_norm=norm)
    return sk, S, status, norm, coef


def assert_state_equal(gpu: State, ref: State, what=""):
    """Bitwise equality of weights, codes and absmax, with a readable failure."""
    for name in ("w", "mq", "ma", "vq", "va"):
        for k, (a, b) in enumerate(zip(getattr(gpu, name), getattr(ref, name))):
            if a.tobytes() != b.tobytes():
                bad = np.flatnonzero(a.view(np.uint8 if a.itemsize == 1 else np.uint32) !=
                                     b.view(np.uint8 if b.itemsize == 1 else np.uint32))
                i = bad[0]
                raise AssertionError(f"{what}: {name}[{k}] differs at {bad.size} positions, "
                                     f"first {i}: gpu {a[i]!r} oracle {b[i]!r}")


def check_stated_tolerance(gpu: State, ref: State, lr: float):
    """The stated bar, as a second check: weights within 1e-6 relative (floor lr),
    codes equal except +-1 at a rate <= 1e-6."""
    n_codes = mism = 0
    for a, b in zip(gpu.w, ref.w):
        d = np.abs(a.astype(np.float64) - b)
        assert np.all(d <= 1e-6 * np.maximum(np.abs(b), lr))
    for name in ("mq", "vq"):
        for a, b in zip(getattr(gpu, name), getattr(ref, name)):
            diff = np.abs(a.astype(np.int32) - b.astype(np.int32))
            assert diff.max(initial=0) <= 1
            mism += int(np.count_nonzero(diff))
            n_codes += a.size
    assert mism <= max(0, n_codes * 1e-6)
