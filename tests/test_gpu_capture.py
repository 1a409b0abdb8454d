"""Descriptor caching at the boundary.  A list call repeated over the same tensors
and workspace finds its descriptors in place and enqueues kernels only, so:

* the whole step (sum of squares -> clip -> fused step) captures into one HIP
  graph; every replay, with new gradients written by eager work in between, is
  bitwise the oracle's step and the same calls made eagerly on a twin state;
* fifty steps enqueue behind a busy GPU without the host waiting for it;
* a workspace written behind the library's back is detected by the kernels (the
  tag in its first word) instead of followed: the norm reports
  LT_STATUS_BAD_WORKSPACE, the step writes nothing; after lt_workspace_release
  the next calls copy the descriptors again and are exact."""
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from golden_io import f32_to_bf16_bits
from gpu_helpers import DEV, HYPER, State, assert_state_equal, to_dev, to_host

pytestmark = pytest.mark.gpu

SIZES = [2048 * 5 + 17, 64, 9000, 2048 * 2, 333, 100003]


def _start(seed, block):
    rng = np.random.default_rng(seed)
    w0 = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in SIZES]
    return rng, State.zero_host(w0, block)


def _grads(rng):
    return [f32_to_bf16_bits((rng.standard_t(3, size=n) * 1e-2).astype(np.float32))
            for n in SIZES]


class Step:
    """The three calls of one step over fixed device buffers and workspaces."""

    def __init__(self, state_dev, block, code_map):
        self.d, self.B, self.map = state_dev, block, code_map
        self.g = [torch.zeros(n, dtype=torch.bfloat16, device=DEV) for n in SIZES]
        self.ws_sq = torch.empty(lt.lt_grad_sqnorm_workspace_bytes(SIZES), dtype=torch.uint8,
                                 device=DEV)
        self.ws_st = torch.empty(lt.lt_step_workspace_bytes(len(SIZES)), dtype=torch.uint8,
                                 device=DEV)
        self.S = torch.zeros(1, dtype=torch.float64, device=DEV)
        self.status = torch.zeros(1, dtype=torch.int32, device=DEV)
        self.coef = torch.zeros(1, dtype=torch.float32, device=DEV)

    def load(self, host_grads):
        for buf, x in zip(self.g, host_grads):
            buf.copy_(to_dev(x))

    def __call__(self, t, max_norm=1.0):
        d = self.d
        lt.lt_grad_sqnorm(self.g, self.S, self.status, workspace=self.ws_sq)
        lt.lt_clip_coef(self.S, max_norm, self.coef)
        lt.lt_hybrid8bit_adamw_step(d.w, self.g, d.mq, d.ma, d.vq, d.va, self.B, step=t,
                                    coef=self.coef, status=self.status, workspace=self.ws_st,
                                    code_map=self.map, **HYPER)

    def release(self):
        lt.lt_workspace_release(self.ws_sq)
        lt.lt_workspace_release(self.ws_st)


def _oracle(ref, g, block, t, omap, max_norm=1.0):
    _, S, st = oracle.grad_sqnorm(g, n_threads=8)
    _, c = oracle.clip_coef(S, max_norm)
    oracle.hybrid8bit_adamw_step(ref.w, g, ref.mq, ref.ma, ref.vq, ref.va, block, step=t,
                                 coef=float(c), status=st, n_threads=8, code_map=omap, **HYPER)
    return S, c


@pytest.mark.parametrize("block,code_map", [(2048, lt.LT_MAP_LINEAR), (2048, lt.LT_MAP_DYNAMIC),
                                            (3072, lt.LT_MAP_LINEAR)])
def test_whole_step_captured_in_one_graph(block, code_map):
    omap = oracle.MAP_DYNAMIC if code_map == lt.LT_MAP_DYNAMIC else oracle.MAP_LINEAR
    rng, ref = _start(7, block)
    step, twin = Step(ref.to_dev(), block, code_map), Step(ref.to_dev(), block, code_map)
    t = 2
    g = _grads(rng)
    for s in (step, twin):  # the uncaptured first calls copy the descriptors in
        s.load(g)
        s(t)
    _oracle(ref, g, block, t, omap)
    torch.cuda.synchronize()
    assert_state_equal(step.d.to_host(), ref, "eager first step")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(t)
    assert_state_equal(step.d.to_host(), ref, "capturing runs nothing")
    for r in range(4):
        g = _grads(rng)
        step.load(g)
        twin.load(g)
        torch.cuda.synchronize()
        graph.replay()
        twin(t)  # the same calls, eagerly, on the twin state
        torch.cuda.synchronize()
        S, c = _oracle(ref, g, block, t, omap)
        assert to_host(step.S)[0].hex() == S.hex() and to_host(step.coef)[0] == c
        got = step.d.to_host()
        assert_state_equal(got, ref, f"replay {r}")
        assert_state_equal(twin.d.to_host(), got, f"eager twin, replay {r}")
    del graph


def test_a_captured_call_without_descriptors_in_place_is_refused():
    rng, ref = _start(8, 2048)
    step = Step(ref.to_dev(), 2048, lt.LT_MAP_LINEAR)
    step.load(_grads(rng))
    torch.cuda.synchronize()
    lt.lt_workspace_release(step.ws_sq)  # whatever this address held before: forgotten
    graph = torch.cuda.CUDAGraph()
    with pytest.raises(lt.LazyTrainError) as e:
        with torch.cuda.graph(graph):
            step.coef.add_(0.0)  # the graph holds a node either way
            lt.lt_grad_sqnorm(step.g, step.S, step.status, workspace=step.ws_sq)
    assert e.value.code == lt.LT_ERR_INVALID_ARG and "captur" in str(e.value)
    torch.cuda.synchronize()
    del graph
    # the same call uncaptured works, and is exact
    lt.lt_grad_sqnorm(step.g, step.S, step.status, workspace=step.ws_sq)
    torch.cuda.synchronize()
    g = [to_host(x) for x in step.g]
    assert to_host(step.S)[0].hex() == oracle.grad_sqnorm(g)[1].hex()


def _sleep_cycles_for(ms):
    """Cycles of torch's spin kernel that last about `ms` on this GPU (bounded)."""
    probe = 10_000_000
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    torch.cuda._sleep(probe)
    b.record()
    b.synchronize()
    per_ms = probe / max(a.elapsed_time(b), 1e-3)
    return int(min(per_ms * ms, 300 * probe))


def test_fifty_steps_enqueue_without_waiting_for_the_gpu():
    block = 2048
    rng, ref = _start(9, block)
    step = Step(ref.to_dev(), block, lt.LT_MAP_LINEAR)
    g = _grads(rng)
    step.load(g)
    step(1)  # descriptors copied in
    _oracle(ref, g, block, 1, oracle.MAP_LINEAR)
    torch.cuda.synchronize()
    cycles = _sleep_cycles_for(3000.0)
    done = torch.cuda.Event()
    t0 = time.perf_counter()
    torch.cuda._sleep(cycles)  # the GPU is busy for about three seconds
    for t in range(2, 52):
        step(t)
    done.record()
    enqueue_s = time.perf_counter() - t0
    still_busy = not done.query()
    torch.cuda.synchronize()
    total_s = time.perf_counter() - t0
    print(f"enqueue of 50 steps {enqueue_s * 1e3:.1f} ms, all done after {total_s * 1e3:.0f} ms",
          flush=True)
    assert still_busy, "the GPU finished before the host had enqueued the steps"
    assert enqueue_s < 0.5 * total_s
    for t in range(2, 52):
        _oracle(ref, g, block, t, oracle.MAP_LINEAR)
    assert_state_equal(step.d.to_host(), ref, "after 51 steps")


def test_a_workspace_written_behind_the_librarys_back_is_not_followed():
    block = 2048
    rng, ref = _start(10, block)
    step = Step(ref.to_dev(), block, lt.LT_MAP_LINEAR)
    g = _grads(rng)
    step.load(g)
    step(1)
    _oracle(ref, g, block, 1, oracle.MAP_LINEAR)
    torch.cuda.synchronize()
    before = step.d.to_host()
    assert_state_equal(before, ref, "first step")
    # overwrite only the tag words: the descriptors stay valid, so nothing could
    # fault even if a kernel followed them
    step.ws_sq[:8].fill_(0xA5)
    step.ws_st[:8].fill_(0xA5)
    step(2)
    torch.cuda.synchronize()
    assert int(to_host(step.status)[0]) == lt.LT_STATUS_BAD_WORKSPACE
    assert np.isnan(to_host(step.S)[0])
    assert_state_equal(step.d.to_host(), before, "stale workspaces: nothing written")
    # the step alone (no status) with its stale workspace writes nothing either
    lt.lt_hybrid8bit_adamw_step(step.d.w, step.g, step.d.mq, step.d.ma, step.d.vq, step.d.va,
                                block, step=2, workspace=step.ws_st, **HYPER)
    torch.cuda.synchronize()
    assert_state_equal(step.d.to_host(), before, "stale step workspace")
    step.release()
    step.status.zero_()
    step(2)  # descriptors copied in again
    _oracle(ref, g, block, 2, oracle.MAP_LINEAR)
    torch.cuda.synchronize()
    assert int(to_host(step.status)[0]) == lt.LT_STATUS_OK
    assert_state_equal(step.d.to_host(), ref, "after release")


def test_clip_coef_status_argument():
    """lt_clip_coef sets the status from S unless it holds a library error."""
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    for s, prior, want in ((4.0, lt.LT_STATUS_NONFINITE, lt.LT_STATUS_OK),
                           (float("inf"), lt.LT_STATUS_OK, lt.LT_STATUS_NONFINITE),
                           (float("nan"), lt.LT_STATUS_OK, lt.LT_STATUS_NONFINITE),
                           (4.0, lt.LT_STATUS_BAD_WORKSPACE, lt.LT_STATUS_BAD_WORKSPACE),
                           (4.0, 77, 77)):
        S.fill_(s)
        st.fill_(prior)
        lt.lt_clip_coef(S, 1.0, coef, status=st)
        assert lt.lt_read_status(st) == want, (s, prior)


def test_a_freed_workspace_is_forgotten():
    """A workspace tensor freed and allocated again at the same address (torch's
    caching allocator hands the same block back) gets its descriptors copied in again:
    the binding releases freed workspaces.  Memory written in between by another
    tensor would otherwise leave a stale tag and a skipped step."""
    block = 2048
    rng, ref = _start(11, block)
    d = ref.to_dev()
    g = _grads(rng)
    gd = [to_dev(x) for x in g]
    n = lt.lt_step_workspace_bytes(len(SIZES))
    addrs = set()
    for t in (1, 2, 3):
        ws = torch.empty(n, dtype=torch.uint8, device=DEV)
        addrs.add(ws.data_ptr())
        lt.lt_hybrid8bit_adamw_step(d.w, gd, d.mq, d.ma, d.vq, d.va, block, step=t, workspace=ws,
                                    **HYPER)
        oracle.hybrid8bit_adamw_step(ref.w, g, ref.mq, ref.ma, ref.vq, ref.va, block, step=t,
                                     n_threads=8, **HYPER)
        torch.cuda.synchronize()
        assert_state_equal(d.to_host(), ref, f"step {t}")
        del ws
        junk = torch.full((n,), 0x5A, dtype=torch.uint8, device=DEV)  # reuses the block
        torch.cuda.synchronize()
        del junk
    print(f"workspace addresses seen: {len(addrs)}", flush=True)
