"""GPU parity of the layer-streamed step at the 27B-class size, in the launch
configuration bench.py times (27B-class decoder layers of hidden 5120, FFN 17408,
40q/8kv heads of 128; block 2048; a ring of 3 device slots on three streams).

* The whole model (64 layers, 21.1e9 parameters), as the benchmark streams it: the
  64 layers cycle over 8 distinct pinned host layers.  The first streamed pass and
  the finish run before anything is written back, so the global sum of squares,
  the norm and the clip coefficient over all 576 tensors are compared bitwise with
  the oracle's.  (Pass 2 writes the shared host state of several layers, so its
  results are not checked here.)
* Eight distinct layers (2.6e9 parameters, every tensor at its full size) from zero
  state, with the gradients copied in twice (linear map) and kept in HBM between the
  passes (dynamic map): S and the coefficient bitwise, and the updated weights, codes
  and scales of every block of every tensor against the oracle run over the same
  host data."""
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
import synth
from gpu_helpers import DEV, to_host

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

HOST_LAYERS = 8
PER_LAYER = 9


def _say(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


@pytest.fixture(scope="module")
def host_model():
    """Pinned host tensors of 8 distinct 27B-class layers: weights and bf16 gradients
    from the generator, zero 8-bit states."""
    w = synth.streamed_27b(HOST_LAYERS)
    n_threads = synth.default_threads()
    B = w.block_size
    h = {name: [] for name in ("w", "g", "mq", "ma", "vq", "va")}
    t0 = time.time()
    for k, n in enumerate(w.numels):
        nb = -(-n // B)
        wt = torch.empty(n, dtype=torch.float32, pin_memory=True)
        synth.fill_ptr(wt.data_ptr(), synth.F32, 0, n, w.seed, synth.STREAM_WEIGHTS, k,
                       w.weight_recipe, n_threads)
        gt = torch.empty(n, dtype=torch.bfloat16, pin_memory=True)
        synth.fill_ptr(gt.data_ptr(), synth.BF16, 0, n, w.seed, synth.grad_stream(w.step), k,
                       w.grad_recipe, n_threads)
        h["w"].append(wt)
        h["g"].append(gt)
        h["mq"].append(torch.zeros(n, dtype=torch.int8, pin_memory=True))
        h["vq"].append(torch.zeros(n, dtype=torch.uint8, pin_memory=True))
        h["ma"].append(torch.zeros(nb, dtype=torch.float32, pin_memory=True))
        h["va"].append(torch.zeros(nb, dtype=torch.float32, pin_memory=True))
    _say(f"8 host layers of 27B-class shape ready ({w.n_params} params, {time.time() - t0:.1f} s)")
    return w, h


def _outputs():
    return (torch.zeros(1, dtype=torch.float64, device=DEV),
            torch.zeros(1, dtype=torch.float32, device=DEV),
            torch.zeros(1, dtype=torch.float32, device=DEV),
            torch.zeros(1, dtype=torch.int32, device=DEV))


def _hyper(w):
    return dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay)


def _grad_bits(t):
    return t.view(torch.int16).numpy().view(np.uint16)


def test_whole_model_norm_and_coefficient_as_benchmarked(host_model):
    w8, h = host_model
    L = 64
    lists = {k: [v[(l % HOST_LAYERS) * PER_LAYER + j] for l in range(L) for j in range(PER_LAYER)]
             for k, v in h.items()}
    first = list(range(0, L * PER_LAYER + 1, PER_LAYER))
    S, coef, norm, status = _outputs()
    cs, hs, ds = torch.cuda.Stream(DEV), torch.cuda.Stream(DEV), torch.cuda.Stream(DEV)
    cs.wait_stream(torch.cuda.current_stream())
    _say("streamed step over 64 layers (21.1e9 params), ring of 3")
    lt.lt_streamed_hybrid8bit_adamw_step(lists["w"], lists["g"], lists["mq"], lists["ma"],
                                         lists["vq"], lists["va"], first, w8.block_size,
                                         step=w8.step, max_norm=w8.max_norm, ring_slots=3,
                                         sq_total=S, coef=coef, status=status, total_norm=norm,
                                         compute_stream=cs, h2d_stream=hs, d2h_stream=ds,
                                         **_hyper(w8))
    cs.synchronize()
    _say("oracle sum of squares over the 576 tensors")
    _, S_o, st_o = oracle.grad_sqnorm([_grad_bits(g) for g in lists["g"]],
                                      n_threads=synth.default_threads())
    n_o, c_o = oracle.clip_coef(S_o, w8.max_norm)
    assert int(to_host(status)[0]) == st_o == oracle.STATUS_OK
    assert to_host(S)[0].hex() == S_o.hex()
    assert to_host(norm)[0] == n_o and to_host(coef)[0] == c_o
    _say(f"S = {S_o!r}, norm {float(n_o):.6g}, coef {float(c_o):.6g}: bitwise equal")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("keep,code_map", [(False, lt.LT_MAP_LINEAR), (True, lt.LT_MAP_DYNAMIC)])
def test_eight_full_size_layers_against_oracle(host_model, keep, code_map):
    w8, h = host_model
    B = w8.block_size
    # fresh state: the weights from the generator, zero codes and scales
    n_threads = synth.default_threads()
    for k, n in enumerate(w8.numels):
        synth.fill_ptr(h["w"][k].data_ptr(), synth.F32, 0, n, w8.seed, synth.STREAM_WEIGHTS, k,
                       w8.weight_recipe, n_threads)
        for name in ("mq", "ma", "vq", "va"):
            h[name][k].zero_()
    first = list(range(0, len(w8.numels) + 1, PER_LAYER))
    S, coef, norm, status = _outputs()
    cs, hs, ds = torch.cuda.Stream(DEV), torch.cuda.Stream(DEV), torch.cuda.Stream(DEV)
    cs.wait_stream(torch.cuda.current_stream())
    _say(f"streamed step over 8 distinct full-size layers from zero state, t = 1, "
         f"gradients kept in HBM: {keep}, code map {code_map}")
    lt.lt_streamed_hybrid8bit_adamw_step(h["w"], h["g"], h["mq"], h["ma"], h["vq"], h["va"],
                                         first, B, step=1, max_norm=w8.max_norm, ring_slots=3,
                                         sq_total=S, coef=coef, status=status, total_norm=norm,
                                         compute_stream=cs, h2d_stream=hs, d2h_stream=ds,
                                         keep_grads=keep, code_map=code_map, **_hyper(w8))
    cs.synchronize()
    _, S_o, st_o = oracle.grad_sqnorm([_grad_bits(g) for g in h["g"]], n_threads=n_threads)
    _, c_o = oracle.clip_coef(S_o, w8.max_norm)
    assert int(to_host(status)[0]) == st_o == oracle.STATUS_OK
    assert to_host(S)[0].hex() == S_o.hex() and to_host(coef)[0] == c_o

    _say("oracle over all 72 tensors (every block)")
    ref_w = [w8.weights(k, n_threads=n_threads) for k in range(len(w8.numels))]
    ref_g = [_grad_bits(g) for g in h["g"]]
    ref_mq = [np.zeros(n, np.int8) for n in w8.numels]
    ref_vq = [np.zeros(n, np.uint8) for n in w8.numels]
    ref_ma = [np.zeros(-(-n // B), np.float32) for n in w8.numels]
    ref_va = [np.zeros(-(-n // B), np.float32) for n in w8.numels]
    omap = oracle.MAP_DYNAMIC if code_map == lt.LT_MAP_DYNAMIC else oracle.MAP_LINEAR
    oracle.hybrid8bit_adamw_step(ref_w, ref_g, ref_mq, ref_ma, ref_vq, ref_va, B, step=1,
                                 coef=float(c_o), status=st_o, n_threads=n_threads,
                                 code_map=omap, **_hyper(w8))
    blocks = 0
    for k in range(len(w8.numels)):
        for name, got, want in (("w", h["w"][k], ref_w[k]), ("m codes", h["mq"][k], ref_mq[k]),
                                ("m absmax", h["ma"][k], ref_ma[k]),
                                ("v codes", h["vq"][k], ref_vq[k]),
                                ("v absmax", h["va"][k], ref_va[k])):
            assert got.numpy().tobytes() == want.tobytes(), f"tensor {k}: {name} differs"
        blocks += ref_ma[k].size
    assert blocks == sum(-(-n // B) for n in w8.numels)
    _say(f"all {blocks} blocks of the 8 layers bitwise equal (keep_grads {keep}, "
         f"code map {code_map})")
