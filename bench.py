"""Benchmark of the Hybrid 8-bit optimizer step on one MI355X.

One "step" is the whole hot path over the resident synthetic workload:
lt_grad_sqnorm (a1-a2) -> lt_clip_coef (a3) -> lt_hybrid8bit_adamw_step (a4-a10),
enqueued on one stream.  The default workload is the 3B-class full model
(tied 151936x2048 embedding + 36 decoder layers: 325 tensors, 3,085,844,480
fp32 master parameters, bf16 gradients, 8-bit block-wise states, block 2048),
resident in HBM before timing starts.

Prints ONE JSON line (rank 0): params/s over the timed steps, the achieved HBM
bandwidth of the whole step and a roofline entry for the dominant kernel (the
fused step kernel) from HIP events around its launches, and the CPU oracle
timed on a bounded sample of the same workload on this host's cores.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E peak
METRIC = "optimizer step params/s + achieved HBM GB/s (% of MI355X peak)"
WORKLOADS = {"full": "full_3b", "layer": "layer_3b", "tiny": "tiny", "stress": "clip_stress",
             "streamed": "streamed_27b"}


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def grad_bytes(gdt) -> int:
    import synth
    return 2 if gdt == synth.BF16 else 4


def step_kernel_bytes(numels, block, gbytes) -> int:
    """Algorithmic HBM bytes of one fused-step launch: per parameter the gradient
    (read), the fp32 weight (read + write) and the two 8-bit codes (read + write);
    per block the two fp32 scales (read + write)."""
    n = sum(numels)
    nb = sum(-(-x // block) for x in numels)
    return n * (gbytes + 8 + 2 + 2) + nb * 16


def norm_bytes(numels, gbytes) -> int:
    """Algorithmic bytes of the sum-of-squares pass: one gradient read."""
    return sum(numels) * gbytes


def build_device_workload(w, dev, n_threads, code_map=0):
    """Generates the workload on the host (pinned staging, one tensor at a time),
    copies it to HBM and builds the 8-bit states with one step from zero state at
    t = 1 on an unclipped prior gradient with lr = 0 (weights stay as drawn)."""
    import torch

    import paper_2608_11919_amd as lt
    import synth

    K, B = len(w.shapes), w.block_size
    gdt_torch = torch.bfloat16 if w.grad_dtype == synth.BF16 else torch.float32
    biggest = max(w.numels)
    stage_w = torch.empty(biggest, dtype=torch.float32, pin_memory=True)
    stage_g = torch.empty(biggest, dtype=gdt_torch, pin_memory=True)
    params, grads = [], []
    mq, vq, ma, va = [], [], [], []
    t0 = time.time()
    for k, n in enumerate(w.numels):
        synth.fill_ptr(stage_w.data_ptr(), synth.F32, 0, n, w.seed, synth.STREAM_WEIGHTS, k,
                       w.weight_recipe, n_threads)
        params.append(stage_w[:n].to(dev, non_blocking=False))
        synth.fill_ptr(stage_g.data_ptr(), w.grad_dtype, 0, n, w.seed, synth.STREAM_PRIOR_GRAD, k,
                       w.grad_recipe, n_threads)
        grads.append(stage_g[:n].to(dev, non_blocking=False))
        mq.append(torch.zeros(n, dtype=torch.int8, device=dev))
        vq.append(torch.zeros(n, dtype=torch.uint8, device=dev))
        ma.append(torch.zeros(-(-n // B), dtype=torch.float32, device=dev))
        va.append(torch.zeros(-(-n // B), dtype=torch.float32, device=dev))
        if k % 50 == 0:
            log(f"generated {k + 1}/{K} tensors ({time.time() - t0:.1f} s)")
    hyper = dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay)
    if w.state_init == "prior_step":
        lt.lt_hybrid8bit_adamw_step(params, grads, mq, ma, vq, va, B, step=1,
                                    code_map=code_map, **dict(hyper, lr=0.0))
        torch.cuda.synchronize()
    # the gradient of the measured steps replaces the prior gradient in place
    first = w.step if w.state_init == "prior_step" else 1
    for k, n in enumerate(w.numels):
        synth.fill_ptr(stage_g.data_ptr(), w.grad_dtype, 0, n, w.seed, synth.grad_stream(first),
                       k, w.grad_recipe, n_threads)
        grads[k].copy_(stage_g[:n])
    torch.cuda.synchronize()
    log(f"workload resident in HBM ({time.time() - t0:.1f} s)")
    return params, grads, mq, ma, vq, va, first


def _oracle_pass(w, ks, n_threads, code_map=0):
    """Generates whole tensors ks of the workload on the host, then times one oracle
    pass over them: sum of squares + clip + step."""
    import numpy as np

    import oracle
    import synth

    B = w.block_size
    ws = [w.weights(k, n_threads=n_threads) for k in ks]
    gs = [w.grads(k, synth.grad_stream(w.step), n_threads=n_threads) for k in ks]
    mq = [np.zeros(x.size, np.int8) for x in ws]
    vq = [np.zeros(x.size, np.uint8) for x in ws]
    ma = [np.zeros(-(-x.size // B), np.float32) for x in ws]
    va = [np.zeros(-(-x.size // B), np.float32) for x in ws]
    hyper = dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay)
    t0 = time.perf_counter()
    _, S, st = oracle.grad_sqnorm(gs, n_threads=n_threads)
    _, c = oracle.clip_coef(S, w.max_norm)
    oracle.hybrid8bit_adamw_step(ws, gs, mq, ma, vq, va, B, step=w.step, coef=float(c), status=st,
                                 n_threads=n_threads, code_map=code_map, **hyper)
    return time.perf_counter() - t0


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, n_threads, target_s: float, code_map=0, max_tensors=None):
    """The oracle as it stands, on a bounded sample of the same workload (whole
    tensors, decoder layers first, the embedding last), timed on this host's cores.
    One decoder layer is timed first to size a sample of about target_s seconds (at
    most max_tensors tensors); the same layer is also timed on one thread."""
    K = len(w.shapes)
    order = list(range(K))
    if len(w.shapes[0]) == 2 and w.shapes[0][0] > 100000:
        order = order[1:] + order[:1]
    first = order[:min(K, 9)]
    n_first = sum(w.numels[k] for k in first)
    dt = _oracle_pass(w, first, n_threads, code_map)
    rate = n_first / dt
    dt1 = _oracle_pass(w, first, 1, code_map)
    ks, total = [], 0
    for k in order:
        if ks and (total + w.numels[k] > rate * target_s or
                   (max_tensors is not None and len(ks) >= max_tensors)):
            break
        ks.append(k)
        total += w.numels[k]
    if ks != first:
        dt = _oracle_pass(w, ks, n_threads, code_map)
    desc = f"{len(ks)} of {K} tensors ({total} of {w.n_params} params) of {w.name}"
    return {"value": total / dt, "unit": "params/s", "cores": n_threads, "kind": "oracle",
            "sample": desc + ": sum of squares + clip + step, one pass", "seconds": round(dt, 3),
            "single_thread": {"value": n_first / dt1, "unit": "params/s",
                              "sample": f"{len(first)} tensors ({n_first} params), one thread",
                              "seconds": round(dt1, 3)},
            "cpu_model": cpu_model(),
            "affinity_cpus": len(os.sched_getaffinity(0))}


def source_digest(path: str) -> str:
    """SHA-256 of a C/HIP source with comments and blank lines dropped and runs of
    whitespace folded, so that edits to comments keep recorded counters valid."""
    import hashlib
    import re
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    lines = [" ".join(line.split()) for line in text.splitlines()]
    return hashlib.sha256("\n".join(x for x in lines if x).encode()).hexdigest()


def counter_traffic(workload_name: str):
    """HBM bytes per launch of the fused step kernel from the committed rocprofv3
    counter summaries (profiles/*_counters.json: FETCH_SIZE and WRITE_SIZE, each
    scaled by a plain copy of known size).  None unless a summary covers this
    workload and the kernel source is the one its counters were taken on."""
    import glob
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*_counters.json"))):
        try:
            with open(path) as f:
                c = json.load(f)
            if c.get("workload") != workload_name:
                continue
            sha = source_digest(os.path.join(ROOT, c["source"]))
        except (OSError, KeyError, ValueError):
            continue
        if sha == c.get("source_digest"):
            return c["kernels"]["k_adamw8_step"]["traffic_bytes"]
    return None


_pinned_keep = []


def pinned(n: int, dtype, zero: bool = False):
    """A CPU tensor of n elements in pinned memory of exactly its size (hipHostMalloc;
    torch's pinned allocator rounds each allocation up to a power of two, which at the
    27B-class model's 169 GB would cost up to twice the memory).  Kept until exit."""
    import ctypes

    import numpy as np
    import torch
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipHostMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t,
                                  ctypes.c_uint]
    hip.hipHostMalloc.restype = ctypes.c_int
    item = torch.empty(0, dtype=dtype).element_size()
    nbytes = max(n * item, 1)
    ptr = ctypes.c_void_p()
    rc = hip.hipHostMalloc(ctypes.byref(ptr), nbytes, 0)
    if rc != 0:
        hip.hipGetLastError()  # the failure would otherwise surface at the next HIP call
        raise RuntimeError(f"hipHostMalloc of {nbytes} bytes failed ({rc})")
    buf = (ctypes.c_uint8 * nbytes).from_address(ptr.value)
    t = torch.from_numpy(np.frombuffer(buf, dtype=np.uint8, count=n * item)).view(dtype)
    _pinned_keep.append(buf)
    if zero:
        t.zero_()
    return t


def pcie_rates(dev, nbytes: int):
    """Pinned host <-> HBM copy rates on this machine: H2D alone, D2H alone and both at
    once on two streams (GB/s each), with hipMemcpyAsync as the streamed step issues
    them."""
    import ctypes

    import torch
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.c_int, ctypes.c_void_p]
    hip.hipMemcpyAsync.restype = ctypes.c_int
    h2d_kind, d2h_kind = 1, 2  # hipMemcpyHostToDevice, hipMemcpyDeviceToHost
    h_in = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    h_out = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    d_a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    d_b = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    s1, s2 = torch.cuda.Stream(dev), torch.cuda.Stream(dev)

    def copy(dst, src, kind, stream):
        rc = hip.hipMemcpyAsync(dst.data_ptr(), src.data_ptr(), nbytes, kind, stream.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"hipMemcpyAsync failed ({rc})")

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fn()
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    def h2d():
        copy(d_a, h_in, h2d_kind, s1)

    def d2h():
        copy(h_out, d_b, d2h_kind, s2)

    def both():
        h2d()
        d2h()

    t_h2d, t_d2h, t_both = timed(h2d), timed(d2h), timed(both)
    return {"h2d_gbps": round(nbytes / t_h2d / 1e9, 2), "d2h_gbps": round(nbytes / t_d2h / 1e9, 2),
            "concurrent_gbps_each": round(nbytes / t_both / 1e9, 2), "probe_bytes": nbytes}


def run_streamed(args, w, dev, n_threads) -> int:
    """a11: the layer-streamed step.  Weights, gradients and 8-bit states live in pinned
    host memory; each step streams the gradients through HBM for the norm (pass 1),
    then every layer in, through the fused step and out (pass 2).  Host memory holds
    args.host_layers distinct layers that the model's layers cycle through (logical
    layer l uses host layer l mod host_layers), which bounds pinned memory while
    moving exactly the bytes of the full model."""
    import torch

    import paper_2608_11919_amd as lt
    import synth

    per_layer = 9
    L = len(w.shapes) // per_layer
    R = min(args.host_layers, L)
    B = w.block_size
    hyper = dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay)
    log(f"{w.name}: {L} layers, {w.n_params} params; {R} distinct pinned host layers")
    rates = pcie_rates(dev, 1 << 31)
    log(f"pinned copies: {rates}")
    t0 = time.time()
    host = {name: [] for name in ("w", "g", "mq", "ma", "vq", "va")}
    for r in range(R):
        for j in range(per_layer):
            k = r * per_layer + j
            n = w.numels[k]
            nb = -(-n // B)
            wt = pinned(n, torch.float32)
            synth.fill_ptr(wt.data_ptr(), synth.F32, 0, n, w.seed, synth.STREAM_WEIGHTS, k,
                           w.weight_recipe, n_threads)
            gt = pinned(n, torch.bfloat16)
            synth.fill_ptr(gt.data_ptr(), synth.BF16, 0, n, w.seed, synth.grad_stream(w.step), k,
                           w.grad_recipe, n_threads)
            host["w"].append(wt)
            host["g"].append(gt)
            host["mq"].append(pinned(n, torch.int8, zero=True))
            host["vq"].append(pinned(n, torch.uint8, zero=True))
            host["ma"].append(pinned(nb, torch.float32, zero=True))
            host["va"].append(pinned(nb, torch.float32, zero=True))
            if args.bf16_copy:
                host.setdefault("wb", []).append(pinned(n, torch.bfloat16))
        log(f"host layer {r + 1}/{R} ready ({time.time() - t0:.1f} s)")
    lists = {name: [v[(l % R) * per_layer + j] for l in range(L) for j in range(per_layer)]
             for name, v in host.items()}
    first = list(range(0, L * per_layer + 1, per_layer))
    S = torch.zeros(1, dtype=torch.float64, device=dev)
    coef = torch.zeros(1, dtype=torch.float32, device=dev)
    norm = torch.zeros(1, dtype=torch.float32, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    cs, hs, ds = torch.cuda.Stream(dev), torch.cuda.Stream(dev), torch.cuda.Stream(dev)
    slots = args.ring_slots
    nbytes = lt.lt_streamed_workspace_bytes(w.numels, first, lt.LT_DTYPE_BF16, B, slots,
                                            args.bf16_copy, args.keep_grads)
    workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    acc = dev_grads = None
    if args.norm_on_arrival:
        # device copies of the distinct host layers' gradients: the gradients as
        # backward leaves them in HBM before they are offloaded
        dev_grads = [g.to(dev) for g in host["g"]]
        acc = lt.GradNormAccumulator(w.numels, dev)
    torch.cuda.synchronize()

    lev = [torch.cuda.Event(enable_timing=True) for _ in range(8 * L)]

    def step(t, events=None):
        if acc is not None:
            with torch.cuda.stream(cs):
                for l in reversed(range(L)):  # backward order
                    r = (l % R) * per_layer
                    acc.add(l * per_layer, dev_grads[r:r + per_layer], stream=cs)
                acc.finish(S, status, stream=cs)
        lt.lt_streamed_hybrid8bit_adamw_step(
            lists["w"], lists["g"], lists["mq"], lists["ma"], lists["vq"], lists["va"], first, B,
            step=t, max_norm=w.max_norm, ring_slots=slots, sq_total=S, coef=coef, status=status,
            total_norm=norm, workspace=workspace, compute_stream=cs, h2d_stream=hs,
            d2h_stream=ds, params_bf16=lists.get("wb"), norm_ready=acc is not None,
            keep_grads=args.keep_grads,
            code_map=lt.LT_MAP_DYNAMIC if args.code_map == "dynamic" else lt.LT_MAP_LINEAR,
            layer_events=events, **hyper)

    t = 1
    for _ in range(args.warmup):
        step(t)
        t += 1
        cs.synchronize()
        log(f"warmup step done")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(t, lev if i == args.steps - 1 else None)  # the last step records its phases
        t += 1
        cs.synchronize()
        log(f"timed step done ({time.perf_counter() - t0:.2f} s)")
    elapsed = time.perf_counter() - t0
    st = lt.lt_read_status(status, cs)
    phases = streamed_phases(lev, L, w, B, args)
    per = elapsed / args.steps
    n = w.n_params
    nb = sum(-(-x // B) for x in w.numels)
    # pass 1 gradients (not with the norm summed on arrival); pass 2 weights, gradients
    # (not when pass 1 left them in HBM), codes, scales
    once = args.keep_grads and not args.norm_on_arrival
    h2d = (0 if args.norm_on_arrival else n * 2) + n * (6 if once else 8) + nb * 8
    d2h = n * (8 if args.bf16_copy else 6) + nb * 8  # weights, codes, scales (bf16 copy) back
    bound = max(h2d / (rates["h2d_gbps"] * 1e9), d2h / (rates["d2h_gbps"] * 1e9))
    out = {
        "metric": METRIC, "value": n / per, "unit": "params/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(per * 1e3, 2),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name + ("+bf16-copy" if args.bf16_copy else "") +
                   ("+norm-on-arrival" if args.norm_on_arrival else "") +
                   ("+grads-kept-in-hbm" if args.keep_grads else "") +
                   ("+dynamic-map" if args.code_map == "dynamic" else ""), "params": n,
                   "tensors": len(w.shapes), "layers": L,
                   "block_size": B, "grad_dtype": "bf16", "ring_slots": slots,
                   "host_layers": R,
                   "host_state": "pinned, every layer distinct" if R == L else
                                 "pinned, cycled over host_layers"},
        "phases_last_step": phases,
        "pcie": {"h2d_bytes_per_step": h2d, "d2h_bytes_per_step": d2h, **rates,
                 "link_bound_ms": round(bound * 1e3, 1),
                 "h2d_gbps_achieved": round(h2d / per / 1e9, 2),
                 "d2h_gbps_achieved": round(d2h / per / 1e9, 2),
                 "frac_of_link_bound": round(bound / per, 4)},
        "status": st, "norm": float(norm.item()), "coef": float(coef.item()),
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample of 4 layers")
        cb = cpu_baseline(w, n_threads, args.cpu_seconds,
                          code_map=lt.LT_MAP_DYNAMIC if args.code_map == "dynamic"
                          else lt.LT_MAP_LINEAR, max_tensors=4 * per_layer)
        cb["extrapolated_step_s"] = round(n / cb["value"], 2)
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)
    return 0


def streamed_phases(ev, L: int, w, B: int, args):
    """Per-phase times of one streamed step from the events the call recorded around
    each layer's work: the summed durations of the pass-1 gradient copies, the pass-2
    copies in, the step kernels and the copies out, their bytes and rates, and the
    span from the first copy in to the last copy out."""
    def total(a, b):
        return sum(ev[8 * i + a].elapsed_time(ev[8 * i + b]) for i in range(L))
    per_layer = len(w.numels) // L
    n = w.n_params
    nb = sum(-(-x // B) for x in w.numels)
    once = args.keep_grads and not args.norm_on_arrival
    out = {}
    p1_bytes = 0 if args.norm_on_arrival else 2 * n
    if p1_bytes:
        ms = total(0, 1)
        out["pass1_h2d"] = {"ms": round(ms, 1), "bytes": p1_bytes,
                            "gbps": round(p1_bytes / ms / 1e6, 1)}
    in_bytes = n * (6 if once else 8) + nb * 8
    out_bytes = n * (8 if args.bf16_copy else 6) + nb * 8
    for name, a, b, nbytes in (("pass2_h2d", 2, 3, in_bytes), ("d2h", 4, 5, out_bytes),
                               ("step_kernels", 6, 7, None)):
        ms = total(a, b)
        out[name] = {"ms": round(ms, 1)}
        if nbytes:
            out[name].update(bytes=nbytes, gbps=round(nbytes / ms / 1e6, 1))
    first = 0 if p1_bytes else 2
    out["span_ms"] = round(ev[first].elapsed_time(ev[8 * (L - 1) + 5]), 1)
    out["note"] = ("each phase's summed per-layer durations; the copies in and out of "
                   "different layers run at the same time, sharing the link")
    return out


def stream_ceiling(n_elements: int, pattern: str = "step8"):
    """Runs the data-movement probe (paper_2608_11919_amd/stream_ceiling, built with
    the library) in a child process, with no arithmetic, at this workload's size: the
    norm's 2 B read per element, and the step's byte pattern per element (step8: 8 B
    read + 6 B written in place; step8_copy: the same + 2 B written to the bf16 copy;
    adamw32: 14 B read + 12 B written, the fp32-state step)."""
    import subprocess
    exe = os.path.join(ROOT, "paper_2608_11919_amd", "stream_ceiling")
    if not os.path.exists(exe):
        log("stream_ceiling is not built; no ceiling reported")
        return None
    r = subprocess.run([exe, str(n_elements), "5", pattern], capture_output=True, text=True,
                       timeout=300)
    if r.returncode != 0:
        log(f"stream_ceiling failed ({r.returncode}): {r.stderr.strip()[-200:]}")
        return None
    return json.loads(r.stdout.strip().splitlines()[-1])


def same_array_probe(params, grads, m_states, v_states, gbytes, state_bytes, dev, stream,
                     reps=3):
    """Times paper_2608_11919_amd/libltprobe.so (csrc/mix_probe.hip) over a step's
    own arrays, in this process: the fused step's per-element bytes (the weight, the
    gradient and both moment states read; the weight and both states written back in
    place; state_bytes 1 for the 8-bit codes, 4 for fp32 moments) in the step kernel's
    geometry and unit order, with no arithmetic.  An even number of passes XORs every
    array back to its contents.  Returns (median ms, bytes)."""
    import ctypes

    import torch
    path = os.path.join(ROOT, "paper_2608_11919_amd", "libltprobe.so")
    if not os.path.exists(path):
        log("libltprobe.so is not built; no same-array probe")
        return None
    L = ctypes.CDLL(path)
    L.ltp_mix_same_arrays.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                      ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_void_p]
    L.ltp_mix_same_arrays.restype = ctypes.c_int
    K = len(params)
    units = [-(-p.numel() // 2048) for p in params]
    prefix = [0]
    for u in units:
        prefix.append(prefix[-1] + u)
    d_prefix = torch.tensor(prefix, dtype=torch.int64, device=dev)
    table = torch.zeros((K, 8), dtype=torch.int64)
    for k in range(K):
        table[k, :5] = torch.tensor([params[k].data_ptr(), grads[k].data_ptr(),
                                     m_states[k].data_ptr(), v_states[k].data_ptr(),
                                     params[k].numel()], dtype=torch.int64)
    d_table = table.to(dev)
    grid = 3 * torch.cuda.get_device_properties(dev).multi_processor_count
    ms = []
    for _ in range(2 * reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        rc = L.ltp_mix_same_arrays(d_prefix.data_ptr(), d_table.data_ptr(), K, prefix[-1], gbytes,
                                   state_bytes, grid, stream.cuda_stream)
        b.record(stream)
        if rc != 0:
            raise RuntimeError(f"ltp_mix_same_arrays failed ({rc})")
        torch.cuda.synchronize()
        ms.append(a.elapsed_time(b))
    n = sum(p.numel() for p in params)
    # per element: the weight read and written, the gradient read, each state read and written
    return sorted(ms)[len(ms) // 2], n * (8 + gbytes + 4 * state_bytes)


def warm_kernels(dev, gdt, B: int, code_map: int, stream, fp32_states: bool):
    """Runs each kernel the timed steps use once, on a scratch list of one block, so that
    the first timed step does not pay for loading their code (the clip-stress workload
    times its first three steps from zero state, with no warmup steps).  The workload's
    own tensors are not touched."""
    import torch

    import paper_2608_11919_amd as lt
    n = B
    w = torch.zeros(n, dtype=torch.float32, device=dev)
    g = torch.zeros(n, dtype=gdt, device=dev)
    S = torch.zeros(1, dtype=torch.float64, device=dev)
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    coef = torch.zeros(1, dtype=torch.float32, device=dev)
    h = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, step=1, coef=coef,
             status=st, stream=stream)
    lt.lt_grad_sqnorm([g], S, st, stream=stream)
    lt.lt_clip_coef(S, 1.0, coef, stream=stream)
    lt.lt_hybrid8bit_adamw_step([w], [g], [torch.zeros(n, dtype=torch.int8, device=dev)],
                                [torch.zeros(1, device=dev)],
                                [torch.zeros(n, dtype=torch.uint8, device=dev)],
                                [torch.zeros(1, device=dev)], B, code_map=code_map, **h)
    if fp32_states:
        lt.lt_adamw_fp32_step([w], [g], [torch.zeros_like(w)], [torch.zeros_like(w)], **h)
    torch.cuda.synchronize()


def copy_probe(dev, nbytes: int, reps: int):
    """A plain copy kernel of known size, for scaling the HBM byte counters."""
    import torch
    x = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    for _ in range(reps):
        torch.mul(x, 1.0, out=y)
    torch.cuda.synchronize()
    log(f"copy probe: {reps} x torch.mul(out=) over {nbytes} bytes read + {nbytes} written")


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="full")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU seconds for the oracle sample")
    ap.add_argument("--slice-fraction", type=float, default=None,
                    help="hybrid operator: only this fraction of parameters keeps 8-bit states, "
                         "the rest fp32 states (the paper's run uses 0.02)")
    ap.add_argument("--block-size", type=int, default=0,
                    help="override the workload's quantization block size (the paper uses 4096)")
    ap.add_argument("--code-map", choices=["linear", "dynamic"], default="linear",
                    help="code map of the 8-bit moments")
    ap.add_argument("--bf16-copy", action="store_true",
                    help="the steps also write a bf16 copy of the updated weights (+2 B/param)")
    ap.add_argument("--keep-grads", action="store_true",
                    help="streamed workload: the gradients stay in HBM from the first pass to "
                         "the second and cross the link once")
    ap.add_argument("--norm-on-arrival", action="store_true",
                    help="streamed workload: the norm is summed layer by layer from gradients "
                         "already in HBM (as they arrive in backward) and the step skips its "
                         "first streamed pass")
    ap.add_argument("--host-layers", type=int, default=8,
                    help="streamed workload: distinct pinned host layers the model cycles over "
                         "(these boxes pin about 63 GB, 24 layers, of the 169 GB all 64 need)")
    ap.add_argument("--ring-slots", type=int, default=3, help="streamed workload: device slots")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the data-movement ceiling probe")
    ap.add_argument("--copy-probe-bytes", type=int, default=0,
                    help="also run a plain copy of this many bytes (counter scaling)")
    ap.add_argument("--flush-bytes", type=int, default=0,
                    help="write a scratch buffer of this many bytes between steps, outside the "
                         "timed events, so no step finds the previous one's data in the 256 MB "
                         "Infinity Cache (for workloads that fit in it); the step time is then "
                         "the mean of the per-step events")
    ap.add_argument("--graph", action="store_true",
                    help="capture one whole step (norm, clip, step at a fixed step index) in a "
                         "HIP graph after the warmup and time replays of it (launch-bound "
                         "small workloads)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the step has no multi-GPU path (it would "
              "shard by chunk-aligned block ranges, with one all-gather of the fp64 chunk "
              "partials for the norm)", file=sys.stderr)
        return 2

    import torch

    import paper_2608_11919_amd as lt
    import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda", 0)
    lt.lib()  # fails loudly when the HIP library is not built
    n_threads = synth.default_threads()
    w = getattr(synth, WORKLOADS[args.workload])()
    if args.block_size:
        import dataclasses
        w = dataclasses.replace(w, block_size=args.block_size)
    K, B = len(w.shapes), w.block_size
    log(f"workload {w.name}: {K} tensors, {w.n_params} params, block {B}")

    if args.copy_probe_bytes:
        copy_probe(dev, args.copy_probe_bytes, 5)
    if args.workload == "streamed":
        return run_streamed(args, w, dev, n_threads)

    code_map = lt.LT_MAP_DYNAMIC if args.code_map == "dynamic" else lt.LT_MAP_LINEAR
    params, grads, mq, ma, vq, va, t_first = build_device_workload(w, dev, n_threads, code_map)
    idx8, idx32 = list(range(K)), []
    if args.slice_fraction is not None:
        mask, _ = lt.lt_select_8bit_slice(w.numels, args.slice_fraction)
        idx8 = [k for k in range(K) if mask[k]]
        idx32 = [k for k in range(K) if not mask[k]]
        for k in idx32:  # the fp32-state tensors need no 8-bit states
            mq[k] = vq[k] = ma[k] = va[k] = None
        torch.cuda.empty_cache()
        exp_avg = [torch.zeros_like(params[k]) for k in idx32]
        exp_avg_sq = [torch.zeros_like(params[k]) for k in idx32]
        log(f"hybrid: {len(idx8)} tensors ({sum(w.numels[k] for k in idx8)} params) with 8-bit "
            f"states, {len(idx32)} with fp32 states")
    sq_total = torch.zeros(1, dtype=torch.float64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    coef = torch.zeros(1, dtype=torch.float32, device=dev)
    norm = torch.zeros(1, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    hyper = dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay)
    ws_sq = torch.empty(lt.lt_grad_sqnorm_workspace_bytes(w.numels), dtype=torch.uint8, device=dev)
    ws_step = torch.empty(lt.lt_step_workspace_bytes(K), dtype=torch.uint8, device=dev)
    ws_32 = torch.empty(max(1, lt.lt_adamw_fp32_workspace_bytes(len(idx32))), dtype=torch.uint8,
                        device=dev)
    p8, g8 = [params[k] for k in idx8], [grads[k] for k in idx8]
    s8 = [[x[k] for k in idx8] for x in (mq, ma, vq, va)]
    p32, g32 = [params[k] for k in idx32], [grads[k] for k in idx32]
    wb8 = wb32 = None
    if args.bf16_copy:
        wb = [torch.empty(n, dtype=torch.bfloat16, device=dev) for n in w.numels]
        wb8, wb32 = [wb[k] for k in idx8], [wb[k] for k in idx32]

    def one_step(t, ev=None, st=None):
        st = stream if st is None else st
        if ev:
            ev[0].record(st)
        lt.lt_grad_sqnorm(grads, sq_total, status, workspace=ws_sq, stream=st)
        lt.lt_clip_coef(sq_total, w.max_norm, coef, total_norm=norm, stream=st)
        if ev:
            ev[1].record(st)
        if p8:
            lt.lt_hybrid8bit_adamw_step(p8, g8, *s8, B, step=t, coef=coef, status=status,
                                        workspace=ws_step, stream=st, params_bf16=wb8,
                                        code_map=code_map, **hyper)
        if p32:
            lt.lt_adamw_fp32_step(p32, g32, exp_avg, exp_avg_sq, step=t, coef=coef,
                                  status=status, workspace=ws_32, stream=st,
                                  params_bf16=wb32, **hyper)
        if ev:
            ev[2].record(st)

    scratch = None
    if args.flush_bytes:
        scratch = torch.empty(args.flush_bytes // 4, dtype=torch.float32, device=dev)

    def flush():
        if scratch is not None:
            scratch.fill_(float(t))  # a kernel that writes every byte (no memset node)

    warm_kernels(dev, grads[0].dtype, B, code_map, stream, bool(idx32))
    t = t_first
    for _ in range(args.warmup):
        flush()
        one_step(t)
        t += 1
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        flush()
        one_step(t, events[i])
        t += 1
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    st = lt.lt_read_status(status)
    graph = None
    if args.graph:
        # The calls above left every descriptor in its workspace, so the step captures
        # whole; each replay is one full step at step index t.  The eager steps above
        # give the per-kernel events; the replays give the step time.
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream(dev)
        side.wait_stream(stream)
        with torch.cuda.graph(graph, stream=side):
            one_step(t, st=side)
        torch.cuda.synchronize()
        log(f"one step captured in a HIP graph (step index {t})")
        gev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        graph.replay()  # a first replay outside the timed region
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            flush()
            gev[i][0].record(stream)
            graph.replay()
            gev[i][1].record(stream)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        st = lt.lt_read_status(status)

    norm_ms = [e[0].elapsed_time(e[1]) for e in events]
    step_ms = [e[1].elapsed_time(e[2]) for e in events]
    whole_ms = [e[0].elapsed_time(e[2]) for e in events]
    if graph is not None:
        whole_ms = [e[0].elapsed_time(e[1]) for e in gev]
    if scratch is not None:
        # the flushes between steps are not step work: the step time is the mean of
        # the per-step events
        elapsed = sum(whole_ms) * 1e-3

    def pct(xs, q):  # nearest-rank percentile
        xs = sorted(xs)
        return round(xs[min(len(xs) - 1, max(0, math.ceil(q * len(xs)) - 1))], 4)

    def spread(xs):
        return {"p10": pct(xs, 0.1), "median": pct(xs, 0.5), "p90": pct(xs, 0.9)}

    avg_step_s = sum(step_ms) / len(step_ms) * 1e-3
    avg_norm_s = sum(norm_ms) / len(norm_ms) * 1e-3
    gb = grad_bytes(w.grad_dtype)
    kbytes = step_kernel_bytes([w.numels[k] for k in idx8], B, gb) + \
        sum(w.numels[k] for k in idx32) * (gb + 24)  # fp32 states: w, m, v read and written
    if args.bf16_copy:
        kbytes += 2 * w.n_params  # the bf16 weight copy written
    nbytes = norm_bytes(w.numels, gb)
    ms_per_step = elapsed / args.steps * 1e3
    step_total_bytes = kbytes + nbytes
    achieved = kbytes / avg_step_s / 1e9
    log(f"status {st}, norm {norm.item():.6g}, coef {coef.item():.6g}; step kernel "
        f"{avg_step_s * 1e3:.3f} ms ({achieved:.0f} GB/s), norm pass {avg_norm_s * 1e3:.3f} ms "
        f"({nbytes / avg_norm_s / 1e9:.0f} GB/s)")

    out_workload = (w.name + (f"-block{B}" if args.block_size else "") +
                    ("+graph" if graph is not None else "") +
                    ("+cache-flushed" if scratch is not None else "") +
                    ("" if not idx32 else f"-hybrid-{args.slice_fraction:g}-8bit") +
                    ("+bf16-copy" if args.bf16_copy else "") +
                    ("+dynamic-map" if args.code_map == "dynamic" else ""))
    out = {
        "metric": METRIC,
        "value": w.n_params / (elapsed / args.steps),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "step_ms_events": spread(whole_ms),
        "timing": ("per-step events, a write of " + str(args.flush_bytes) + " bytes between "
                   "steps outside them" if scratch is not None else
                   "wall clock over the timed steps") +
                  ("; replays of one captured step" if graph is not None else ""),
        "config": {"workload": out_workload,
                   "params": w.n_params, "tensors": K, "block_size": B,
                   "params_8bit": sum(w.numels[k] for k in idx8),
                   "grad_dtype": "bf16" if w.grad_dtype == synth.BF16 else "f32",
                   "states": "int8 m / uint8 v, fp32 absmax per block, " + args.code_map +
                             " code map",
                   "master": "fp32", "norm_accumulation": "f64",
                   "hyper": {"lr": w.lr, "betas": [w.beta1, w.beta2], "eps": w.eps,
                             "weight_decay": w.weight_decay, "max_norm": w.max_norm}},
        "hbm_gbps": round(step_total_bytes / (elapsed / args.steps) / 1e9, 1),
        "hbm_frac": round(step_total_bytes / (elapsed / args.steps) / 1e9 / PEAK_HBM_GBPS, 4),
        "bytes_per_param": round(step_total_bytes / w.n_params, 4),
        "kernels_ms": {"norm_pass": round(avg_norm_s * 1e3, 4),
                       "adamw8_step": round(avg_step_s * 1e3, 4)},
        "kernels_ms_spread": {"norm_pass": spread(norm_ms), "adamw8_step": spread(step_ms)},
        "roofline": {"kernel": "k_adamw8_step" if not idx32 else "k_adamw8_step + k_adamw32_step",
                     "bound": "hbm", "achieved": round(achieved, 1),
                     "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": counter_traffic(out_workload) if not idx32 else None,
                     "bytes_per_launch": kbytes},
        "status": st,
    }
    if not args.no_ceiling and not args.bf16_copy:
        # each step kernel's byte pattern over its own arrays; the hybrid step's two
        # kernels run one after the other, so their probe times add
        runs = []
        if p8:
            runs.append(("k_adamw8_step", same_array_probe(p8, g8, s8[0], s8[2], gb, 1, dev,
                                                           stream)))
        if p32:
            runs.append(("k_adamw32_step", same_array_probe(p32, g32, exp_avg, exp_avg_sq, gb,
                                                            4, dev, stream)))
        if runs and all(r is not None for _, r in runs):
            p_ms = sum(r[0] for _, r in runs)
            p_bytes = sum(r[1] for _, r in runs)
            p_gbps = p_bytes / (p_ms * 1e-3) / 1e9
            # the step's rate counts its block scales (16 B per block), the probe's does not
            out["same_array_probe"] = {
                "probe": "csrc/mix_probe.hip over the step's own arrays in this process: "
                         "each step kernel's bytes per element, geometry and unit order, no "
                         "arithmetic (scales not moved)",
                "ms": round(p_ms, 4), "bytes": p_bytes, "gbps": round(p_gbps, 1),
                "frac_of_peak": round(p_gbps / PEAK_HBM_GBPS, 4),
                "step_kernel_frac_of_probe": round(achieved / p_gbps, 4)}
            if len(runs) > 1:
                out["same_array_probe"]["kernels"] = {
                    k: {"ms": round(r[0], 4), "bytes": r[1],
                        "gbps": round(r[1] / (r[0] * 1e-3) / 1e9, 1)} for k, r in runs}
            log(f"same-array probe: {p_ms:.3f} ms, {p_gbps:.0f} GB/s; the step runs at "
                f"{achieved / p_gbps:.3f} of it")
    if not args.no_ceiling and gb == 2:
        # the probe pattern of each step kernel, at the whole model's size; the hybrid
        # step's two kernels are priced at their own patterns' rates
        n8 = sum(w.numels[k] for k in idx8)
        b8 = step_kernel_bytes([w.numels[k] for k in idx8], B, gb) + (2 * n8 if args.bf16_copy else 0)
        parts = []  # (pattern, algorithmic bytes of that kernel's launch)
        if idx8:
            parts.append(("step8_copy" if args.bf16_copy else "step8", b8))
        if idx32:
            # no probe pattern for the fp32-state step with the copy
            parts = parts + [("adamw32", kbytes - b8)] if not args.bf16_copy else []
        log(f"measuring the data-movement ceiling of the same byte patterns: "
            f"{[p for p, _ in parts]}")
        probes = [(p, nb, stream_ceiling(w.n_params, p)) for p, nb in parts]
        if probes and all(c is not None for _, _, c in probes):
            mix_ms = sum(c["mix_ms"] * nb / c["mix_bytes"] for _, nb, c in probes)
            read = min((c for _, _, c in probes), key=lambda c: c["read_ms"])
            mix_gbps = kbytes / (mix_ms * 1e-3) / 1e9
            out["ceiling"] = {
                "probe": "stream_ceiling: each step kernel's bytes per element (" +
                         " + ".join(f"{p} for {nb} B" for p, nb, _ in probes) +
                         ") and the norm's 2 B read per element, no arithmetic, same array "
                         "layout, at the whole model's size",
                "mix_gbps": round(mix_gbps, 1), "read_gbps": read["read_gbps"],
                "step_kernel_frac_of_mix": round(achieved / mix_gbps, 4),
                "norm_pass_frac_of_read": round(nbytes / avg_norm_s / 1e9 / read["read_gbps"], 4),
                "whole_step_ceiling_ms": round(mix_ms + read["read_ms"] * nbytes /
                                               read["read_bytes"], 4)}
            if len(probes) > 1:
                out["ceiling"]["patterns"] = {p: c["mix_gbps"] for p, _, c in probes}
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(w, n_threads, args.cpu_seconds, code_map)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
