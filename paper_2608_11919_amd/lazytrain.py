"""Python binding of liblazytrain.so (include/lazytrain.h), argument marshalling only.

Every function has the name of the C entry point it calls.  Tensors are
torch tensors on one HIP device; the binding checks devices, dtypes, sizes and
contiguity, passes ``data_ptr()``s and the stream handle, and raises on any
error code.  bf16 gradients may be torch.bfloat16 tensors (or raw bf16 bits in
int16/uint16 tensors).  All arithmetic runs in the HIP kernels; if the library
is not built this module raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
import math
import os
import weakref
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblazytrain.so")

LT_OK, LT_ERR_INVALID_ARG, LT_ERR_ALIGNMENT, LT_ERR_HIP, LT_ERR_WORKSPACE = range(5)
LT_STATUS_OK, LT_STATUS_NONFINITE, LT_STATUS_BAD_WORKSPACE = 0, 1, 2
LT_DTYPE_F32, LT_DTYPE_BF16 = 0, 1
LT_MAP_LINEAR, LT_MAP_DYNAMIC = 0, 1
ERROR_NAMES = {1: "LT_ERR_INVALID_ARG", 2: "LT_ERR_ALIGNMENT", 3: "LT_ERR_HIP",
               4: "LT_ERR_WORKSPACE"}

_lib = None


class LazyTrainError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


class NonFiniteAbort(RuntimeError):
    """Raised by Hybrid8bitAdamW once it has seen its limit of consecutive steps
    skipped for a non-finite gradient norm (App. C safety checks: non-finite steps
    are skipped, and training stops after three of them in a row)."""

    def __init__(self, skips: int):
        super().__init__(f"{skips} consecutive steps skipped for non-finite gradients")
        self.skips = skips


def lib() -> ctypes.CDLL:
    """Loads liblazytrain.so, raising if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(there is no fallback path)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64p = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64)
    vpp = ctypes.POINTER(ctypes.c_void_p)
    L.lt_grad_sqnorm_workspace_bytes.argtypes = [i64p, ctypes.c_int]
    L.lt_grad_sqnorm_workspace_bytes.restype = ctypes.c_size_t
    L.lt_grad_sqnorm.argtypes = [vpp, i64p, ctypes.c_int, ctypes.c_int, vp, ctypes.c_size_t,
                                 vp, vp, vp, vp]
    L.lt_grad_sqnorm_noalloc.argtypes = [vpp, i64p, ctypes.c_int, ctypes.c_int, vp, vp, vp, vp]
    L.lt_clip_coef.argtypes = [vp, ctypes.c_float, vp, vp, vp, vp]
    L.lt_grad_chunk_count.argtypes = [i64p, ctypes.c_int]
    L.lt_grad_chunk_count.restype = ctypes.c_int64
    L.lt_grad_sqnorm_partials_workspace_bytes.argtypes = [ctypes.c_int]
    L.lt_grad_sqnorm_partials_workspace_bytes.restype = ctypes.c_size_t
    L.lt_grad_sqnorm_partials.argtypes = [vpp, i64p, ctypes.c_int, ctypes.c_int, vp, vp,
                                          ctypes.c_size_t, vp]
    L.lt_grad_sqnorm_finish_workspace_bytes.argtypes = [ctypes.c_int]
    L.lt_grad_sqnorm_finish_workspace_bytes.restype = ctypes.c_size_t
    L.lt_grad_sqnorm_finish.argtypes = [i64p, ctypes.c_int, vp, vp, ctypes.c_size_t, vp, vp, vp,
                                        vp]
    L.lt_step_workspace_bytes.argtypes = [ctypes.c_int]
    L.lt_step_workspace_bytes.restype = ctypes.c_size_t
    L.lt_hybrid8bit_adamw_step.argtypes = [vpp, vpp, ctypes.c_int, vpp, vpp, vpp, vpp, vpp,
                                           i64p, ctypes.c_int, ctypes.c_int, ctypes.c_int] + [
                                               ctypes.c_double] * 5 + [
                                               ctypes.c_int64, vp, vp, vp, vp, ctypes.c_size_t, vp]
    ip = ctypes.POINTER(ctypes.c_int)
    L.lt_streamed_workspace_bytes.argtypes = [i64p, ctypes.c_int, ip, ctypes.c_int, ctypes.c_int,
                                              ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                              ctypes.c_int]
    L.lt_streamed_workspace_bytes.restype = ctypes.c_size_t
    L.lt_streamed_hybrid8bit_adamw_step.argtypes = [
        vpp, vpp, ctypes.c_int, vpp, vpp, vpp, vpp, vpp, i64p, ctypes.c_int, ip, ctypes.c_int,
        ctypes.c_int, ctypes.c_int] + [ctypes.c_double] * 5 + [ctypes.c_int64, ctypes.c_float, ctypes.c_int,
                                                 ctypes.c_int, ctypes.c_int, vp, ctypes.c_size_t,
                                                 vp, vp, vp, vp, vpp, vp, vp, vp]
    L.lt_adamw_fp32_workspace_bytes.argtypes = [ctypes.c_int]
    L.lt_adamw_fp32_workspace_bytes.restype = ctypes.c_size_t
    L.lt_adamw_fp32_step.argtypes = [vpp, vpp, ctypes.c_int, vpp, vpp, vpp, i64p, ctypes.c_int] + [
        ctypes.c_double] * 5 + [ctypes.c_int64, vp, vp, vp, vp, ctypes.c_size_t, vp]
    L.lt_step_state_bytes.argtypes = [ctypes.c_int64]
    L.lt_step_state_bytes.restype = ctypes.c_size_t
    L.lt_step_table.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_int64, ctypes.c_int64,
                                vp]
    L.lt_step_state_init.argtypes = [vp, ctypes.c_size_t, ctypes.c_int64, ctypes.c_double,
                                     ctypes.c_double, ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_int32, vp, vp]
    L.lt_step_state_advance.argtypes = [vp, vp, vp]
    L.lt_select_8bit_slice.argtypes = [i64p, ctypes.c_int, ctypes.c_double,
                                       ctypes.POINTER(ctypes.c_uint8),
                                       ctypes.POINTER(ctypes.c_int64)]
    L.lt_read_status.argtypes = [vp, vp, ctypes.POINTER(ctypes.c_int32)]
    L.lt_set_max_workgroups.argtypes = [ctypes.c_int]
    L.lt_workspace_release.argtypes = [vp]
    L.lt_last_error.argtypes = []
    L.lt_last_error.restype = ctypes.c_char_p
    for name in ("lt_grad_sqnorm", "lt_clip_coef", "lt_hybrid8bit_adamw_step", "lt_read_status",
                 "lt_grad_sqnorm_partials", "lt_grad_sqnorm_finish",
                 "lt_set_max_workgroups", "lt_streamed_hybrid8bit_adamw_step",
                 "lt_adamw_fp32_step", "lt_select_8bit_slice", "lt_workspace_release",
                 "lt_grad_sqnorm_noalloc", "lt_step_table", "lt_step_state_init",
                 "lt_step_state_advance"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(rc: int) -> None:
    if rc != LT_OK:
        raise LazyTrainError(rc, lib().lt_last_error().decode())


def _stream_handle(stream, device) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _ptr_array(tensors) -> ctypes.Array:
    return (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])


def _numel_array(tensors) -> ctypes.Array:
    return (ctypes.c_int64 * len(tensors))(*[t.numel() for t in tensors])


def _grad_dtype(grads) -> int:
    if not grads:
        return LT_DTYPE_F32  # an empty list reads nothing
    dt = grads[0].dtype
    if any(g.dtype != dt for g in grads):
        raise TypeError("all gradients must share one dtype")
    if dt == torch.float32:
        return LT_DTYPE_F32
    if dt in (torch.bfloat16, torch.int16, torch.uint16):
        return LT_DTYPE_BF16
    raise TypeError(f"gradient dtype must be float32 or bfloat16, got {dt}")


def _device_of(tensors, *others):
    """The device of a tensor list: its first tensor's, else that of the first
    given scalar tensor, else the current HIP device (an empty list)."""
    for t in list(tensors) + [o for o in others if o is not None]:
        return t.device
    return torch.device("cuda", torch.cuda.current_device())


def _check_tensors(tensors, device, dtype=None, what="tensor"):
    for i, t in enumerate(tensors):
        if t.device != device:
            raise ValueError(f"{what}[{i}] is on {t.device}, expected {device}")
        if not t.is_contiguous():
            raise ValueError(f"{what}[{i}] must be contiguous")
        if dtype is not None and t.dtype != dtype:
            raise TypeError(f"{what}[{i}] has dtype {t.dtype}, expected {dtype}")


def _bf16_list(copies, params, device):
    """The optional bf16 weight-copy list: None, or one tensor (or None) per parameter
    with the parameter's element count."""
    if copies is None:
        return None
    if len(copies) != len(params):
        raise ValueError("params_bf16 needs one entry (a tensor or None) per parameter")
    for i, (c, p) in enumerate(zip(copies, params)):
        if c is None:
            continue
        if c.device != device or not c.is_contiguous():
            raise ValueError(f"params_bf16[{i}] must be contiguous on {device}")
        if c.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
            raise TypeError(f"params_bf16[{i}] must be bfloat16, got {c.dtype}")
        if c.numel() != p.numel():
            raise ValueError(f"params_bf16[{i}] must have {p.numel()} elements")
    return (ctypes.c_void_p * len(copies))(*[0 if c is None else c.data_ptr() for c in copies])


def _scalar(t: Optional[torch.Tensor], device, dtype, what) -> int:
    if t is None:
        return 0
    if t.device != device or t.dtype != dtype or t.numel() < 1:
        raise ValueError(f"{what} must be a {dtype} tensor on {device}")
    return t.data_ptr()


_workspaces = {}
_finalizers = {}


def _forget(ptr: int, key: int) -> None:
    _finalizers.pop(key, None)
    try:
        lib().lt_workspace_release(ptr)
    except Exception:  # interpreter shutdown: nothing left to forget for
        pass


def _track(ws: torch.Tensor) -> None:
    """When the workspace tensor is freed, the library forgets what it wrote there
    (lt_workspace_release), so that a later workspace at the same address gets its
    descriptors copied in again.  Pass the same tensor to every call (a fresh view
    per call is released after each call and so copies the descriptors each time)."""
    key = id(ws)
    f = _finalizers.get(key)
    if f is not None and f.alive:
        return
    _finalizers[key] = weakref.finalize(ws, _forget, ws.data_ptr(), key)


def _workspace(device, nbytes: int, workspace: Optional[torch.Tensor], stream,
               kind: str) -> torch.Tensor:
    """The caller's workspace, or one cached per (device, stream, kind of call), so
    that a call repeated over the same tensors finds its descriptors in place (the
    library then copies nothing; see include/lazytrain.h).  A cached workspace is
    allocated on the stream that uses it, so that when a larger one replaces it the
    caching allocator hands its memory out again only in that stream's order; the
    library is told to forget the old one first."""
    if workspace is not None:
        if workspace.device != device or workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError(f"workspace must hold {nbytes} bytes on {device}")
        _track(workspace)
        return workspace
    key = (device, _stream_handle(stream, device), kind)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        if ws is not None:
            lt_workspace_release(ws)
        if stream is None:
            s = torch.cuda.current_stream(device)
        elif hasattr(stream, "cuda_stream"):
            s = stream
        else:
            s = torch.cuda.ExternalStream(int(stream), device=device)
        with torch.cuda.stream(s):
            ws = torch.empty(max(nbytes, 4096), dtype=torch.uint8, device=device)
        _workspaces[key] = ws
        _track(ws)
    return ws


# ------------------------------------------------------------------ entry points

def lt_grad_sqnorm_workspace_bytes(numels: Sequence[int]) -> int:
    arr = (ctypes.c_int64 * len(numels))(*numels)
    return int(lib().lt_grad_sqnorm_workspace_bytes(arr, len(numels)))


def lt_step_workspace_bytes(n_tensors: int) -> int:
    return int(lib().lt_step_workspace_bytes(n_tensors))


def lt_grad_sqnorm(grads: Sequence[torch.Tensor], sq_total: torch.Tensor, status: torch.Tensor,
                   sq_per_tensor: Optional[torch.Tensor] = None,
                   workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """Steps a1-a2: S_k, S and the non-finite status into device tensors (float64,
    float64[1], int32[1]).  An empty list, and empty tensors, sum to 0."""
    device = sq_total.device
    _check_tensors(grads, device, what="grads")
    gdt = _grad_dtype(grads)
    if sq_per_tensor is not None and sq_per_tensor.numel() < len(grads):
        raise ValueError("sq_per_tensor needs one float64 per tensor")
    nbytes = lt_grad_sqnorm_workspace_bytes([g.numel() for g in grads])
    ws = _workspace(device, nbytes, workspace, stream, "sqnorm")
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_grad_sqnorm(
            _ptr_array(grads), _numel_array(grads), len(grads), gdt, ws.data_ptr(),
            ws.numel() * ws.element_size(), _scalar(sq_per_tensor, device, torch.float64, "sq_per_tensor"),
            _scalar(sq_total, device, torch.float64, "sq_total"),
            _scalar(status, device, torch.int32, "status"), _stream_handle(stream, device)))


def lt_grad_sqnorm_noalloc(grads: Sequence[torch.Tensor], sq_total: torch.Tensor,
                           status: torch.Tensor, sq_per_tensor: Optional[torch.Tensor] = None,
                           stream=None) -> None:
    """lt_grad_sqnorm without a workspace: the library's own device scratch holds the
    descriptors and partial sums, and the call allocates nothing (see the header)."""
    device = sq_total.device
    _check_tensors(grads, device, what="grads")
    gdt = _grad_dtype(grads)
    if sq_per_tensor is not None and sq_per_tensor.numel() < len(grads):
        raise ValueError("sq_per_tensor needs one float64 per tensor")
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_grad_sqnorm_noalloc(
            _ptr_array(grads), _numel_array(grads), len(grads), gdt,
            _scalar(sq_per_tensor, device, torch.float64, "sq_per_tensor"),
            _scalar(sq_total, device, torch.float64, "sq_total"),
            _scalar(status, device, torch.int32, "status"), _stream_handle(stream, device)))


def lt_clip_coef(sq_total: torch.Tensor, max_norm: float, coef: torch.Tensor,
                 total_norm: Optional[torch.Tensor] = None,
                 status: Optional[torch.Tensor] = None, stream=None) -> None:
    """Step a3: norm and clip coefficient into device float32 tensors; status (an
    int32 device tensor, optional) is set from the sum of squares unless it holds a
    library error."""
    device = sq_total.device
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_clip_coef(_scalar(sq_total, device, torch.float64, "sq_total"),
                                  float(max_norm),
                                  _scalar(total_norm, device, torch.float32, "total_norm"),
                                  _scalar(coef, device, torch.float32, "coef"),
                                  _scalar(status, device, torch.int32, "status"),
                                  _stream_handle(stream, device)))


def lt_grad_chunk_count(numels: Sequence[int]) -> int:
    arr = (ctypes.c_int64 * len(numels))(*numels)
    return int(lib().lt_grad_chunk_count(arr, len(numels)))


def lt_grad_sqnorm_partials(grads: Sequence[torch.Tensor], partials: torch.Tensor,
                            workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """a1 on part of a model as its gradients arrive: chunk partials into
    ``partials``, a float64 device view of the model-wide array starting at these
    tensors' first chunk (see include/lazytrain.h)."""
    device = partials.device
    _check_tensors(grads, device, what="grads")
    gdt = _grad_dtype(grads)
    need = lt_grad_chunk_count([g.numel() for g in grads])
    if partials.device != device or partials.dtype != torch.float64 or \
            not partials.is_contiguous() or partials.numel() < need:
        raise ValueError(f"partials must be a contiguous float64 device view of >= {need} entries")
    ws = _workspace(device, int(lib().lt_grad_sqnorm_partials_workspace_bytes(len(grads))),
                    workspace, stream, "partials")
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_grad_sqnorm_partials(
            _ptr_array(grads), _numel_array(grads), len(grads), gdt, partials.data_ptr(),
            ws.data_ptr(), ws.numel() * ws.element_size(), _stream_handle(stream, device)))


def lt_grad_sqnorm_finish(numels: Sequence[int], partials: torch.Tensor, sq_total: torch.Tensor,
                          status: torch.Tensor, sq_per_tensor: Optional[torch.Tensor] = None,
                          workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """a2 from the model-wide partials: S_k, S and the status, bitwise as
    lt_grad_sqnorm over the whole list."""
    device = partials.device
    if partials.dtype != torch.float64 or partials.numel() < lt_grad_chunk_count(numels):
        raise ValueError("partials must hold one float64 per chunk of the model")
    if sq_per_tensor is not None and sq_per_tensor.numel() < len(numels):
        raise ValueError("sq_per_tensor needs one float64 per tensor")
    ws = _workspace(device, int(lib().lt_grad_sqnorm_finish_workspace_bytes(len(numels))),
                    workspace, stream, "finish")
    arr = (ctypes.c_int64 * len(numels))(*numels)
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_grad_sqnorm_finish(
            arr, len(numels), partials.data_ptr(), ws.data_ptr(), ws.numel() * ws.element_size(),
            _scalar(sq_per_tensor, device, torch.float64, "sq_per_tensor"),
            _scalar(sq_total, device, torch.float64, "sq_total"),
            _scalar(status, device, torch.int32, "status"), _stream_handle(stream, device)))


class GradNormAccumulator:
    """Sums a model's gradients part by part as they arrive (in any order), then
    finishes S and the status: lt_grad_sqnorm_partials on each part at its chunk
    offset, lt_grad_sqnorm_finish at the end."""

    def __init__(self, numels: Sequence[int], device):
        self.numels = [int(n) for n in numels]
        self.offsets = [0]
        for n in self.numels:
            self.offsets.append(self.offsets[-1] + -(-n // 8192))
        self.partials = torch.empty(self.offsets[-1], dtype=torch.float64, device=device)

    def add(self, first: int, grads: Sequence[torch.Tensor], stream=None) -> None:
        """Gradients of tensors first .. first + len(grads) - 1 of the model."""
        if first < 0 or first + len(grads) > len(self.numels) or \
                any(g.numel() != self.numels[first + i] for i, g in enumerate(grads)):
            raise ValueError("gradients do not match the model's tensors at this index")
        lt_grad_sqnorm_partials(grads, self.partials[self.offsets[first]:], stream=stream)

    def finish(self, sq_total: torch.Tensor, status: torch.Tensor,
               sq_per_tensor: Optional[torch.Tensor] = None, stream=None) -> None:
        lt_grad_sqnorm_finish(self.numels, self.partials, sq_total, status, sq_per_tensor,
                              stream=stream)


def lt_hybrid8bit_adamw_step(params: Sequence[torch.Tensor], grads: Sequence[torch.Tensor],
                             m_codes: Sequence[torch.Tensor], m_absmax: Sequence[torch.Tensor],
                             v_codes: Sequence[torch.Tensor], v_absmax: Sequence[torch.Tensor],
                             block_size: int, lr: float, beta1: float, beta2: float, eps: float,
                             weight_decay: float, step: int,
                             coef: Optional[torch.Tensor] = None,
                             status: Optional[torch.Tensor] = None,
                             workspace: Optional[torch.Tensor] = None, stream=None,
                             params_bf16=None, code_map: int = LT_MAP_LINEAR,
                             step_state: Optional[torch.Tensor] = None) -> None:
    """Steps a4-a10 in place on params, codes and absmax (see include/lazytrain.h);
    params_bf16 (optional, one bf16 tensor or None per parameter) receives the bf16
    copy of the updated weights; code_map selects the linear or dynamic codes;
    step_state (optional, a device uint8 tensor from lt_step_state_init) supplies the
    step index on the device instead of `step`."""
    k = len(params)
    if not (len(grads) == len(m_codes) == len(m_absmax) == len(v_codes) == len(v_absmax) == k):
        raise ValueError("tensor lists must be of equal length")
    device = _device_of(params, coef, status)
    _check_tensors(params, device, torch.float32, "params")
    _check_tensors(grads, device, what="grads")
    _check_tensors(m_codes, device, torch.int8, "m_codes")
    _check_tensors(v_codes, device, torch.uint8, "v_codes")
    _check_tensors(m_absmax, device, torch.float32, "m_absmax")
    _check_tensors(v_absmax, device, torch.float32, "v_absmax")
    gdt = _grad_dtype(grads)
    if int(block_size) < 1:
        raise LazyTrainError(LT_ERR_INVALID_ARG, "block_size must be a multiple of 64 in "
                             "[64, 65536]")
    for i in range(k):
        n = params[i].numel()
        nb = -(-n // block_size)
        if grads[i].numel() != n or m_codes[i].numel() != n or v_codes[i].numel() != n:
            raise ValueError(f"tensor {i}: params, grads and codes must have {n} elements")
        if m_absmax[i].numel() < nb or v_absmax[i].numel() < nb:
            raise ValueError(f"tensor {i}: absmax arrays need ceil({n}/{block_size}) = {nb} entries")
    wb = _bf16_list(params_bf16, params, device)
    ws = _workspace(device, lt_step_workspace_bytes(k), workspace, stream, "step8")
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_hybrid8bit_adamw_step(
            _ptr_array(params), _ptr_array(grads), gdt, _ptr_array(m_codes), _ptr_array(m_absmax),
            _ptr_array(v_codes), _ptr_array(v_absmax), wb, _numel_array(params), k, int(block_size),
            int(code_map),
            float(lr), float(beta1), float(beta2), float(eps), float(weight_decay), int(step),
            _scalar(coef, device, torch.float32, "coef"), _scalar(status, device, torch.int32, "status"),
            _state_ptr(step_state, device), ws.data_ptr(), ws.numel() * ws.element_size(),
            _stream_handle(stream, device)))


def lt_streamed_workspace_bytes(numels: Sequence[int], layer_first: Sequence[int],
                                grad_dtype: int, block_size: int, ring_slots: int,
                                bf16_copy: bool = False, keep_grads: bool = False) -> int:
    n = (ctypes.c_int64 * len(numels))(*numels)
    f = (ctypes.c_int * len(layer_first))(*layer_first)
    return int(lib().lt_streamed_workspace_bytes(n, len(numels), f, len(layer_first) - 1,
                                                 grad_dtype, block_size, ring_slots,
                                                 int(bool(bf16_copy)), int(bool(keep_grads))))


def lt_streamed_hybrid8bit_adamw_step(params, grads, m_codes, m_absmax, v_codes, v_absmax,
                                      layer_first: Sequence[int], block_size: int, lr: float,
                                      beta1: float, beta2: float, eps: float,
                                      weight_decay: float, step: int, max_norm: float,
                                      ring_slots: int, sq_total: torch.Tensor,
                                      coef: torch.Tensor, status: torch.Tensor,
                                      total_norm: Optional[torch.Tensor] = None,
                                      workspace: Optional[torch.Tensor] = None,
                                      compute_stream=None, h2d_stream=None,
                                      d2h_stream=None, params_bf16=None,
                                      norm_ready: bool = False,
                                      code_map: int = LT_MAP_LINEAR,
                                      keep_grads: bool = False, layer_events=None) -> None:
    """Step a11: host-resident tensors (CPU, ideally pinned) streamed layer by layer
    through HBM; scalar outputs are device tensors (see include/lazytrain.h).
    params_bf16 (optional, host bf16 tensors or None) receives the bf16 weight copy.
    With norm_ready, sq_total and status already hold S and its status (summed as the
    gradients arrived) and the first streamed pass is skipped.  With keep_grads every
    gradient stays in HBM from the first pass to the second (2 or 4 B/param of
    workspace), so it crosses the link once.  layer_events (optional): 8 torch.cuda.Event
    (or None) per layer, recorded around each layer's copies and kernels (see the
    header for which is which)."""
    k = len(params)
    if k == 0 or not (len(grads) == len(m_codes) == len(m_absmax) == len(v_codes) ==
                      len(v_absmax) == k):
        raise ValueError("tensor lists must be non-empty and of equal length")
    cpu = torch.device("cpu")
    _check_tensors(params, cpu, torch.float32, "params")
    _check_tensors(grads, cpu, what="grads")
    _check_tensors(m_codes, cpu, torch.int8, "m_codes")
    _check_tensors(v_codes, cpu, torch.uint8, "v_codes")
    _check_tensors(m_absmax, cpu, torch.float32, "m_absmax")
    _check_tensors(v_absmax, cpu, torch.float32, "v_absmax")
    gdt = _grad_dtype(grads)
    if int(block_size) < 1:
        raise LazyTrainError(LT_ERR_INVALID_ARG, "block_size must be a multiple of 64 in "
                             "[64, 65536]")
    for i in range(k):
        n = params[i].numel()
        nb = -(-n // block_size)
        if grads[i].numel() != n or m_codes[i].numel() != n or v_codes[i].numel() != n:
            raise ValueError(f"tensor {i}: params, grads and codes must have {n} elements")
        if m_absmax[i].numel() < nb or v_absmax[i].numel() < nb:
            raise ValueError(f"tensor {i}: absmax arrays need {nb} entries")
    device = sq_total.device
    wb = _bf16_list(params_bf16, params, cpu)
    numels = [p.numel() for p in params]
    nbytes = lt_streamed_workspace_bytes(numels, layer_first, gdt, block_size, ring_slots,
                                         wb is not None, keep_grads)
    if nbytes == 0:
        raise ValueError("invalid layer_first, block_size or ring_slots")
    cs = _stream_handle(compute_stream, device)
    workspace = _workspace(device, nbytes, workspace, compute_stream, "streamed")
    if compute_stream is not None and hasattr(compute_stream, "cuda_stream"):
        workspace.record_stream(compute_stream)  # in use on that stream until the step is done
    first = (ctypes.c_int * len(layer_first))(*layer_first)
    events = None
    if layer_events is not None:
        if len(layer_events) != 8 * (len(layer_first) - 1):
            raise ValueError("layer_events needs 8 entries per layer")
        for e in layer_events:
            if e is not None and not e.cuda_event:  # torch creates an event at its first record
                e.record(torch.cuda.current_stream(device))
        events = (ctypes.c_void_p * len(layer_events))(
            *[0 if e is None else e.cuda_event for e in layer_events])
    hs = _stream_handle(h2d_stream, device) if h2d_stream is not None else cs
    ds = _stream_handle(d2h_stream, device) if d2h_stream is not None else cs
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_streamed_hybrid8bit_adamw_step(
            _ptr_array(params), _ptr_array(grads), gdt, _ptr_array(m_codes), _ptr_array(m_absmax),
            _ptr_array(v_codes), _ptr_array(v_absmax), wb, _numel_array(params), k, first,
            len(layer_first) - 1, int(block_size), int(code_map), float(lr), float(beta1),
            float(beta2), float(eps),
            float(weight_decay), int(step), float(max_norm), int(bool(norm_ready)),
            int(bool(keep_grads)), int(ring_slots),
            workspace.data_ptr(),
            workspace.numel() * workspace.element_size(),
            _scalar(sq_total, device, torch.float64, "sq_total"),
            _scalar(total_norm, device, torch.float32, "total_norm"),
            _scalar(coef, device, torch.float32, "coef"), _scalar(status, device, torch.int32, "status"),
            events, cs, hs, ds))


def lt_adamw_fp32_workspace_bytes(n_tensors: int) -> int:
    return int(lib().lt_adamw_fp32_workspace_bytes(n_tensors))


def lt_adamw_fp32_step(params: Sequence[torch.Tensor], grads: Sequence[torch.Tensor],
                       exp_avg: Sequence[torch.Tensor], exp_avg_sq: Sequence[torch.Tensor],
                       lr: float, beta1: float, beta2: float, eps: float, weight_decay: float,
                       step: int, coef: Optional[torch.Tensor] = None,
                       status: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None, stream=None,
                       params_bf16=None, step_state: Optional[torch.Tensor] = None) -> None:
    """fp32-state AdamW, in place on params, exp_avg and exp_avg_sq (device tensors);
    params_bf16 as in lt_hybrid8bit_adamw_step."""
    k = len(params)
    if not (len(grads) == len(exp_avg) == len(exp_avg_sq) == k):
        raise ValueError("tensor lists must be of equal length")
    device = _device_of(params, coef, status)
    _check_tensors(params, device, torch.float32, "params")
    _check_tensors(grads, device, what="grads")
    _check_tensors(exp_avg, device, torch.float32, "exp_avg")
    _check_tensors(exp_avg_sq, device, torch.float32, "exp_avg_sq")
    gdt = _grad_dtype(grads)
    for i in range(k):
        n = params[i].numel()
        if grads[i].numel() != n or exp_avg[i].numel() != n or exp_avg_sq[i].numel() != n:
            raise ValueError(f"tensor {i}: params, grads and states must have {n} elements")
    wb = _bf16_list(params_bf16, params, device)
    ws = _workspace(device, lt_adamw_fp32_workspace_bytes(k), workspace, stream, "step32")
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_adamw_fp32_step(
            _ptr_array(params), _ptr_array(grads), gdt, _ptr_array(exp_avg), _ptr_array(exp_avg_sq),
            wb, _numel_array(params), k, float(lr), float(beta1), float(beta2), float(eps),
            float(weight_decay), int(step), _scalar(coef, device, torch.float32, "coef"),
            _scalar(status, device, torch.int32, "status"), _state_ptr(step_state, device),
            ws.data_ptr(), ws.numel() * ws.element_size(), _stream_handle(stream, device)))


def lt_select_8bit_slice(numels: Sequence[int], fraction: float):
    """Returns (list of bools: tensor takes 8-bit states, parameters chosen)."""
    n = (ctypes.c_int64 * len(numels))(*numels)
    out = (ctypes.c_uint8 * len(numels))()
    chosen = ctypes.c_int64()
    _check(lib().lt_select_8bit_slice(n, len(numels), float(fraction), out, ctypes.byref(chosen)))
    return [bool(x) for x in out], chosen.value


def _state_ptr(state: Optional[torch.Tensor], device) -> int:
    if state is None:
        return 0
    if state.device != device or state.dtype != torch.uint8 or not state.is_contiguous():
        raise ValueError(f"step_state must be a contiguous uint8 tensor on {device}")
    return state.data_ptr()


STEP_STATE_HEADER = 64  # bytes of lt_step_state before the table


def lt_step_state_bytes(table_len: int) -> int:
    return int(lib().lt_step_state_bytes(int(table_len)))


def lt_step_table(beta1: float, beta2: float, t_first: int, count: int):
    """Host table entries of steps t_first .. t_first + count - 1, as a numpy structured
    array (one_minus_beta1_t float64, rbc2 float32)."""
    import numpy as np
    out = np.zeros(count, dtype=[("one_minus_beta1_t", "<f8"), ("rbc2", "<f4"),
                                 ("reserved", "<f4")])
    _check(lib().lt_step_table(float(beta1), float(beta2), int(t_first), int(count),
                               out.ctypes.data if count else None))
    return out


def lt_step_state_init(state: torch.Tensor, table_len: int, beta1: float, beta2: float,
                       applied: int = 0, skips: int = 0, max_skips: int = 0,
                       from_state: Optional[torch.Tensor] = None, stream=None) -> None:
    """Writes a device step state (see include/lazytrain.h) into a uint8 tensor."""
    device = state.device
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_step_state_init(
            _state_ptr(state, device), state.numel(), int(table_len), float(beta1), float(beta2),
            int(applied), int(skips), int(max_skips), _state_ptr(from_state, device),
            _stream_handle(stream, device)))


def lt_step_state_advance(state: torch.Tensor, status: torch.Tensor, stream=None) -> None:
    device = state.device
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_step_state_advance(_state_ptr(state, device),
                                           _scalar(status, device, torch.int32, "status"),
                                           _stream_handle(stream, device)))


def lt_read_status(status: torch.Tensor, stream=None) -> int:
    """Reads the device status word (synchronizes the stream)."""
    out = ctypes.c_int32()
    device = status.device
    with torch.cuda.device(device):  # the library works on the current device
        _check(lib().lt_read_status(_scalar(status, device, torch.int32, "status"),
                                    _stream_handle(stream, device), ctypes.byref(out)))
    return out.value


def lt_set_max_workgroups(max_workgroups: int) -> None:
    _check(lib().lt_set_max_workgroups(int(max_workgroups)))


def lt_workspace_release(workspace) -> None:
    """Makes the library forget what it wrote into a workspace (a tensor or a device
    address); call it before freeing or reusing a workspace passed to earlier calls."""
    ptr = workspace.data_ptr() if hasattr(workspace, "data_ptr") else int(workspace)
    _check(lib().lt_workspace_release(ptr))


# ------------------------------------------------------------- optimizer object

class Hybrid8bitAdamW:
    """Runs one clipped step per call over a list of fp32 master tensors:
    lt_grad_sqnorm -> lt_clip_coef -> the fused steps, all enqueued on one stream
    without a host synchronization.  With ``slice_fraction`` None every tensor keeps
    8-bit states; otherwise lt_select_8bit_slice picks the tensors that do (the
    paper's 2% slice) and the others keep fp32 states (lt_adamw_fp32_step), all under
    one global norm.

    The step count lives on the device (a step state, see lt_step_state_init): each
    step takes its index and bias corrections there, and lt_step_state_advance counts
    it, so ``step()`` never waits for an earlier step and can run any number of steps
    ahead of the GPU.  A step whose norm is not finite writes nothing and does not
    count; after ``max_consecutive_skips`` of them in a row (App. C: three; None
    never stops) the device skips every later step too.  The host learns of both
    from status snapshots copied behind each step and read without waiting:
    ``step()`` raises NonFiniteAbort once it has seen the stop, ``last_status()``
    waits for the last step and raises then.  ``step_count`` and
    ``consecutive_skips`` are the device's as last seen (exact after
    ``last_status()``).  With ``bf16_copy`` the steps also keep ``params_bf16``, a
    bf16 copy of every parameter for the next forward pass, written by the step
    kernels (valid after the first step).  The moments take the non-linear
    decade-tree codes by default (``code_map``): with the linear codes a second
    moment far below its block's largest rounds to code 0 while the first moment
    does not, and the update then divides by little more than eps (the drift tests
    measure hundreds of lr against fp64 AdamW); pass LT_MAP_LINEAR for the linear
    codes."""

    TABLE = 4096     # step-table entries to start with; doubled on the device as needed
    SNAPSHOTS = 64   # status snapshots in flight (step() waits only beyond this many)

    def __init__(self, params: Sequence[torch.Tensor], lr: float = 1e-5,
                 betas=(0.9, 0.999), eps: float = 1e-8, weight_decay: float = 0.01,
                 max_norm: float = 1.0, block_size: int = 4096,
                 slice_fraction: Optional[float] = None, bf16_copy: bool = False,
                 code_map: int = LT_MAP_DYNAMIC, max_consecutive_skips: Optional[int] = 3):
        self.params = list(params)
        if not self.params:
            raise ValueError("no parameters")
        if max_consecutive_skips is not None and max_consecutive_skips < 1:
            raise ValueError("max_consecutive_skips must be >= 1 or None")
        self.max_consecutive_skips = max_consecutive_skips
        dev = self.params[0].device
        self.device = dev
        self.lr, self.betas, self.eps, self.weight_decay = lr, betas, eps, weight_decay
        self.max_norm, self.block_size, self.code_map = max_norm, block_size, code_map
        if slice_fraction is None:
            self.is_8bit = [True] * len(self.params)
        else:
            self.is_8bit, _ = lt_select_8bit_slice([p.numel() for p in self.params],
                                                   slice_fraction)
        self.idx8 = [i for i, b in enumerate(self.is_8bit) if b]
        self.idx32 = [i for i, b in enumerate(self.is_8bit) if not b]
        p8 = [self.params[i] for i in self.idx8]
        self.m_codes = [torch.zeros(p.numel(), dtype=torch.int8, device=dev) for p in p8]
        self.v_codes = [torch.zeros(p.numel(), dtype=torch.uint8, device=dev) for p in p8]
        nb = [-(-p.numel() // block_size) for p in p8]
        self.m_absmax = [torch.zeros(n, dtype=torch.float32, device=dev) for n in nb]
        self.v_absmax = [torch.zeros(n, dtype=torch.float32, device=dev) for n in nb]
        self.exp_avg = [torch.zeros_like(self.params[i]).reshape(-1) for i in self.idx32]
        self.exp_avg_sq = [torch.zeros_like(self.params[i]).reshape(-1) for i in self.idx32]
        self.sq_total = torch.zeros(1, dtype=torch.float64, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.coef = torch.ones(1, dtype=torch.float32, device=dev)
        self.total_norm = torch.zeros(1, dtype=torch.float32, device=dev)
        self.params_bf16 = [torch.empty(p.numel(), dtype=torch.bfloat16, device=dev)
                            for p in self.params] if bf16_copy else None
        # snapshots: per step, the state's first 32 bytes and the status, in pinned memory
        self._snap = torch.zeros((self.SNAPSHOTS, 48), dtype=torch.uint8, pin_memory=True)
        self._snap_events = [None] * self.SNAPSHOTS
        self._pending = []  # snapshot slots enqueued and not yet read, oldest first
        self._next_slot = 0
        self._reset_state(0, 0)
        # the zeroed states and the step state were written on the current stream; steps
        # may come on any stream
        torch.cuda.synchronize(dev)

    # ------------------------------------------------------------ step state
    def _reset_state(self, applied: int, skips: int, stream=None) -> None:
        """A fresh device step state with this count (enqueued on the stream)."""
        self._table_len = max(self.TABLE, 2 * (applied + 1))
        self._state = torch.empty(lt_step_state_bytes(self._table_len), dtype=torch.uint8,
                                  device=self.device)
        lt_step_state_init(self._state, self._table_len, self.betas[0], self.betas[1],
                           applied=applied, skips=skips,
                           max_skips=self.max_consecutive_skips or 0, stream=stream)
        self._bound = applied  # the device count cannot exceed this
        self._seen = {"applied": applied, "skips": skips, "stopped": 0,
                      "status": LT_STATUS_OK}

    def _grow_state(self, stream) -> None:
        """Doubles the step table; the count moves over on the device, unread."""
        old = self._state
        self._table_len *= 2
        self._state = torch.empty(lt_step_state_bytes(self._table_len), dtype=torch.uint8,
                                  device=self.device)
        lt_step_state_init(self._state, self._table_len, self.betas[0], self.betas[1],
                           max_skips=self.max_consecutive_skips or 0, from_state=old,
                           stream=stream)
        old.record_stream(self._torch_stream(stream))

    def _read_snapshot(self, slot: int) -> None:
        import struct
        raw = bytes(self._snap[slot].numpy())
        applied, _, skips, _, stopped = struct.unpack_from("<qqiii", raw, 0)
        status = struct.unpack_from("<i", raw, 32)[0]
        self._seen = {"applied": applied, "skips": skips, "stopped": stopped, "status": status}
        if status == LT_STATUS_BAD_WORKSPACE:
            raise LazyTrainError(LT_ERR_WORKSPACE, "a workspace lost its descriptors (it was "
                                 "written or freed without lt_workspace_release)")

    def _observe(self, wait: bool) -> None:
        """Reads the snapshots whose copies have completed (all of them with wait)."""
        while self._pending:
            slot = self._pending[0]
            ev = self._snap_events[slot]
            if wait:
                ev.synchronize()
            elif not ev.query():
                return
            self._pending.pop(0)
            self._read_snapshot(slot)

    @property
    def step_count(self) -> int:
        """Steps applied, as last seen from the device."""
        return self._seen["applied"]

    @property
    def consecutive_skips(self) -> int:
        return self._seen["skips"]

    @consecutive_skips.setter
    def consecutive_skips(self, value: int) -> None:
        """Sets the device's count of skips in a row (and clears a stop), in stream
        order, so that a caller can go on after NonFiniteAbort."""
        self._observe(wait=True)
        v = torch.tensor([int(value)], dtype=torch.int32).view(torch.uint8)
        self._state[16:20].copy_(v)                        # skips
        self._state[24:28].zero_()                         # stopped
        torch.cuda.synchronize(self.device)  # before steps on any stream read it
        self._seen = dict(self._seen, skips=int(value), stopped=0)

    def _raise_if_stopped(self) -> None:
        if self._seen["stopped"] == 1:
            raise NonFiniteAbort(self._seen["skips"])
        if self._seen["stopped"] == 2:
            raise LazyTrainError(LT_ERR_INVALID_ARG, "the step table ran out")

    def _torch_stream(self, stream):
        dev = self.params[0].device
        if stream is None:
            return torch.cuda.current_stream(dev)
        if hasattr(stream, "cuda_stream"):
            return stream
        return torch.cuda.ExternalStream(int(stream), device=dev)

    # ------------------------------------------------------------------ step
    def step(self, grads: Sequence[torch.Tensor], stream=None) -> None:
        """One clipped step with one gradient per parameter, in the order of the
        parameters (a zero-element parameter takes a zero-element gradient)."""
        grads = list(grads)
        if len(grads) != len(self.params):
            raise ValueError(f"step() needs one gradient per parameter: got {len(grads)} "
                             f"for {len(self.params)} parameters")
        for i, (g, p) in enumerate(zip(grads, self.params)):
            if g is None:
                raise ValueError(f"gradient {i} is None (every parameter needs a gradient; "
                                 "pass zeros for a parameter that received none)")
            if g.numel() != p.numel():
                raise ValueError(f"gradient {i} has {g.numel()} elements, its parameter "
                                 f"{p.numel()}")
        self._observe(wait=False)
        self._raise_if_stopped()
        if self._bound + 1 > self._table_len:
            self._grow_state(stream)
        lt_grad_sqnorm(grads, self.sq_total, self.status, stream=stream)
        clip = self.max_norm if self.max_norm is not None else math.inf
        lt_clip_coef(self.sq_total, clip, self.coef, self.total_norm, stream=stream)
        hyper = dict(lr=self.lr, beta1=self.betas[0], beta2=self.betas[1], eps=self.eps,
                     weight_decay=self.weight_decay, step=0, coef=self.coef, status=self.status,
                     stream=stream, step_state=self._state)
        wb = self.params_bf16
        if self.idx8:
            lt_hybrid8bit_adamw_step([self.params[i] for i in self.idx8],
                                     [grads[i] for i in self.idx8], self.m_codes, self.m_absmax,
                                     self.v_codes, self.v_absmax, self.block_size,
                                     params_bf16=None if wb is None else [wb[i] for i in self.idx8],
                                     code_map=self.code_map, **hyper)
        if self.idx32:
            lt_adamw_fp32_step([self.params[i] for i in self.idx32],
                               [grads[i] for i in self.idx32], self.exp_avg, self.exp_avg_sq,
                               params_bf16=None if wb is None else [wb[i] for i in self.idx32],
                               **hyper)
        lt_step_state_advance(self._state, self.status, stream=stream)
        self._bound += 1
        # a snapshot of the count and the status, read later without waiting
        slot = self._next_slot
        self._next_slot = (slot + 1) % self.SNAPSHOTS
        if slot in self._pending:  # more than SNAPSHOTS steps ahead: wait for the oldest
            self._observe(wait=True)
        s = self._torch_stream(stream)
        with torch.cuda.stream(s):
            self._snap[slot, :32].copy_(self._state[:32], non_blocking=True)
            self._snap[slot, 32:36].copy_(self.status.view(torch.uint8), non_blocking=True)
        ev = torch.cuda.Event()
        ev.record(s)
        self._snap_events[slot] = ev
        self._pending.append(slot)

    def last_status(self, stream=None) -> int:
        """Waits for the last step only (not for work enqueued after it) and returns
        its status; raises NonFiniteAbort if the device has stopped after
        max_consecutive_skips skips in a row."""
        if self._pending:
            self._observe(wait=True)
        else:
            self._seen["status"] = lt_read_status(self.status, stream)
        self._raise_if_stopped()
        return self._seen["status"]

    def state_dict(self, stream=None) -> dict:
        """The optimizer state for a checkpoint: the step count, the hyperparameters,
        which tensors are 8-bit, and host copies of the codes, scales and fp32 moments
        (the master weights are the caller's parameters).  Waits for the last step."""
        self._observe(wait=True)
        host = lambda ts: [t.detach().cpu().clone() for t in ts]
        return {
            "step_count": self.step_count,
            "consecutive_skips": self.consecutive_skips,
            "hyper": {"lr": self.lr, "betas": tuple(self.betas), "eps": self.eps,
                      "weight_decay": self.weight_decay, "max_norm": self.max_norm,
                      "block_size": self.block_size, "code_map": self.code_map},
            "is_8bit": list(self.is_8bit),
            "m_codes": host(self.m_codes), "m_absmax": host(self.m_absmax),
            "v_codes": host(self.v_codes), "v_absmax": host(self.v_absmax),
            "exp_avg": host(self.exp_avg), "exp_avg_sq": host(self.exp_avg_sq),
        }

    def load_state_dict(self, state: dict) -> None:
        """Restores a state_dict() into an optimizer built over parameters of the same
        shapes with the same slice; the next step continues bitwise as if never
        interrupted."""
        if list(state["is_8bit"]) != list(self.is_8bit):
            raise ValueError("the checkpoint's 8-bit slice differs from this optimizer's")
        h = state["hyper"]
        if h["block_size"] != self.block_size or h["code_map"] != self.code_map:
            raise ValueError("the checkpoint's block size or code map differs")
        self.lr, self.betas, self.eps = h["lr"], tuple(h["betas"]), h["eps"]
        self.weight_decay, self.max_norm = h["weight_decay"], h["max_norm"]
        for name in ("m_codes", "m_absmax", "v_codes", "v_absmax", "exp_avg", "exp_avg_sq"):
            mine, saved = getattr(self, name), state[name]
            if len(mine) != len(saved):
                raise ValueError(f"{name}: {len(saved)} tensors in the checkpoint, "
                                 f"{len(mine)} here")
            for a, b in zip(mine, saved):
                if a.shape != b.shape or a.dtype != b.dtype:
                    raise ValueError(f"{name}: shape or dtype differs from the checkpoint")
                a.copy_(b)
        self._observe(wait=True)
        self._reset_state(int(state["step_count"]), int(state.get("consecutive_skips", 0)))
        torch.cuda.synchronize(self.device)


class StreamedHybrid8bitAdamW:
    """The optimizer object of the layer-streamed step (lt_streamed_hybrid8bit_adamw_step):
    the fp32 master weights (the caller's CPU tensors, pinned for overlapped copies) and
    the 8-bit states (pinned host memory allocated here) stay in host memory and pass
    through HBM layer by layer, as the paper keeps parameters and optimizer states in
    CPU memory (Sec. 3.5).  ``layer_first`` splits the parameter list into layers
    (layer i is parameters [layer_first[i], layer_first[i + 1])).  The workspace, the
    device scalars and three streams are allocated once.  With ``keep_grads`` (the
    default) the gradients stay in HBM between the two passes and cross the link once.
    ``step()`` returns when the host state is updated and gives the step's status; a
    skipped step (non-finite norm) changes nothing and counts towards
    ``max_consecutive_skips`` as in Hybrid8bitAdamW (NonFiniteAbort)."""

    def __init__(self, params: Sequence[torch.Tensor], layer_first: Sequence[int], device,
                 lr: float = 1e-5, betas=(0.9, 0.999), eps: float = 1e-8,
                 weight_decay: float = 0.01, max_norm: float = 1.0, block_size: int = 4096,
                 ring_slots: int = 3, keep_grads: bool = True, code_map: int = LT_MAP_DYNAMIC,
                 max_consecutive_skips: Optional[int] = 3, grad_dtype=torch.bfloat16):
        self.params = list(params)
        if not self.params:
            raise ValueError("no parameters")
        cpu = torch.device("cpu")
        _check_tensors(self.params, cpu, torch.float32, "params")
        if max_consecutive_skips is not None and max_consecutive_skips < 1:
            raise ValueError("max_consecutive_skips must be >= 1 or None")
        if grad_dtype not in (torch.bfloat16, torch.float32):
            raise ValueError("grad_dtype must be torch.bfloat16 or torch.float32")
        self.device = torch.device(device)
        self.layer_first = list(layer_first)
        self.lr, self.betas, self.eps, self.weight_decay = lr, betas, eps, weight_decay
        self.max_norm, self.block_size, self.code_map = max_norm, block_size, code_map
        self.ring_slots, self.keep_grads = ring_slots, keep_grads
        self.max_consecutive_skips = max_consecutive_skips
        numels = [p.numel() for p in self.params]
        gdt = LT_DTYPE_BF16 if grad_dtype == torch.bfloat16 else LT_DTYPE_F32
        nbytes = lt_streamed_workspace_bytes(numels, self.layer_first, gdt, block_size,
                                             ring_slots, False, keep_grads)
        if nbytes == 0:
            raise ValueError("invalid layer_first, block_size or ring_slots")
        pinned = lambda n, dt: torch.zeros(n, dtype=dt, pin_memory=True)
        nb = [-(-n // block_size) for n in numels]
        self.m_codes = [pinned(n, torch.int8) for n in numels]
        self.v_codes = [pinned(n, torch.uint8) for n in numels]
        self.m_absmax = [pinned(n, torch.float32) for n in nb]
        self.v_absmax = [pinned(n, torch.float32) for n in nb]
        dev = self.device
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        self.sq_total = torch.zeros(1, dtype=torch.float64, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.coef = torch.ones(1, dtype=torch.float32, device=dev)
        self.total_norm = torch.zeros(1, dtype=torch.float32, device=dev)
        self.streams = [torch.cuda.Stream(dev) for _ in range(3)]  # compute, in, out
        self.step_count = 0  # steps applied (skipped steps do not count)
        self.consecutive_skips = 0

    def step(self, grads: Sequence[torch.Tensor]) -> int:
        """One clipped step with one host gradient per parameter (CPU tensors, pinned
        for overlapped copies).  Returns LT_STATUS_OK or LT_STATUS_NONFINITE once the
        updated weights, codes and scales are in host memory."""
        if (self.max_consecutive_skips is not None and
                self.consecutive_skips >= self.max_consecutive_skips):
            raise NonFiniteAbort(self.consecutive_skips)
        grads = list(grads)
        if len(grads) != len(self.params):
            raise ValueError(f"step() needs one gradient per parameter: got {len(grads)} "
                             f"for {len(self.params)} parameters")
        cs, hs, ds = self.streams
        cs.wait_stream(torch.cuda.current_stream(self.device))
        t = self.step_count + 1
        lt_streamed_hybrid8bit_adamw_step(
            self.params, grads, self.m_codes, self.m_absmax, self.v_codes, self.v_absmax,
            self.layer_first, self.block_size, lr=self.lr, beta1=self.betas[0],
            beta2=self.betas[1], eps=self.eps, weight_decay=self.weight_decay, step=t,
            max_norm=self.max_norm if self.max_norm is not None else math.inf,
            ring_slots=self.ring_slots, sq_total=self.sq_total, coef=self.coef,
            status=self.status, total_norm=self.total_norm, workspace=self.workspace,
            compute_stream=cs, h2d_stream=hs, d2h_stream=ds, code_map=self.code_map,
            keep_grads=self.keep_grads)
        st = lt_read_status(self.status, cs)  # waits for the call's work, copies out included
        if st == LT_STATUS_BAD_WORKSPACE:
            raise LazyTrainError(LT_ERR_WORKSPACE, "the workspace lost its descriptors")
        if st == LT_STATUS_NONFINITE:
            self.consecutive_skips += 1
        else:
            self.consecutive_skips = 0
            self.step_count = t
        if (self.max_consecutive_skips is not None and
                self.consecutive_skips >= self.max_consecutive_skips):
            raise NonFiniteAbort(self.consecutive_skips)
        return st

    def state_dict(self) -> dict:
        """The step count, hyperparameters and copies of the 8-bit states (the master
        weights are the caller's parameters)."""
        copy = lambda ts: [t.clone() for t in ts]
        return {"step_count": self.step_count, "consecutive_skips": self.consecutive_skips,
                "hyper": {"lr": self.lr, "betas": tuple(self.betas), "eps": self.eps,
                          "weight_decay": self.weight_decay, "max_norm": self.max_norm,
                          "block_size": self.block_size, "code_map": self.code_map},
                "m_codes": copy(self.m_codes), "m_absmax": copy(self.m_absmax),
                "v_codes": copy(self.v_codes), "v_absmax": copy(self.v_absmax)}

    def load_state_dict(self, state: dict) -> None:
        h = state["hyper"]
        if h["block_size"] != self.block_size or h["code_map"] != self.code_map:
            raise ValueError("the checkpoint's block size or code map differs")
        for name in ("m_codes", "m_absmax", "v_codes", "v_absmax"):
            mine, saved = getattr(self, name), state[name]
            if len(mine) != len(saved) or any(a.shape != b.shape or a.dtype != b.dtype
                                               for a, b in zip(mine, saved)):
                raise ValueError(f"{name}: the checkpoint's tensors differ from this optimizer's")
            for a, b in zip(mine, saved):
                a.copy_(b)
        self.lr, self.betas, self.eps = h["lr"], tuple(h["betas"]), h["eps"]
        self.weight_decay, self.max_norm = h["weight_decay"], h["max_norm"]
        self.step_count = int(state["step_count"])
        self.consecutive_skips = int(state.get("consecutive_skips", 0))
