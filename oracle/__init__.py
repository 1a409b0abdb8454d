"""CPU oracle of the Hybrid 8-bit optimizer step -- TEST INFRASTRUCTURE.

Thin ctypes marshalling over ``liblazytrain_oracle.so`` (plain C, see
``lazytrain_oracle.h``).  Arrays are numpy arrays on the host; bf16 tensors are
carried as ``uint16`` arrays of raw bf16 bits.  Only the tests, the package
smoke check and the benchmark's CPU-baseline leg may import this module; the
product path never does.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

F32, BF16 = 0, 1
STATUS_OK, STATUS_NONFINITE = 0, 1
CHUNK = 8192

_HERE = os.path.dirname(os.path.abspath(__file__))
# LTO_LIBRARY names another build of the same source (the tests build copies
# with one planted mistake each and check that the pins reject them).
_LIB_PATH = os.environ.get("LTO_LIBRARY") or os.path.join(_HERE, "liblazytrain_oracle.so")
_lib = None

_i64p = ctypes.POINTER(ctypes.c_int64)


class _Scalars(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in
                ("beta1", "beta2", "eps", "c1", "c2", "decay", "step_size", "rbc2")]
_vpp = ctypes.POINTER(ctypes.c_void_p)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        if os.environ.get("LTO_LIBRARY"):
            raise FileNotFoundError(f"LTO_LIBRARY names a missing file: {_LIB_PATH}")
        from . import build as _build  # builds the oracle's own C library

        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.lto_grad_sqnorm.argtypes = [_vpp, _i64p, ctypes.c_int, ctypes.c_int,
                                    ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_int32), ctypes.c_int]
    lib.lto_grad_sqnorm.restype = ctypes.c_int
    lib.lto_grad_sqnorm_naive.argtypes = [_vpp, _i64p, ctypes.c_int, ctypes.c_int]
    lib.lto_grad_sqnorm_naive.restype = ctypes.c_double
    lib.lto_clip_coef.argtypes = [ctypes.c_double, ctypes.c_float,
                                  ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_float)]
    lib.lto_clip_coef.restype = None
    fp = ctypes.POINTER(ctypes.c_float)
    lib.lto_step_scalars.argtypes = [ctypes.c_double] * 5 + [ctypes.c_int64,
                                                              ctypes.POINTER(_Scalars)]
    lib.lto_step_scalars.restype = None
    lib.lto_hybrid8bit_adamw_step.argtypes = [
        _vpp, _vpp, ctypes.c_int, _vpp, _vpp, _vpp, _vpp, _i64p, ctypes.c_int, ctypes.c_int64,
        ctypes.c_int, ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_double,
        ctypes.c_double,
        ctypes.c_int64, fp, ctypes.POINTER(ctypes.c_int32), ctypes.c_int]
    lib.lto_hybrid8bit_adamw_step.restype = ctypes.c_int
    for name, qt in (("signed", ctypes.c_int8), ("unsigned", ctypes.c_uint8),
                     ("dynamic_signed", ctypes.c_int8), ("dynamic_unsigned", ctypes.c_uint8)):
        qf = getattr(lib, "lto_quantize_" + name)
        qf.argtypes = [fp, ctypes.c_int64, ctypes.POINTER(qt), fp]
        qf.restype = None
        df = getattr(lib, "lto_dequantize_" + name)
        df.argtypes = [ctypes.POINTER(qt), ctypes.c_int64, ctypes.c_float, fp]
        df.restype = None
    lib.lto_dynamic_map.argtypes = [ctypes.c_int, fp]
    lib.lto_dynamic_map.restype = None
    lib.lto_adamw_fp32_step.argtypes = [fp, ctypes.c_void_p, ctypes.c_int, fp, fp,
                                        ctypes.c_int64] + [ctypes.c_double] * 5 + [
                                            ctypes.c_int64, ctypes.c_float]
    lib.lto_adamw_fp32_step.restype = None
    lib.lto_round_bf16.argtypes = [fp, ctypes.c_int64, ctypes.POINTER(ctypes.c_uint16)]
    lib.lto_round_bf16.restype = None
    _lib = lib
    return lib


def _gdt(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"gradient dtype must be float32 or uint16 (bf16 bits), got {a.dtype}")


def _contig(arrays, dtype):
    for a in arrays:
        if a.dtype != dtype or not a.flags["C_CONTIGUOUS"]:
            raise TypeError(f"expected C-contiguous {dtype}, got {a.dtype}")


def _ptrs(arrays):
    return (ctypes.c_void_p * max(1, len(arrays)))(*[a.ctypes.data for a in arrays])


def _numels(arrays):
    return (ctypes.c_int64 * max(1, len(arrays)))(*[a.size for a in arrays])


def grad_sqnorm(grads, n_threads: int = 1):
    """Returns (S_k as float64 array, S, status) in the fixed reduction order."""
    gdt = _gdt(grads[0]) if grads else F32
    _contig(grads, grads[0].dtype if grads else np.float32)
    sk = np.zeros(max(1, len(grads)), dtype=np.float64)
    s = ctypes.c_double()
    st = ctypes.c_int32()
    rc = _load().lto_grad_sqnorm(_ptrs(grads), _numels(grads), len(grads), gdt,
                                 sk.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                 ctypes.byref(s), ctypes.byref(st), n_threads)
    if rc != 0:
        raise ValueError(f"lto_grad_sqnorm failed ({rc})")
    return sk[: len(grads)], s.value, st.value


def grad_sqnorm_naive(grads) -> float:
    return _load().lto_grad_sqnorm_naive(_ptrs(grads), _numels(grads), len(grads),
                                         _gdt(grads[0]) if grads else F32)


def clip_coef(sq_total: float, max_norm: float):
    """Returns (norm, coef) as numpy float32 scalars."""
    n = ctypes.c_float()
    c = ctypes.c_float()
    _load().lto_clip_coef(sq_total, max_norm, ctypes.byref(n), ctypes.byref(c))
    return np.float32(n.value), np.float32(c.value)


def step_scalars(lr, beta1, beta2, eps, weight_decay, step):
    """Returns a dict of the fp32 step scalars (numpy float32 values)."""
    out = _Scalars()
    _load().lto_step_scalars(lr, beta1, beta2, eps, weight_decay, step, ctypes.byref(out))
    return {n: np.float32(getattr(out, n)) for n, _ in _Scalars._fields_}


MAP_LINEAR, MAP_DYNAMIC = 0, 1


def hybrid8bit_adamw_step(params, grads, m_codes, m_absmax, v_codes, v_absmax, block_size: int,
                          lr: float, beta1: float, beta2: float, eps: float, weight_decay: float,
                          step: int, coef=None, status=None, n_threads: int = 1,
                          code_map: int = MAP_LINEAR) -> None:
    """In-place step over lists of numpy arrays (see lazytrain_oracle.h)."""
    k = len(params)
    if not (len(grads) == len(m_codes) == len(m_absmax) == len(v_codes) == len(v_absmax) == k):
        raise ValueError("tensor lists must have equal length")
    _contig(params, np.float32)
    _contig(m_codes, np.int8)
    _contig(v_codes, np.uint8)
    _contig(m_absmax, np.float32)
    _contig(v_absmax, np.float32)
    gdt = _gdt(grads[0]) if k else F32
    _contig(grads, grads[0].dtype if k else np.float32)
    for p, g, mq, ma, vq, va in zip(params, grads, m_codes, m_absmax, v_codes, v_absmax):
        nb = -(-p.size // block_size)
        if not (g.size == mq.size == vq.size == p.size and ma.size >= nb and va.size >= nb):
            raise ValueError("inconsistent tensor sizes")
    c = ctypes.byref(ctypes.c_float(coef)) if coef is not None else None
    st = ctypes.byref(ctypes.c_int32(status)) if status is not None else None
    rc = _load().lto_hybrid8bit_adamw_step(
        _ptrs(params), _ptrs(grads), gdt, _ptrs(m_codes), _ptrs(m_absmax), _ptrs(v_codes),
        _ptrs(v_absmax), _numels(params), k, block_size, code_map, lr, beta1, beta2, eps,
        weight_decay,
        step, c, st, n_threads)
    if rc != 0:
        raise ValueError(f"lto_hybrid8bit_adamw_step failed ({rc})")


def _fp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def quantize_signed(x: np.ndarray):
    x = np.ascontiguousarray(x, dtype=np.float32)
    q = np.zeros(x.size, dtype=np.int8)
    a = ctypes.c_float()
    _load().lto_quantize_signed(_fp(x), x.size, q.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)),
                                ctypes.byref(a))
    return q, np.float32(a.value)


def quantize_unsigned(x: np.ndarray):
    x = np.ascontiguousarray(x, dtype=np.float32)
    q = np.zeros(x.size, dtype=np.uint8)
    a = ctypes.c_float()
    _load().lto_quantize_unsigned(_fp(x), x.size,
                                  q.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                                  ctypes.byref(a))
    return q, np.float32(a.value)


def dequantize_signed(q: np.ndarray, absmax: float) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.int8)
    x = np.zeros(q.size, dtype=np.float32)
    _load().lto_dequantize_signed(q.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)), q.size,
                                  absmax, _fp(x))
    return x


def dequantize_unsigned(q: np.ndarray, absmax: float) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.uint8)
    x = np.zeros(q.size, dtype=np.float32)
    _load().lto_dequantize_unsigned(q.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), q.size,
                                    absmax, _fp(x))
    return x


def adamw_fp32_step(w, grad, m, v, lr, beta1, beta2, eps, weight_decay, step, coef=1.0) -> None:
    """fp32-state AdamW, in place on numpy float32 arrays w, m, v."""
    _contig([w, m, v], np.float32)
    _load().lto_adamw_fp32_step(_fp(w), grad.ctypes.data, _gdt(grad), _fp(m), _fp(v), w.size,
                                lr, beta1, beta2, eps, weight_decay, step, coef)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) of float32 values: round to nearest even on the
    dropped bits, NaN to a quiet NaN of the same sign."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty(x.shape, dtype=np.uint16)
    _load().lto_round_bf16(_fp(x), x.size, y.ctypes.data_as(ctypes.POINTER(ctypes.c_uint16)))
    return y


def dynamic_map(signed: bool) -> np.ndarray:
    """The dynamic code map's magnitudes: 128 (signed) or 256 (unsigned) float32."""
    t = np.zeros(128 if signed else 256, dtype=np.float32)
    _load().lto_dynamic_map(1 if signed else 0, _fp(t))
    return t


def _quantize(name, x, qtype):
    x = np.ascontiguousarray(x, dtype=np.float32)
    q = np.zeros(x.size, dtype=qtype)
    a = ctypes.c_float()
    ct = ctypes.c_int8 if qtype == np.int8 else ctypes.c_uint8
    getattr(_load(), "lto_quantize_" + name)(_fp(x), x.size, q.ctypes.data_as(ctypes.POINTER(ct)),
                                              ctypes.byref(a))
    return q, a.value


def _dequantize(name, q, absmax, qtype):
    q = np.ascontiguousarray(q, dtype=qtype)
    x = np.zeros(q.size, dtype=np.float32)
    ct = ctypes.c_int8 if qtype == np.int8 else ctypes.c_uint8
    getattr(_load(), "lto_dequantize_" + name)(q.ctypes.data_as(ctypes.POINTER(ct)), q.size,
                                                absmax, _fp(x))
    return x


def quantize_dynamic_signed(x):
    """Sign-magnitude dynamic codes (int8 storage) and the absmax of one block."""
    return _quantize("dynamic_signed", x, np.int8)


def quantize_dynamic_unsigned(x):
    return _quantize("dynamic_unsigned", x, np.uint8)


def dequantize_dynamic_signed(q, absmax: float):
    return _dequantize("dynamic_signed", q, absmax, np.int8)


def dequantize_dynamic_unsigned(q, absmax: float):
    return _dequantize("dynamic_unsigned", q, absmax, np.uint8)
