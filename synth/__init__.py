"""Seeded synthetic workloads for the optimizer step.

The workloads take the *shapes* of the dense decoders the paper trains (Sec. 4.1
setup: Qwen2.5-3B up to the 27B-class Qwen3.6 model; App. C model
configuration) with synthetic values; no dataset items or trained weights are
used.  Values come from ``libltsynth.so`` (counter-based SplitMix64 plus
Box-Muller, see ``ltsynth.c``), so any slice of any tensor can be regenerated
on its own.  This module draws numbers only; it holds none of the optimizer's
arithmetic and is shared by the oracle's tests and the GPU path.

Streams: 0 = weights, 1 = the prior step's gradient (used to build the 8-bit
states), 2 + t = the gradient applied at step t, 101 = zero-block mask;
outlier masks use stream + 1000.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

F32, BF16 = 0, 1
NORMAL, STUDENT_T3 = 0, 1
OUTLIER_NONE, OUTLIER_SCALE, OUTLIER_SET = 0, 1, 2

STREAM_WEIGHTS = 0
STREAM_PRIOR_GRAD = 1
STREAM_ZERO_MASK = 101


def grad_stream(step: int) -> int:
    return 2 + step


_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libltsynth.so")
_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _build

            _build.build()
        lib = ctypes.CDLL(_LIB_PATH)
        lib.lts_fill.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                 ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int,
                                 ctypes.c_double, ctypes.c_double, ctypes.c_int, ctypes.c_double,
                                 ctypes.c_int64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_int]
        lib.lts_fill.restype = None
        lib.lts_block_is_zero.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                          ctypes.c_int64, ctypes.c_int64]
        lib.lts_block_is_zero.restype = ctypes.c_int
        _lib = lib
    return _lib


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


@dataclass(frozen=True)
class Recipe:
    """How one family of values is drawn."""
    dist: int = NORMAL
    scale: float = 1.0
    outlier_p: float = 0.0
    outlier_mode: int = OUTLIER_NONE
    outlier_value: float = 0.0
    zero_block: int = 0
    zero_mod: int = 0


def fill_ptr(ptr: int, dtype: int, offset: int, n: int, seed: int, stream: int, tensor: int,
             recipe: Recipe, n_threads: Optional[int] = None) -> None:
    """Write elements [offset, offset + n) of one tensor to host memory at ptr."""
    _load().lts_fill(ptr, dtype, offset, n, seed, stream, tensor, recipe.dist, recipe.scale,
                     recipe.outlier_p, recipe.outlier_mode, recipe.outlier_value,
                     recipe.zero_block, STREAM_ZERO_MASK, recipe.zero_mod,
                     n_threads or default_threads())


def draw(dtype: int, n: int, seed: int, stream: int, tensor: int, recipe: Recipe, offset: int = 0,
         n_threads: Optional[int] = None) -> np.ndarray:
    out = np.empty(n, dtype=np.float32 if dtype == F32 else np.uint16)
    if n:
        fill_ptr(out.ctypes.data, dtype, offset, n, seed, stream, tensor, recipe, n_threads)
    return out


def block_is_zero(seed: int, tensor: int, block: int, zero_mod: int) -> bool:
    return bool(_load().lts_block_is_zero(seed, STREAM_ZERO_MASK, tensor, block, zero_mod))


# ------------------------------------------------------------------ workloads

def layer_shapes(hidden: int, ffn: int, q_heads: int, kv_heads: int, head_dim: int):
    """Parameter tensors of one dense decoder layer, in the order
    q, k, v, o, gate, up, down, norm1, norm2 (shapes are (out, in))."""
    q = q_heads * head_dim
    kv = kv_heads * head_dim
    return [(q, hidden), (kv, hidden), (kv, hidden), (hidden, q), (ffn, hidden), (ffn, hidden),
            (hidden, ffn), (hidden,), (hidden,)]


LAYER_3B = layer_shapes(2048, 11008, 16, 2, 128)
LAYER_27B = layer_shapes(5120, 17408, 40, 8, 128)
EMBED_3B = (151936, 2048)

LR, BETA1, BETA2, EPS, WEIGHT_DECAY, MAX_NORM = 1e-4, 0.9, 0.999, 1e-8, 0.01, 1.0


@dataclass
class Workload:
    name: str
    seed: int
    shapes: List[Tuple[int, ...]]
    grad_dtype: int
    block_size: int
    step: int                      # t of the first measured step
    grad_recipe: Recipe
    weight_recipe: Recipe = field(default_factory=lambda: Recipe(NORMAL, 0.02))
    state_init: str = "prior_step"  # "prior_step" or "zero"
    n_steps: int = 1
    lr: float = LR
    beta1: float = BETA1
    beta2: float = BETA2
    eps: float = EPS
    weight_decay: float = WEIGHT_DECAY
    max_norm: float = MAX_NORM

    @property
    def numels(self) -> List[int]:
        return [math.prod(s) for s in self.shapes]

    @property
    def n_params(self) -> int:
        return sum(self.numels)

    def weights(self, k: int, offset: int = 0, n: Optional[int] = None, **kw) -> np.ndarray:
        n = self.numels[k] - offset if n is None else n
        return draw(F32, n, self.seed, STREAM_WEIGHTS, k, self.weight_recipe, offset, **kw)

    def grads(self, k: int, stream: int, offset: int = 0, n: Optional[int] = None,
              **kw) -> np.ndarray:
        n = self.numels[k] - offset if n is None else n
        return draw(self.grad_dtype, n, self.seed, stream, k, self.grad_recipe, offset, **kw)

    def prior_grads(self, k: int, offset: int = 0, n: Optional[int] = None, **kw) -> np.ndarray:
        return self.grads(k, STREAM_PRIOR_GRAD, offset, n, **kw)


def _t3_grads() -> Recipe:
    # "bf16, ~N(0, 1e-3) with heavy-tailed outliers (Student-t, df 3)": 1e-3 * t3.
    return Recipe(STUDENT_T3, 1e-3)


def tiny() -> Workload:
    """4 fp32 tensors, ~2.6M params, block 256, step 2, clipping active."""
    return Workload("tiny-4-tensors-fp32", 0, [(512, 1024), (1024, 1024), (2048, 512), (1024,)],
                    F32, 256, 2, Recipe(NORMAL, 1e-3, 0.01, OUTLIER_SCALE, 100.0))


def layer_3b() -> Workload:
    """One 3B-class decoder layer: 9 tensors, 77.1M params, bf16 grads, block 2048."""
    return Workload("3b-class-layer", 1, list(LAYER_3B), BF16, 2048, 2, _t3_grads())


def full_3b() -> Workload:
    """3B-class model: tied embedding + 36 layers, 325 tensors, 3.09B params."""
    return Workload("3b-class-full-model", 2, [EMBED_3B] + 36 * list(LAYER_3B), BF16, 2048, 2,
                    _t3_grads())


def streamed_27b(n_layers: int = 64) -> Workload:
    """27B-class decoder layers only (hidden 5120, FFN 17408, 40q/8kv heads of 128)."""
    return Workload("27b-class-streamed", 3, n_layers * list(LAYER_27B), BF16, 2048, 2,
                    _t3_grads())


def clip_stress() -> Workload:
    """3B-class shapes; base grads scaled so the base norm is ~1e3, 0.1% of the entries
    set to +-1e4 (bf16 rounds them to +-9984), 1 in 64 blocks all zero in every step;
    zero initial state, three steps from t = 1."""
    shapes = [EMBED_3B] + 36 * list(LAYER_3B)
    n = sum(math.prod(s) for s in shapes)
    return Workload("3b-class-clip-stress", 4, shapes, BF16, 2048, 1,
                    Recipe(NORMAL, 1e3 / math.sqrt(n), 1e-3, OUTLIER_SET, 1e4, 2048, 64),
                    state_init="zero", n_steps=3)


WORKLOADS = {0: tiny, 1: layer_3b, 2: full_3b, 3: streamed_27b, 4: clip_stress}
