"""MI355X-native Hybrid 8-bit AdamW step with fast gradient clipping.

The hot path (LazyTrain, Sec. 3.5) runs in hand-written gfx950 HIP kernels
behind the C ABI of ``include/lazytrain.h``; this package is its Python
binding.  Importing it does not load the library; the first call does, and
raises if the library has not been built.
"""
from .lazytrain import (  # noqa: F401
    LT_OK, LT_ERR_INVALID_ARG, LT_ERR_ALIGNMENT, LT_ERR_HIP, LT_ERR_WORKSPACE,
    LT_DTYPE_BF16, LT_DTYPE_F32, LT_MAP_DYNAMIC, LT_MAP_LINEAR, LT_STATUS_BAD_WORKSPACE,
    LT_STATUS_NONFINITE, LT_STATUS_OK, Hybrid8bitAdamW, LazyTrainError, NonFiniteAbort, lib,
    lt_clip_coef, lt_grad_sqnorm, lt_grad_sqnorm_workspace_bytes, lt_hybrid8bit_adamw_step,
    lt_read_status, lt_set_max_workgroups, lt_step_workspace_bytes,
    lt_streamed_hybrid8bit_adamw_step, lt_streamed_workspace_bytes, lt_adamw_fp32_step,
    lt_adamw_fp32_workspace_bytes, lt_select_8bit_slice, lt_grad_chunk_count,
    lt_grad_sqnorm_partials, lt_grad_sqnorm_finish, lt_workspace_release, lt_grad_sqnorm_noalloc,
    lt_step_state_bytes, lt_step_table, lt_step_state_init, lt_step_state_advance,
    GradNormAccumulator,
    StreamedHybrid8bitAdamW)
