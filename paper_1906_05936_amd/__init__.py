"""Layered SGD (Yu et al., arXiv 1906.05936) gradient aggregation and update on
AMD Instinct MI355X.

The computation lives in liblsgd.so (hand-written HIP for gfx950) behind the C
ABI of include/lsgd.h; this package is its Python binding. Importing it fails
loudly if the library has not been built: there is no fallback path.
"""
from ._lib import (BF16, COPY_OUT_AUTO, COPY_OUT_FUSED, COPY_OUT_SEPARATE, F32, LIB_PATH,
                   MAX_REPLICAS, MAX_WORKERS, REDUCE_LITERAL, REDUCE_MEAN_OF_MEANS, XCD_CHUNK_AUTO,
                   LrSchedule, LsgdError, Plan, copy_out, get_copy_out_mode, get_launch_shape, global_mean,
                   group_mean, lr_at, lr_schedule, lr_schedule_step, set_copy_out_mode,
                   set_launch_shape, sgd_step, step, stream_copy, set_step_replicas, get_step_replicas)

__all__ = ["BF16", "COPY_OUT_AUTO", "COPY_OUT_FUSED", "COPY_OUT_SEPARATE", "F32", "LIB_PATH", "MAX_REPLICAS", "MAX_WORKERS", "REDUCE_LITERAL",
           "REDUCE_MEAN_OF_MEANS", "XCD_CHUNK_AUTO", "LrSchedule", "LsgdError", "Plan",
           "copy_out", "get_copy_out_mode", "get_launch_shape", "global_mean", "group_mean", "lr_at", "lr_schedule",
           "lr_schedule_step", "set_copy_out_mode", "set_launch_shape", "sgd_step", "step", "stream_copy",
           "set_step_replicas", "get_step_replicas"]
