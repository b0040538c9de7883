"""STRIDE scoring, early-stop and restart path on AMD Instinct MI355X (gfx950).

The computation lives in ``libstride.so`` (hand-written HIP kernels behind the C
ABI declared in ``include/stride.h``); this package is its Python binding.
"""
from .stride import (  # noqa: F401
    NEG_INF, STRIDE_BF16, STRIDE_F32, STRIDE_FLAG_BAD_DOMAIN, STRIDE_FLAG_BAD_OFFSETS,
    STRIDE_FLAG_EMPTY_TURN, STRIDE_FLAG_NONFINITE, STRIDE_FLAG_SPIN_LIMIT, STRIDE_FLAG_TOKEN_OOB,
    STRIDE_MAX_DOMAINS, STRIDE_UNIT_TOKEN, STRIDE_UNIT_TURN, Layout, Path, Records, StrideDataError,
    StrideError, flag_names,
    library,
    stride_fused_workspace_size, stride_opd_grad, stride_probe_copy, stride_probe_read,
    stride_probe_read_flat, stride_restart_turn,
    stride_score, stride_score_fused, stride_stop, stride_stop_noalloc, stride_stop_step,
    stride_workspace_size)
