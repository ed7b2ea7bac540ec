"""MI355X (gfx950) XAttention prefill path: antidiagonal block scoring,
threshold block selection and block-sparse attention as HIP kernels behind a
C ABI (include/xattn.h). This package holds the kernels' sources (csrc/), the
in-tree build (build.py), a thin ctypes binding (binding.py) and the
minimum-threshold prediction driver (threshold.py)."""
from .binding import (  # noqa: F401
    BLOCK, Dims, XAttnError, forward_layout, forward_workspace_size, head_error,
    head_error_mean, lib, lib_path, make_dims, score_workspace_size, threshold_dp,
    threshold_levels, threshold_predict, version,
    xattn_block_sparse_attn, xattn_dense_attn, xattn_forward, xattn_forward_noalloc,
    xattn_forward_scheduled,
    xattn_score, xattn_score_pattern, xattn_select, xattn_select_heads, xattn_select_ratio,
    xattn_select_topk,
)
from .threshold import predict_thresholds  # noqa: F401,E402
