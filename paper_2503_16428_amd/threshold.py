"""Minimum-threshold prediction driver (XAttention Sec. 3.3) on one layer.

Performance proxy: each query head's output error against the dense output,
err = |o - o_dense|^2 / |o_dense|^2 averaged over the batch
(xattn_head_error_mean), measured after 0 .. max_adjust threshold reductions
of 10 % from tau0 (xattn_threshold_levels; one xattn_forward per level, every
head at the same threshold: a head's output depends on its own threshold
only). xattn_threshold_predict then spends exactly `adjustments` reductions
where they add the least error and returns the per-head thresholds. This
module only sequences those library calls and moves the table to the host.
"""
from __future__ import annotations

import torch

from . import binding as B


def predict_thresholds(q, k, v, adjustments: int, tau0: float = 0.9, max_adjust: int = 1,
                       causal: bool = True, block: int = B.BLOCK, stride: int = 8):
    """Per-query-head thresholds for one layer. Returns a dict with tau_h
    (float32 [hq]), adjust (int32 [hq]), err ([hq][max_adjust + 1], the error
    table, batch elements averaged), levels (the thresholds of the table's
    columns) and total_err (the least total error)."""
    d = B.make_dims(q, k, causal)
    levels = B.threshold_levels(tau0, max_adjust)
    o_ref, _ = B.xattn_dense_attn(q, k, v, causal, want_lse=False)
    ws = torch.empty(B.forward_workspace_size(d, block, stride), dtype=torch.uint8,
                     device=q.device)
    o = torch.empty_like(q)
    table = torch.empty((d.hq, max_adjust + 1), dtype=torch.float64, device=q.device)
    for a in range(max_adjust + 1):
        B.xattn_forward(q, k, v, causal, block, stride, float(levels[a]), o=o, workspace=ws)
        table[:, a] = B.head_error_mean(o, o_ref, causal)
    err = table.cpu().numpy()
    adjust, tau_h, total = B.threshold_predict(err, adjustments, tau0)
    return {"tau_h": tau_h, "adjust": adjust, "err": err, "levels": levels,
            "total_err": total}
