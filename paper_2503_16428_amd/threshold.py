"""Minimum-threshold prediction driver (XAttention Sec. 3.3) on one layer.

Performance proxy: minus each query head's output error against the dense
output, err = |o - o_dense|^2 / |o_dense|^2 (xattn_head_error), measured
after 0 .. max_adjust threshold reductions of 10 % from tau0 (one
xattn_forward per level, every head at the same threshold: a head's output
depends on its own threshold only). The dynamic program (xattn_threshold_dp)
then spends exactly `adjustments` reductions where they cost the least.
"""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B


def adjusted_thresholds(tau0: float, adjust) -> np.ndarray:
    """t_h = tau0 * 0.9^a_h as float32 (the threshold the selection receives)."""
    return np.array([np.float32(tau0 * 0.9 ** int(a)) for a in adjust], dtype=np.float32)


def predict_thresholds(q, k, v, adjustments: int, tau0: float = 0.9, max_adjust: int = 1,
                       causal: bool = True, block: int = B.BLOCK, stride: int = 8):
    """Per-query-head thresholds for one layer. Returns a dict with tau_h
    (float32 [hq]), adjust (int32 [hq]), err ([hq][max_adjust + 1], the proxy
    table, batch elements averaged), best (the table optimum)."""
    d = B.make_dims(q, k, causal)
    o_ref, _ = B.xattn_dense_attn(q, k, v, causal, want_lse=False)
    ws = torch.empty(B.forward_workspace_size(d, block, stride), dtype=torch.uint8,
                     device=q.device)
    o = torch.empty_like(q)
    errs = []
    for a in range(max_adjust + 1):
        tau = float(np.float32(tau0 * 0.9 ** a))
        B.xattn_forward(q, k, v, causal, block, stride, tau, o=o, workspace=ws)
        e = B.head_error(o, o_ref, causal).cpu().numpy().reshape(d.batch, d.hq)
        errs.append(e.mean(axis=0))
    err = np.stack(errs, axis=1)                     # [hq][max_adjust + 1]
    adjust, best = B.threshold_dp(-err, adjustments)
    return {"tau_h": adjusted_thresholds(tau0, adjust), "adjust": adjust, "err": err,
            "best": best}
