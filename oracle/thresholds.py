"""Minimum-threshold prediction, oracle side (XAttention Sec. 3.3) -- TEST
INFRASTRUCTURE, never used by the GPU library.

The paper's table D[h][m] holds the best performance reachable with exactly m
threshold adjustments spread over the first h heads; each adjustment lowers
one head's threshold by 10 % (t <- 0.9 t), and the recurrence takes, for head
h, either no adjustment (D[h-1][m]) or one more relative to D[h-1][m-1]. The
performance here is a per-head proxy (the build has no benchmark models):
perf[h][a] is the performance contribution of head h after a adjustments,
and the performance of a configuration is the sum over heads (heads select
and attend independently, so an output-error proxy is exactly additive).

Readings (listed with reasons in the design notes): a head takes at most
A_max adjustments (A_max = 1 is the printed two-way recurrence); on equal
performance the option with fewer adjustments of the current head wins;
the result is the configuration of D[H][M].
"""
from __future__ import annotations

import math

import numpy as np


def threshold_dp(perf, M: int):
    """perf: [H][A+1] floats. Returns (adjust[H] ints summing to M, best value).
    Plain loops in the order of the recurrence: heads in index order, for
    each m the options a = 0 .. min(m, A) tried in increasing a, a strictly
    larger value replacing the current one."""
    perf = [[float(x) for x in row] for row in perf]
    H = len(perf)
    A = len(perf[0]) - 1
    if not (0 <= M <= H * A):
        raise ValueError("M must lie in [0, H * A]")
    NEG = -math.inf
    # D[h][m] for h = 0 .. H (h = 0: no heads yet)
    D = [[NEG] * (M + 1) for _ in range(H + 1)]
    take = [[0] * (M + 1) for _ in range(H + 1)]
    D[0][0] = 0.0
    for h in range(1, H + 1):
        row = perf[h - 1]
        for m in range(M + 1):
            best, arg = NEG, 0
            for a in range(0, min(m, A) + 1):
                prev = D[h - 1][m - a]
                if prev == NEG:
                    continue
                val = prev + row[a]
                if val > best:
                    best, arg = val, a
            D[h][m] = best
            take[h][m] = arg
    adjust = [0] * H
    m = M
    for h in range(H, 0, -1):
        adjust[h - 1] = take[h][m]
        m -= take[h][m]
    assert m == 0
    return adjust, D[H][M]


def thresholds_from_adjustments(tau0, adjust):
    """t_h = tau0 * 0.9^a_h (one 10 % reduction per adjustment), as float32."""
    return np.array([np.float32(tau0 * 0.9 ** a) for a in adjust], dtype=np.float32)


def head_errors(o, o_ref):
    """Relative squared error per head: sum (o - o_ref)^2 / sum o_ref^2 over
    the head's [L][d] outputs, in fp64. o, o_ref: float arrays [H][L][d]."""
    o = np.asarray(o, dtype=np.float64)
    r = np.asarray(o_ref, dtype=np.float64)
    num = ((o - r) ** 2).reshape(o.shape[0], -1).sum(axis=1)
    den = (r ** 2).reshape(r.shape[0], -1).sum(axis=1)
    return num / den
