"""Shared helpers of the GPU parity tests (tolerances, index comparison)."""
from __future__ import annotations

import math

import numpy as np

import workloads as W

# Output bar for attention (bf16 inputs, fp32 accumulation, bf16 output).
OUT_MAX_ABS = 2e-2
OUT_MEAN_ABS = 5e-3
# Index sets may differ only for blocks whose cumulative-mass margin to tau
# is below this, or whose score is within the scoring error bound of the cut.
MARGIN = 1e-3
U32 = 2.0 ** -24   # fp32 unit roundoff


def dev_bf16(u16: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).cuda()


def host_f32(t) -> np.ndarray:
    import torch
    if t.dtype == torch.bfloat16:
        u = t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        return W.bf16_bits_to_f32(u)
    return t.float().cpu().numpy()


def logit_error_bound(q, k, S, rows_h, rows_b, hq_per_kv, B=128, qsub=None):
    """Rigorous bound on |z_gpu - z_exact| for the reduced logits of the given
    rows: the GPU sums n = S*d exact bf16 products in fp32 (any order), so
    |error| <= gamma_n * sum |q_e k_e| with gamma_n = n u / (1 - n u), then
    scales by 1/(S sqrt d) (one more rounding). qsub: the sub-row pairing
    (default the antidiagonal, S-1-t)."""
    D = q.shape[-1]
    n = S * D
    gamma = n * U32 / (1 - n * U32)
    worst = 0.0
    nr = B // S
    pair = np.arange(S)[::-1] if qsub is None else np.asarray(qsub)
    for h, b in zip(rows_h, rows_b):
        qa = np.abs(W.bf16_bits_to_f32(q[h]))
        ka = np.abs(W.bf16_bits_to_f32(k[h // hq_per_kv]))
        R0 = b * nr
        Qr = np.stack([qa[(R0 + r) * S + pair].reshape(-1) for r in range(nr)])
        Kt = ka.reshape(-1, n)
        worst = max(worst, float((Qr @ Kt.T).max()))
    return (gamma * worst + U32 * 4 * worst / n) / (S * math.sqrt(D))


def score_tolerance(dz: float):
    """|s_gpu - s_exact| <= rtol * s_exact + atol: a logit error dz moves every
    softmax term by a factor within exp(+-2 dz); fp32 exp/sum/normalise add a
    few hundred ulps relative, and 1e-7 absolute covers values near the fp32
    resolution of a row that sums to 1."""
    rtol = math.expm1(2 * dz) + 512 * U32
    return rtol, 1e-7


def compare_scores(got, want, dz):
    rtol, atol = score_tolerance(dz)
    err = np.abs(got.astype(np.float64) - want)
    bad = err > rtol * want + atol
    return {"max_abs": float(err.max()), "rtol": rtol, "atol": atol, "n_bad": int(bad.sum()),
            "max_rel_sig": float((err / np.maximum(want, 1e-6)).max())}


def compare_index_sets(gpu_idx, gpu_cnt, ora_idx, ora_cnt, ora_scores, row_b, tau, causal,
                       score_rtol):
    """Per row: equal sets, or every differing block explained by the margin
    rule (oracle cumulative mass before it within MARGIN of tau) or the tie
    rule (its oracle score within the scoring error bound of the cut score).
    Returns (n_equal, n_margin_rows, n_tie_rows, unexplained list)."""
    n_eq = n_margin = n_tie = 0
    bad = []
    for r in range(len(row_b)):
        g = set(gpu_idx[r, :gpu_cnt[r]].tolist())
        o = set(ora_idx[r, :ora_cnt[r]].tolist())
        if g == o:
            n_eq += 1
            continue
        m = row_b[r] + 1 if causal else ora_scores.shape[1]
        s = ora_scores[r, :m]
        T = s.sum()
        order = sorted(range(m), key=lambda j: (-s[j], j))
        pos = {j: p for p, j in enumerate(order)}
        csum = np.concatenate([[0.0], np.cumsum([s[j] for j in order])]) / T
        cut = s[order[ora_cnt[r] - 1]]
        kinds = set()
        for j in g ^ o:
            if abs(csum[pos[j]] - tau) < MARGIN or abs(csum[pos[j] + 1] - tau) < MARGIN:
                kinds.add("margin")
            elif abs(s[j] - cut) <= score_rtol * max(s[j], cut) + 1e-7:
                kinds.add("tie")
            else:
                kinds.add("bad")
        if "bad" in kinds:
            bad.append((r, sorted(g - o), sorted(o - g)))
        elif "margin" in kinds:
            n_margin += 1
        else:
            n_tie += 1
    return n_eq, n_margin, n_tie, bad
