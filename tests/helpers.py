"""Shared helpers of the GPU parity tests (tolerances, index comparison)."""
from __future__ import annotations

import math

import numpy as np

import oracle
import workloads as W

# Output bar for attention (bf16 inputs, fp32 accumulation, bf16 output).
OUT_MAX_ABS = 2e-2
OUT_MEAN_ABS = 5e-3
# Scores (the rows of Alg. 1's block scores, each summing to 1): asserted
# |s_gpu - s| <= SCORE_RTOL * max(s, SCORE_FLOOR). Measured errors stay near
# 3e-5 relative; the rigorous worst-case bound (logit_error_bound) is far
# looser and is only reported.
SCORE_RTOL = 1e-4
SCORE_FLOOR = 1e-6
# Index sets (find_blocks of Sec. 3.2) may differ only in blocks whose
# oracle cumulative mass before or after them lies within MARGIN of tau, or,
# at equal counts, in blocks whose oracle score is within TIE of the cut
# score (the last oracle-selected block).
MARGIN = 1e-3
TIE = 1e-6
# At most this fraction of a test's rows (plus one) may be explained that way.
MAX_EXPLAINED_FRAC = 0.05
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
    (default the antidiagonal, S-1-t). Reported next to the asserted bound."""
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
    """The rigorous relative bound implied by a logit error dz: every softmax
    term moves by a factor within exp(+-2 dz); fp32 exp/sum/normalise add a
    few hundred ulps. Reported only (it is 100-1000x the asserted bound)."""
    return math.expm1(2 * dz) + 512 * U32, 1e-7


def compare_scores(got, want, dz=None):
    """Asserted bound: |got - want| <= SCORE_RTOL * max(want, SCORE_FLOOR)."""
    got = np.asarray(got, np.float64)
    err = np.abs(got - want)
    bound = SCORE_RTOL * np.maximum(want, SCORE_FLOOR)
    rep = {"max_abs": float(err.max()),
           "max_rel": float((err / np.maximum(want, SCORE_FLOOR)).max()),
           "n_bad": int((err > bound).sum()), "rtol": SCORE_RTOL, "floor": SCORE_FLOOR}
    if dz is not None:
        rep["rigorous_rtol"] = score_tolerance(dz)[0]
    return rep


def compare_index_sets(gpu_idx, gpu_cnt, ora_idx, ora_cnt, ora_scores, row_b, tau, causal):
    """Per row: equal sets, or every differing block explained by the margin
    rule (oracle cumulative mass before or after it within MARGIN of tau, as a
    fraction of the row total) or, when the counts agree, the tie rule (its
    oracle score within TIE of the cut score). Returns (n_equal,
    n_margin_rows, n_tie_rows, unexplained list)."""
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
            elif len(g) == len(o) and abs(s[j] - cut) <= TIE:
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


def assert_index_sets(gpu_idx, gpu_cnt, ora_idx, ora_cnt, ora_scores, row_b, tau, causal,
                      tag=""):
    """compare_index_sets, printed, with no unexplained row and the explained
    rows capped. Returns the boolean mask of rows with identical lists."""
    n_eq, n_m, n_t, bad = compare_index_sets(gpu_idx, gpu_cnt, ora_idx, ora_cnt, ora_scores,
                                             row_b, tau, causal)
    n = len(row_b)
    print(f"  {tag}index rows: {n} total, equal={n_eq} margin={n_m} tie={n_t} "
          f"unexplained={len(bad)}", flush=True)
    assert not bad, bad[:3]
    assert n_m + n_t <= 1 + MAX_EXPLAINED_FRAC * n, (n_m, n_t, n)
    return np.array([np.array_equal(gpu_idx[r, :gpu_cnt[r]], ora_idx[r, :ora_cnt[r]])
                     for r in range(n)])


def assert_attention_on_lists(x, B, idx, cnt, causal, rows, o_gpu, tag=""):
    """The oracle's attention over the GPU's own index lists (so the check
    isolates the attention kernel, whatever the selection did), on every
    given row: max-abs and mean-abs bars. o_gpu: float [rows][B][d]."""
    o_ref, _ = oracle.sparse_attn_rows(x["q"], x["k"], x["v"], B, idx, cnt, causal, rows=rows)
    err = np.abs(o_gpu.astype(np.float64) - o_ref)
    per_row = err.reshape(len(err), -1).max(axis=1)
    r = int(per_row.argmax())
    print(f"  {tag}attention on the GPU lists, {len(err)} rows: max_abs={err.max():.3e} "
          f"mean_abs={err.mean():.3e} (worst row head {rows[0][r]} block {rows[1][r]}, "
          f"max |o| there {np.abs(o_ref[r]).max():.2f})", flush=True)
    assert err.max() <= OUT_MAX_ABS and err.mean() <= OUT_MEAN_ABS
    return err
