"""GPU parity of the scoring-pattern variants (the pattern ablation, Sec. 4.5,
Table 4): diagonal and random sub-block pairings against the oracle, the
antidiagonal pairing bitwise equal to xattn_score, and on the 128K layer the
density and the covered fraction of the exact attention mass per pattern
(reported only: the accuracy comparison of the ablation needs real models)."""
import numpy as np
import pytest

import oracle
import workloads as W

from .helpers import assert_index_sets, compare_scores, dev_bf16, logit_error_bound

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2503_16428_amd as X  # noqa: E402

CASES = [
    # (seq, hq, hkv, stride, causal): several 256-row tiles, a ragged reduced
    # length (4736 / 4 = 1184 rows), non-causal, the largest stride
    (4096, 4, 2, 8, True),
    (4736, 2, 1, 4, True),
    (6144, 2, 1, 16, False),
    (8192, 2, 2, 64, True),
]


@pytest.mark.parametrize("pattern", ["diagonal", "random"])
@pytest.mark.parametrize("seq,hq,hkv,S,causal", CASES)
def test_pattern_scores_match_oracle(pattern, seq, hq, hkv, S, causal):
    w = W.small(f"pat_{pattern}", seq, hq=hq, hkv=hkv, stride=S, causal=causal, seed=seq + S)
    print(f"{pattern} seq={seq} hq={hq} S={S} causal={causal}", flush=True)
    x = W.generate(w)
    qsub = W.sub_row_pairing(pattern, S, seed=S)
    q, k = dev_bf16(x["q"]), dev_bf16(x["k"])
    sc = X.xattn_score_pattern(q, k, causal, w.block, S, qsub)
    torch.cuda.synchronize()
    rh, rb = oracle.all_rows(hq, w.n_blocks)
    want = oracle.score_pattern_rows(x["q"], x["k"], w.block, S, qsub, causal, rows=(rh, rb))
    dz = logit_error_bound(x["q"], x["k"], S, rh, rb, hq // hkv, w.block, qsub=qsub)
    rep = compare_scores(sc.cpu().numpy().reshape(-1, w.n_blocks), want, dz)
    print(f"  scores {rep}", flush=True)
    assert rep["n_bad"] == 0


def test_antidiagonal_pairing_is_xattn_score():
    w = W.small("pat_anti", 4096, hq=4, hkv=2, stride=8, seed=5)
    x = W.generate(w)
    q, k = dev_bf16(x["q"]), dev_bf16(x["k"])
    a = X.xattn_score(q, k, True, 128, 8)
    b = X.xattn_score_pattern(q, k, True, 128, 8, W.sub_row_pairing("antidiagonal", 8))
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_patterns_on_the_128k_layer():
    # 128K tokens, 32 q / 8 kv heads, S = 16, tau = 0.9: sampled rows against
    # the oracle per pattern; density of the whole layer and the exact
    # attention mass the selected blocks cover on the sampled rows.
    w = W.WORKLOADS["c3"]
    x = W.generate(w, threads=16)
    q, k = dev_bf16(x["q"]), dev_bf16(x["k"])
    dims = X.make_dims(q, k, True)
    NB = w.n_blocks
    rh = np.array([0, 0, 13, 13, 31, 31], np.int32)
    rb = np.array([300, 1023, 511, 1000, 64, 777], np.int32)
    true_mass, _ = oracle.block_mass_rows(x["q"], x["k"], w.block, w.stride, True,
                                          rows=(rh, rb))
    report = {}
    for pattern in ("antidiagonal", "diagonal", "random"):
        qsub = W.sub_row_pairing(pattern, w.stride, seed=1)
        sc = X.xattn_score_pattern(q, k, True, w.block, w.stride, qsub)
        idx, cnt = X.xattn_select(sc, dims, w.tau)
        torch.cuda.synchronize()
        want = oracle.score_pattern_rows(x["q"], x["k"], w.block, w.stride, qsub, True,
                                         rows=(rh, rb))
        dz = logit_error_bound(x["q"], x["k"], w.stride, rh, rb, 4, w.block, qsub=qsub)
        got = sc.cpu().numpy().reshape(-1, NB)[rh * NB + rb]
        rep = compare_scores(got, want, dz)
        assert rep["n_bad"] == 0, (pattern, rep)
        gi = idx.cpu().numpy().reshape(-1, NB)[rh * NB + rb]
        gc = cnt.cpu().numpy().reshape(-1)[rh * NB + rb]
        oi, oc = oracle.select_rows(want, rb, w.tau)
        assert_index_sets(gi, gc, oi, oc, want, rb, w.tau, True, tag=f"{pattern} ")
        cov = np.mean([true_mass[r, gi[r, :gc[r]]].sum() for r in range(len(rh))])
        c_all = cnt.cpu().numpy().astype(np.int64)
        dens = c_all.sum() / (np.arange(1, NB + 1).sum() * dims.heads)
        report[pattern] = (float(dens), float(cov))
        print(f"  {pattern:12s} density {dens:.4f}  covered exact mass {cov:.4f}", flush=True)
    assert all(0.0 < d <= 1.0 and 0.0 < c <= 1.0 + 1e-9 for d, c in report.values())
