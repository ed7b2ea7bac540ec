"""GPU parity of the selection modes beyond a single threshold: one threshold
per query head, Top-K and Top-Ratio (the selection-strategy ablation of
Sec. 4.5 / Table 6). The decisions are integer work on fp32 scores, so the
GPU's index lists must equal the oracle's run on the same fp32 scores exactly,
for every row; end to end against the oracle's fp64 scores, a differing block
must sit within the scoring error of the selection cut."""
import numpy as np
import pytest

import oracle
import workloads as W

from .helpers import (OUT_MAX_ABS, OUT_MEAN_ABS, TIE, assert_index_sets, compare_scores,
                      dev_bf16, host_f32)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2503_16428_amd as X  # noqa: E402


def gpu_scores(w, x, x2=None):
    """Scores of one layer; with x2, of the batch of two layers (x, x2)."""
    q, k = dev_bf16(x["q"]), dev_bf16(x["k"])
    if x2 is not None:
        q = torch.stack([q, dev_bf16(x2["q"])])
        k = torch.stack([k, dev_bf16(x2["k"])])
    dims = X.make_dims(q, k, w.causal)
    sc = X.xattn_score(q, k, w.causal, w.block, w.stride)
    torch.cuda.synchronize()
    return q, k, dims, sc


def rows_of(dims, NB):
    H = dims.heads
    return np.repeat(np.arange(H), NB), np.tile(np.arange(NB), H).astype(np.int32)


def assert_lists_equal(gi, gc, oi, oc):
    gi = gi.cpu().numpy().reshape(len(oc), -1)
    gc = gc.cpu().numpy().reshape(-1)
    assert np.array_equal(gc, oc), np.nonzero(gc != oc)[0][:5]
    for r in range(len(oc)):
        assert np.array_equal(gi[r, :gc[r]], oi[r, :oc[r]]), r


def oracle_mode(mode, s, rh, rb, param, hq, causal):
    if mode == "heads":
        return oracle.select_heads_rows(s, rh, rb, param, hq, causal)
    per_row = np.asarray(param)[rh % hq]
    if mode == "topk":
        return oracle.select_topk_rows(s, rb, per_row, causal)
    return oracle.select_ratio_rows(s, rb, per_row, causal)


def gpu_mode(mode, sc, dims, param):
    f = {"heads": X.xattn_select_heads, "topk": X.xattn_select_topk,
         "ratio": X.xattn_select_ratio}[mode]
    idx, cnt = f(sc, dims, param)
    torch.cuda.synchronize()
    return idx, cnt


CASES = [
    # (seq, hq, hkv, stride, causal, batch): several tiles, ragged NB (not a
    # multiple of 64), non-causal, batch 2
    (4096, 4, 2, 8, True, 1),
    (12800, 2, 1, 16, True, 1),
    (9216, 3, 3, 8, False, 1),
    (2048, 4, 2, 4, True, 2),
]
PARAMS = {
    "heads": lambda hq: np.linspace(0.55, 0.97, hq).astype(np.float32),
    "topk": lambda hq: (np.arange(hq) * 3 + 2).astype(np.int32),
    "ratio": lambda hq: np.linspace(0.05, 0.6, hq).astype(np.float32),
}


@pytest.mark.parametrize("mode", ["heads", "topk", "ratio"])
@pytest.mark.parametrize("seq,hq,hkv,S,causal,batch", CASES)
def test_mode_equals_oracle_on_gpu_scores(mode, seq, hq, hkv, S, causal, batch):
    w = W.small(f"sel_{mode}", seq, hq=hq, hkv=hkv, stride=S, tau=0.9, seed=seq + hq,
                causal=causal)
    print(f"{mode} seq={seq} hq={hq} S={S} causal={causal} batch={batch}", flush=True)
    x = W.generate(w)
    x2 = W.generate(w.with_(base_seed=w.base_seed + 1)) if batch == 2 else None
    q, k, dims, sc = gpu_scores(w, x, x2)
    NB = w.n_blocks
    param = PARAMS[mode](hq)
    gi, gc = gpu_mode(mode, sc, dims, param)
    rh, rb = rows_of(dims, NB)
    s = sc.cpu().numpy().reshape(-1, NB).astype(np.float64)
    oi, oc = oracle_mode(mode, s, rh, rb, param, hq, causal)
    assert_lists_equal(gi, gc, oi, oc)


def test_uniform_heads_equal_single_threshold_and_tau_one_heads_take_all():
    w = W.small("sel_uniform", 4096, hq=4, hkv=2, stride=8, tau=0.9, seed=3)
    x = W.generate(w)
    q, k, dims, sc = gpu_scores(w, x)
    i1, c1 = X.xattn_select(sc, dims, 0.9)
    i2, c2 = X.xattn_select_heads(sc, dims, [0.9] * 4)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)
    for r in range(c1.numel()):
        n = int(c1.view(-1)[r])
        assert torch.equal(i1.view(-1, w.n_blocks)[r, :n], i2.view(-1, w.n_blocks)[r, :n])
    _, c3 = X.xattn_select_heads(sc, dims, [0.9, 1.0, 0.5, 7.0])
    _, ck = X.xattn_select_topk(sc, dims, [1, 10**6, 1, 10**6])
    _, cr = X.xattn_select_ratio(sc, dims, [0.01, 1.0, 0.01, 3.0])
    torch.cuda.synchronize()
    cand = np.arange(1, w.n_blocks + 1)
    for c in (c3, ck, cr):
        c = c.cpu().numpy()
        assert np.array_equal(c[1], cand) and np.array_equal(c[3], cand)
    assert np.all(ck.cpu().numpy()[[0, 2]] == 1) and np.all(cr.cpu().numpy()[[0, 2]] == 1)


@pytest.mark.parametrize("mode", ["heads", "topk", "ratio"])
def test_full_size_128k_modes(mode):
    # 128K tokens, 32 query / 8 KV heads, S = 16: every row against the oracle
    # on the GPU's fp32 scores (exact), and end to end on sampled rows.
    w = W.WORKLOADS["c3"]
    print(f"full-size {w.name} mode={mode}", flush=True)
    x = W.generate(w, threads=16)
    q, k, dims, sc = gpu_scores(w, x)
    NB = w.n_blocks
    param = {"heads": np.linspace(0.7, 0.97, 32).astype(np.float32),
             "topk": np.full(32, 24, np.int32),
             "ratio": np.full(32, 0.04, np.float32)}[mode]
    gi, gc = gpu_mode(mode, sc, dims, param)
    rh, rb = rows_of(dims, NB)
    s = sc.cpu().numpy().reshape(-1, NB).astype(np.float64)
    oi, oc = oracle_mode(mode, s, rh, rb, param, 32, True)
    assert_lists_equal(gi, gc, oi, oc)

    # end to end: oracle scores (fp64) on sampled rows; differing blocks must
    # lie within the score tolerance of the cut
    heads = np.array([0, 13, 31], np.int32)
    blocks = np.array([0, 5, 400, 1022, 1023], np.int32)
    srh, srb = np.repeat(heads, len(blocks)), np.tile(blocks, len(heads))
    f = oracle.score_rows(x["q"], x["k"], w.block, w.stride, True, rows=(srh, srb))
    rep = compare_scores(s[srh * NB + srb], f)
    print(f"  scores {rep}", flush=True)
    assert rep["n_bad"] == 0
    ei, ec = oracle_mode(mode, f, srh, srb, param, 32, True)
    gi_h = gi.cpu().numpy().reshape(-1, NB)
    gc_h = gc.cpu().numpy().reshape(-1)
    rows_g = srh * NB + srb
    gi_s, gc_s = gi_h[rows_g], gc_h[rows_g]
    same = int(sum(set(gi_s[r, :gc_s[r]]) == set(ei[r, :ec[r]]) for r in range(len(srh))))
    if mode == "heads":
        # find_blocks: differing blocks explained by the margin or tie rule
        for hh in np.unique(srh):
            sel = np.nonzero(srh == hh)[0]
            assert_index_sets(gi_s[sel], gc_s[sel], ei[sel], ec[sel], f[sel], srb[sel],
                              float(param[hh]), True, tag=f"head {hh} ")
    else:
        # fixed size: the counts agree, and a differing block's oracle score
        # is within TIE of the cut (the k-th largest oracle score)
        n_tie = 0
        for r in range(len(srh)):
            assert gc_s[r] == ec[r], (r, gc_s[r], ec[r])
            g, e = set(gi_s[r, :gc_s[r]].tolist()), set(ei[r, :ec[r]].tolist())
            cut = min(f[r, j] for j in e)
            for j in g ^ e:
                assert abs(f[r, j] - cut) <= TIE, (r, j, f[r, j], cut)
            n_tie += g != e
        print(f"  {mode}: tie-explained rows {n_tie}", flush=True)
        assert n_tie <= 1 + 0.05 * len(srh)
    print(f"  {mode}: {same}/{len(srh)} sampled rows identical end to end", flush=True)
    assert same >= len(srh) // 2

    # attention over the mode's lists, against the oracle on the same lists
    v = dev_bf16(x["v"])
    o, _ = X.xattn_block_sparse_attn(q, k, v, gi, gc, True, w.block)
    torch.cuda.synchronize()
    pick = (np.array([13, 31], np.int32), np.array([400, 1023], np.int32))
    rows_idx = [int(h) * NB + int(b) for h, b in zip(*pick)]
    o_ref, _ = oracle.sparse_attn_rows(x["q"], x["k"], x["v"], w.block, gi_h[rows_idx],
                                       gc_h[rows_idx], True, rows=pick)
    og = host_f32(o).reshape(32, w.seq, 128)
    got = np.stack([og[h, b * 128:(b + 1) * 128] for h, b in zip(*pick)])
    err = np.abs(got - o_ref)
    print(f"  attention on {mode} lists: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= OUT_MAX_ABS and err.mean() <= OUT_MEAN_ABS
