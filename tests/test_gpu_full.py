"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (score -> select -> sparse attention with caller-owned
buffers), checked against the fp64 oracle on sampled (head, query block)
rows, plus properties that hold at any size, and edge cases (single block,
maximum length, degenerate ties, extreme thresholds)."""
import numpy as np
import pytest

import oracle
import workloads as W

from .helpers import (OUT_MAX_ABS, OUT_MEAN_ABS, assert_attention_on_lists,
                      assert_index_sets, compare_scores, dev_bf16, host_f32, logit_error_bound)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2503_16428_amd as X  # noqa: E402


def run_path(w, x):
    """The benchmark's step: xattn_score / xattn_select / xattn_block_sparse_attn."""
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    dims = X.make_dims(q, k, w.causal)
    NB = w.n_blocks
    scores = torch.empty((dims.heads, NB, NB), dtype=torch.float32, device="cuda")
    idx = torch.empty((dims.heads, NB, NB), dtype=torch.int32, device="cuda")
    cnt = torch.empty((dims.heads, NB), dtype=torch.int32, device="cuda")
    ws = torch.empty(X.score_workspace_size(dims, w.block, w.stride), dtype=torch.uint8,
                     device="cuda")
    X.xattn_score(q, k, w.causal, w.block, w.stride, scores=scores, workspace=ws)
    X.xattn_select(scores, dims, w.tau, w.block, idx=idx, cnt=cnt)
    o, lse = X.xattn_block_sparse_attn(q, k, v, idx, cnt, w.causal, w.block)
    torch.cuda.synchronize()
    return dict(q=q, k=k, v=v, dims=dims, scores=scores, idx=idx, cnt=cnt, o=o, lse=lse)


def sample_rows(w, n_heads=3):
    H, NB = w.hq * w.batch, w.n_blocks
    heads = sorted({0, H // 2, H - 1})[:n_heads]
    blocks = sorted({0, 1, NB // 3, NB - 2, NB - 1})
    rh = np.array([h for h in heads for _ in blocks], np.int32)
    rb = np.array([b for _ in heads for b in blocks], np.int32)
    return rh, rb


def worst_output_rows(w, g, n):
    """The n (head, query block) rows holding the largest |o| of the GPU
    output: where the bf16 rounding of the output and of P costs the most."""
    NB = w.n_blocks
    m = g["o"].view(-1, NB, w.block * w.head_dim).abs().amax(-1).float().view(-1)
    top = torch.topk(m, n).indices.cpu().numpy()
    return (top // NB).astype(np.int32), (top % NB).astype(np.int32)


def with_rows(rows, extra):
    seen = set(zip(*rows))
    add = [(h, b) for h, b in zip(*extra) if (h, b) not in seen]
    if not add:
        return rows
    rh = np.concatenate([rows[0], np.array([h for h, _ in add], np.int32)])
    rb = np.concatenate([rows[1], np.array([b for _, b in add], np.int32)])
    return rh, rb


def check_sampled(w, x, g, rows):
    """Scores, index lists and outputs of the given rows against the oracle:
    scores to the asserted bound; index lists exact up to margin / tie
    explained rows (reported, capped); the attention of every row against the
    oracle run on the GPU's own lists; end to end against the oracle's whole
    pipeline on the rows whose lists agree (the others are counted)."""
    rh, rb = rows
    NB = w.n_blocks
    f = oracle.forward_rows(x["q"], x["k"], x["v"], w.block, w.stride, w.tau, w.causal,
                            rows=rows)
    sc = g["scores"].cpu().numpy().reshape(-1, NB, NB)[rh, rb]
    dz = logit_error_bound(x["q"], x["k"], w.stride, rh[:4], rb[:4], w.hq // w.hkv, w.block)
    rep = compare_scores(sc, f["scores"], dz)
    print(f"  {w.name} S={w.stride} tau={w.tau}: scores {rep}", flush=True)
    assert rep["n_bad"] == 0
    gi = g["idx"].cpu().numpy().reshape(-1, NB, NB)[rh, rb]
    gc = g["cnt"].cpu().numpy().reshape(-1, NB)[rh, rb]
    same = assert_index_sets(gi, gc, f["idx"], f["cnt"], f["scores"], rb, w.tau, w.causal)
    o = host_f32(g["o"]).reshape(-1, w.seq, w.head_dim)
    og = np.stack([o[h, b * w.block:(b + 1) * w.block] for h, b in zip(rh, rb)])
    assert_attention_on_lists(x, w.block, gi, gc, w.causal, rows, og)
    err = np.abs(og[same].astype(np.float64) - f["o"][same])
    print(f"  end to end on {same.sum()}/{len(rh)} rows with the oracle's lists "
          f"({len(rh) - same.sum()} rows with explained list differences): "
          f"max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
    assert err.max() <= OUT_MAX_ABS and err.mean() <= OUT_MEAN_ABS


def check_properties(w, g):
    NB = w.n_blocks
    sc = g["scores"]
    rs = sc.sum(-1)
    assert torch.allclose(rs, torch.ones_like(rs), atol=1e-4), float((rs - 1).abs().max())
    cnt = g["cnt"].cpu().numpy().reshape(-1, NB)
    cand = (np.arange(NB) + 1) if w.causal else np.full(NB, NB)
    assert np.all(cnt >= 1) and np.all(cnt <= cand[None, :])
    idx = g["idx"].cpu().numpy().reshape(-1, NB, NB)
    for h in range(0, idx.shape[0], max(1, idx.shape[0] // 4)):
        for b in range(0, NB, max(1, NB // 16)):
            sel = idx[h, b, :cnt[h, b]]
            assert np.all(np.diff(sel) > 0) and sel[0] >= 0 and sel[-1] < cand[b]
    assert torch.isfinite(g["lse"]).all()


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c5"])
def test_full_size_workload(name):
    w = W.WORKLOADS[name]
    print(f"full-size {w.name}", flush=True)
    x = W.generate(w, threads=16)
    g = run_path(w, x)
    check_properties(w, g)
    if name == "c1":
        rows = oracle.all_rows(w.hq, w.n_blocks)
    else:
        # position-chosen rows plus the rows holding the largest outputs
        rows = with_rows(sample_rows(w), worst_output_rows(w, g, 6))
    check_sampled(w, x, g, rows)
    # repeated launches at full size are bitwise identical (no LDS races)
    g2 = run_path(w, x)
    assert torch.equal(g["scores"], g2["scores"]) and torch.equal(g["cnt"], g2["cnt"])
    assert torch.equal(g["o"].view(torch.int16), g2["o"].view(torch.int16))
    assert torch.equal(g["lse"], g2["lse"])


@pytest.mark.parametrize("tau,S", W.C4_SWEEP)
def test_c4_sweep_point(tau, S):
    w = W.WORKLOADS["c4"].with_(tau=tau, stride=S)
    print(f"c4 sweep tau={tau} S={S}", flush=True)
    x = _c4_inputs()
    g = run_path(w, x)
    check_properties(w, g)
    dens = g["cnt"].sum().item() / (np.arange(1, w.n_blocks + 1).sum() * w.hq)
    print(f"  density {dens:.4f}", flush=True)
    if tau >= 1.0:
        # dense-equivalence at full size: every causal block, bitwise equal to dense mode
        assert dens == 1.0
        od, ld = X.xattn_dense_attn(g["q"], g["k"], g["v"], True)
        torch.cuda.synchronize()
        assert torch.equal(od.view(torch.int16), g["o"].view(torch.int16))
        assert torch.equal(ld, g["lse"])
        rows = (np.array([3, 17], np.int32), np.array([0, w.n_blocks - 1], np.int32))
        o_ref, _ = oracle.dense_attn_rows(x["q"], x["k"], x["v"], 128, True, rows=rows)
        o = host_f32(g["o"]).reshape(w.hq, w.seq, 128)
        og = np.stack([o[h, b * 128:(b + 1) * 128] for h, b in zip(*rows)])
        err = np.abs(og - o_ref)
        print(f"  dense rows vs oracle: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
        assert err.max() <= OUT_MAX_ABS and err.mean() <= OUT_MEAN_ABS
    else:
        rh, rb = sample_rows(w, n_heads=2)
        check_sampled(w, x, g, with_rows((rh[::2], rb[::2]), worst_output_rows(w, g, 2)))


_C4 = {}


def _c4_inputs():
    if "x" not in _C4:
        _C4["x"] = W.generate(W.WORKLOADS["c4"], threads=16)
    return _C4["x"]


def test_single_block_sequence():
    w = W.small("one_block", 128, hq=2, hkv=1, stride=16, tau=0.5, seed=9)
    x = W.generate(w)
    g = run_path(w, x)
    assert g["cnt"].cpu().numpy().tolist() == [[1], [1]]
    assert torch.allclose(g["scores"], torch.ones_like(g["scores"]))
    check_sampled(w, x, g, oracle.all_rows(2, 1))


def test_maximum_length_262144():
    w = W.small("max_len", 262144, hq=1, hkv=1, stride=16, tau=0.9, seed=31)
    print("max length 262144 (2048 blocks)", flush=True)
    x = W.generate(w, threads=16)
    g = run_path(w, x)
    check_properties(w, g)
    rows = (np.array([0, 0, 0], np.int32), np.array([0, 1024, 2047], np.int32))
    check_sampled(w, x, g, rows)
    # the forward pass at 2048 blocks per row: bitwise the separate calls
    o, lse, views = X.xattn_forward(g["q"], g["k"], g["v"], True, w.block, w.stride, w.tau,
                                    want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(views["scores"], g["scores"]) and torch.equal(views["cnt"], g["cnt"])
    assert torch.equal(o.view(torch.int16), g["o"].view(torch.int16))
    assert torch.equal(lse, g["lse"])


def test_zero_queries_tie_everywhere():
    # Q = 0: uniform reduced softmax, block masses by closed form; selection
    # breaks the many exact ties toward low block indices.
    w = W.small("zero_q", 2048, hq=2, hkv=1, stride=8, tau=0.5, seed=4)
    x = W.generate(w)
    x["q"] = np.zeros_like(x["q"])
    g = run_path(w, x)
    rows = oracle.all_rows(2, w.n_blocks)
    check_sampled(w, x, g, rows)


@pytest.mark.parametrize("tau", [1e-6, 0.999999, 3.0])
def test_extreme_thresholds(tau):
    w = W.small("tau_edge", 2048, hq=2, hkv=1, stride=8, tau=tau, seed=5)
    x = W.generate(w)
    g = run_path(w, x)
    cnt = g["cnt"].cpu().numpy()
    if tau >= 1.0:
        assert np.array_equal(cnt, np.tile(np.arange(1, 17), (2, 1)))
    if tau <= 1e-6:
        assert np.all(cnt == 1)
    check_sampled(w, x, g, oracle.all_rows(2, w.n_blocks))


def test_batch_two_matches_two_single_batches():
    w = W.small("b2", 1024, hq=4, hkv=2, stride=8, tau=0.9, seed=77)
    x = W.generate(w)
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    qb = torch.cat([q, q.flip(0)]).view(2, 4, 1024, 128)
    kb = torch.cat([k, k.flip(0)]).view(2, 2, 1024, 128)
    vb = torch.cat([v, v.flip(0)]).view(2, 2, 1024, 128)
    ob, _, _ = X.xattn_forward(qb, kb, vb, causal=True, stride=8, tau=0.9)
    o1, _, _ = X.xattn_forward(q, k, v, causal=True, stride=8, tau=0.9)
    o2, _, _ = X.xattn_forward(q.flip(0).contiguous(), k.flip(0).contiguous(),
                               v.flip(0).contiguous(), causal=True, stride=8, tau=0.9)
    torch.cuda.synchronize()
    assert torch.equal(ob.view(8, 1024, 128)[:4].view(torch.int16), o1.view(torch.int16))
    assert torch.equal(ob.view(8, 1024, 128)[4:].view(torch.int16), o2.view(torch.int16))
