"""GPU parity: every kernel against the fp64 CPU oracle on the same seeded
inputs, through the C ABI (thin ctypes binding). Small sizes that span
several tiles and a ragged tail; full-size sampled rows live in
test_gpu_full.py."""
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


def _inputs(L, hq, hkv, seed, kind="clustered"):
    w = W.small("t", L, hq=hq, hkv=hkv, seed=seed, kind=kind)
    return W.generate(w)


def _attn_err(o_gpu, o_ref):
    e = np.abs(o_gpu.astype(np.float64) - o_ref)
    return float(e.max()), float(e.mean())


@pytest.mark.parametrize("causal", [True, False])
def test_dense_attention_matches_oracle(causal):
    L, hq, hkv = 640, 4, 2
    x = _inputs(L, hq, hkv, seed=101)
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    print(f"dense attn L={L} hq={hq} hkv={hkv} causal={causal}", flush=True)
    o, lse = X.xattn_dense_attn(q, k, v, causal=causal)
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.dense_attn_rows(x["q"], x["k"], x["v"], 128, causal)
    mx, mean = _attn_err(host_f32(o).reshape(o_ref.shape), o_ref)
    print(f"  max_abs={mx:.3e} mean_abs={mean:.3e}")
    assert mx <= OUT_MAX_ABS and mean <= OUT_MEAN_ABS
    np.testing.assert_allclose(host_f32(lse).reshape(lse_ref.shape), lse_ref, rtol=2e-3, atol=2e-2)


@pytest.mark.parametrize("causal", [True, False])
def test_sparse_attention_on_generated_lists(causal):
    L, hq, hkv = 1280, 4, 1
    NB = L // 128
    x = _inputs(L, hq, hkv, seed=102)
    rng = np.random.default_rng(7)
    idx = np.full((hq * NB, NB), -1, np.int32)
    cnt = np.zeros(hq * NB, np.int32)
    for r in range(hq * NB):
        b = r % NB
        cand = np.arange(b + 1) if causal else np.arange(NB)
        n = rng.integers(0, len(cand) + 1)          # includes empty lists
        sel = np.sort(rng.choice(cand, n, replace=False))
        idx[r, :n] = sel
        cnt[r] = n
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    di = torch.from_numpy(idx.reshape(hq, NB, NB)).cuda()
    dc = torch.from_numpy(cnt.reshape(hq, NB)).cuda()
    print(f"sparse attn generated lists L={L} causal={causal}", flush=True)
    o, lse = X.xattn_block_sparse_attn(q, k, v, di, dc, causal=causal)
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.sparse_attn_rows(x["q"], x["k"], x["v"], 128, idx, cnt, causal)
    og = host_f32(o).reshape(o_ref.shape)
    lg = host_f32(lse).reshape(lse_ref.shape)
    empty = ~np.isfinite(lse_ref)
    assert np.all(og[empty] == 0) and np.all(np.isneginf(lg[empty]))
    mx, mean = _attn_err(og[~empty], o_ref[~empty])
    print(f"  max_abs={mx:.3e} mean_abs={mean:.3e} empty_queries={int(empty.sum())}")
    assert mx <= OUT_MAX_ABS and mean <= OUT_MEAN_ABS
    np.testing.assert_allclose(lg[~empty], lse_ref[~empty], rtol=2e-3, atol=2e-2)


@pytest.mark.parametrize("causal", [True, False])
def test_dense_is_bitwise_sparse_with_full_lists(causal):
    L, hq, hkv = 768, 2, 1
    NB = L // 128
    x = _inputs(L, hq, hkv, seed=103)
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    idx = np.full((hq, NB, NB), -1, np.int32)
    cnt = np.zeros((hq, NB), np.int32)
    for b in range(NB):
        m = b + 1 if causal else NB
        idx[:, b, :m] = np.arange(m)
        cnt[:, b] = m
    o1, l1 = X.xattn_dense_attn(q, k, v, causal=causal)
    o2, l2 = X.xattn_block_sparse_attn(q, k, v, torch.from_numpy(idx).cuda(),
                                       torch.from_numpy(cnt).cuda(), causal=causal)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)


@pytest.mark.parametrize("S", [1, 2, 4, 8, 16, 32, 64])
@pytest.mark.parametrize("causal", [True, False])
def test_scores_match_oracle(S, causal):
    L = 128 * 37 if S > 1 else 128 * 21      # ragged reduced tiles for S >= 2
    hq, hkv = 2, 1
    x = _inputs(L, hq, hkv, seed=200 + S)
    q, k = dev_bf16(x["q"]), dev_bf16(x["k"])
    print(f"score S={S} L={L} causal={causal}", flush=True)
    sc = X.xattn_score(q, k, causal=causal, stride=S)
    torch.cuda.synchronize()
    NB = L // 128
    want = oracle.score_rows(x["q"], x["k"], 128, S, causal)
    got = host_f32(sc).reshape(want.shape)
    rh, rb = oracle.all_rows(hq, NB)
    sel = np.arange(0, len(rh), 5)
    dz = logit_error_bound(x["q"], x["k"], S, rh[sel], rb[sel], hq // hkv)
    rep = compare_scores(got, want, dz)
    print(f"  {rep}")
    assert rep["n_bad"] == 0
    if causal:
        assert np.all(got[np.triu(np.ones((NB, NB), bool), 1)[rb]] == 0)
    np.testing.assert_allclose(got.sum(-1), 1.0, atol=1e-4)


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("NB", [5, 64, 65, 300, 1024, 2048])
def test_select_is_bit_exact_on_same_scores(NB, causal):
    rows = 64 if NB >= 1024 else 200
    s, rb = W.random_score_rows(rows, NB, seed=NB, causal=causal)
    s2, _ = W.random_score_rows(rows, NB, seed=NB + 1, causal=causal, ties=True)
    H = 2
    # a score tensor [H][NB][NB] whose row (h, b) is one generated row
    full = np.zeros((H, NB, NB), np.float32)
    for r in range(rows):
        h, b = r % H, (int(rb[r]) if causal else r % NB)
        full[h, b] = (s if r % 2 == 0 else s2)[r]
    dims = X.Dims(1, H, 1, NB * 128, 128, int(causal))
    for tau in (0.5, 0.8, 0.9, 0.95, 1.0):
        print(f"select NB={NB} causal={causal} tau={tau}", flush=True)
        idx, cnt = X.xattn_select(torch.from_numpy(full).cuda(), dims, tau)
        torch.cuda.synchronize()
        idx, cnt = idx.cpu().numpy(), cnt.cpu().numpy()
        flat = full.reshape(H * NB, NB).astype(np.float64)
        allb = np.tile(np.arange(NB, dtype=np.int32), H)
        oi, oc = oracle.select_rows(flat, allb, tau, causal)
        gc = cnt.reshape(-1)
        gi = idx.reshape(H * NB, NB)
        assert np.array_equal(gc, oc)
        for r in range(H * NB):
            assert np.array_equal(gi[r, :gc[r]], oi[r, :oc[r]]), (r, tau)


def _structured_rows(kind, n, NB, rng):
    """Score rows whose search interval either empties fast (a few large,
    well separated masses over a tiny floor) or stays crowded (hundreds of
    equal masses at the cut, or a dense uniform spread)."""
    if kind == "separated":
        r = np.full((n, NB), 1e-7)
        for i in range(n):
            top = rng.choice(NB, 24, replace=False)
            r[i, top] = 0.6 ** np.arange(24) * rng.uniform(0.5, 1.0)
    elif kind == "crowded_ties":
        r = np.full((n, NB), 1e-7)
        for i in range(n):
            pick = rng.permutation(NB)
            r[i, pick[:400]] = 0.002
            r[i, pick[400:410]] = 0.02
    else:  # uniform
        r = rng.uniform(0.0, 1e-3, (n, NB))
    return r.astype(np.float32)


@pytest.mark.parametrize("kind", ["separated", "crowded_ties", "uniform"])
def test_select_search_paths_bit_exact(kind):
    """Rows of 1024 candidates, threshold and Top-K: the search either
    finishes on the few values left in its interval or keeps scanning every
    candidate; both must give the oracle's lists exactly."""
    NB, H = 1024, 2
    rng = np.random.default_rng({"separated": 11, "crowded_ties": 12, "uniform": 13}[kind])
    full = _structured_rows(kind, H * NB, NB, rng).reshape(H, NB, NB)
    dims = X.Dims(1, H, 1, NB * 128, 128, 0)
    flat = full.reshape(H * NB, NB).astype(np.float64)
    allb = np.tile(np.arange(NB, dtype=np.int32), H)
    dev = torch.from_numpy(full).cuda()
    for tau in (0.5, 0.9, 0.99):
        print(f"select paths kind={kind} tau={tau}", flush=True)
        idx, cnt = X.xattn_select(dev, dims, tau)
        torch.cuda.synchronize()
        oi, oc = oracle.select_rows(flat, allb, tau, False)
        gi, gc = idx.cpu().numpy().reshape(H * NB, NB), cnt.cpu().numpy().reshape(-1)
        assert np.array_equal(gc, oc)
        for r in range(H * NB):
            assert np.array_equal(gi[r, :gc[r]], oi[r, :oc[r]]), (r, tau)
    for k in (1, 37, 500):
        print(f"select paths kind={kind} topk={k}", flush=True)
        idx, cnt = X.xattn_select_topk(dev, dims, k)
        torch.cuda.synchronize()
        oi, oc = oracle.select_topk_rows(flat, allb, np.int32(k), False)
        gi, gc = idx.cpu().numpy().reshape(H * NB, NB), cnt.cpu().numpy().reshape(-1)
        assert np.array_equal(gc, oc)
        for r in range(H * NB):
            assert np.array_equal(gi[r, :gc[r]], oi[r, :oc[r]]), (r, k)


def test_select_on_oracle_scores_rounded_to_fp32():
    L, hq, hkv, S = 2048, 4, 2, 8
    x = _inputs(L, hq, hkv, seed=301)
    NB = L // 128
    sc = oracle.score_rows(x["q"], x["k"], 128, S, True).astype(np.float32)
    dims = X.Dims(1, hq, hkv, L, 128, 1)
    idx, cnt = X.xattn_select(torch.from_numpy(sc.reshape(hq, NB, NB)).cuda(), dims, 0.9)
    torch.cuda.synchronize()
    _, rb = oracle.all_rows(hq, NB)
    oi, oc = oracle.select_rows(sc.astype(np.float64), rb, 0.9, True)
    gi, gc = idx.cpu().numpy().reshape(hq * NB, NB), cnt.cpu().numpy().reshape(-1)
    assert np.array_equal(gc, oc)
    for r in range(hq * NB):
        assert np.array_equal(gi[r, :gc[r]], oi[r, :oc[r]])


@pytest.mark.parametrize("causal,S,kind,L,hq,hkv", [
    (True, 8, "clustered", 3072, 4, 2), (True, 16, "clustered_local", 3072, 4, 2),
    (False, 16, "clustered", 3072, 4, 2),
    # query-head groups of 8 and 16, odd group counts, plain multi-head
    (True, 8, "clustered", 2048, 8, 1), (True, 4, "clustered", 2048, 16, 2),
    (True, 8, "clustered_local", 1536, 16, 1), (False, 8, "clustered", 1536, 6, 3),
    (True, 16, "clustered", 2560, 3, 3)])
def test_forward_end_to_end_small(causal, S, kind, L, hq, hkv):
    tau = 0.9
    x = _inputs(L, hq, hkv, seed=401, kind=kind)
    NB = L // 128
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    print(f"forward L={L} hq={hq} hkv={hkv} S={S} causal={causal} kind={kind}", flush=True)
    o, _, views = X.xattn_forward(q, k, v, causal=causal, stride=S, tau=tau)
    torch.cuda.synchronize()
    f = oracle.forward_rows(x["q"], x["k"], x["v"], 128, S, tau, causal)
    rh, rb = oracle.all_rows(hq, NB)
    dz = logit_error_bound(x["q"], x["k"], S, rh[::7], rb[::7], hq // hkv)
    rep = compare_scores(host_f32(views["scores"]).reshape(f["scores"].shape), f["scores"], dz)
    print(f"  scores {rep}")
    assert rep["n_bad"] == 0
    gi = views["idx"].cpu().numpy().reshape(hq * NB, NB)
    gc = views["cnt"].cpu().numpy().reshape(-1)
    dens = gc.sum() / (np.arange(1, NB + 1).sum() * hq if causal else NB * NB * hq)
    print(f"  density={dens:.3f}")
    same = assert_index_sets(gi, gc, f["idx"], f["cnt"], f["scores"], rb, tau, causal)
    og = host_f32(o).reshape(f["o"].shape)
    assert_attention_on_lists(x, 128, gi, gc, causal, (rh, rb), og)
    mx, mean = _attn_err(og[same], f["o"][same])
    print(f"  end to end on {same.sum()}/{len(rh)} rows with the oracle's lists: "
          f"max_abs={mx:.3e} mean_abs={mean:.3e}")
    assert mx <= OUT_MAX_ABS and mean <= OUT_MEAN_ABS


@pytest.mark.parametrize("L,hq,hkv,S,causal", [
    (128 * 37, 4, 2, 8, True), (128 * 37, 2, 1, 4, False), (128 * 21, 2, 1, 1, True),
    (8192, 2, 2, 64, True), (3072, 2, 1, 16, False), (128, 2, 1, 16, True)])
def test_forward_equals_the_three_calls_bitwise(L, hq, hkv, S, causal):
    """xattn_forward (its workspace holding the packed scoring scratch behind
    the scores and lists) against xattn_score + xattn_select +
    xattn_block_sparse_attn with their own buffers: scores, lists, outputs and
    LSE bitwise equal."""
    x = _inputs(L, hq, hkv, seed=900 + S)
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    print(f"forward vs three calls L={L} S={S} causal={causal}", flush=True)
    o1, l1, views = X.xattn_forward(q, k, v, causal=causal, stride=S, tau=0.9, want_lse=True)
    sc = X.xattn_score(q, k, causal=causal, stride=S)
    dims = X.make_dims(q, k, causal)
    idx, cnt = X.xattn_select(sc, dims, 0.9)
    o2, l2 = X.xattn_block_sparse_attn(q, k, v, idx, cnt, causal=causal)
    torch.cuda.synchronize()
    assert torch.equal(views["scores"], sc)
    assert torch.equal(views["cnt"], cnt)
    NB = L // 128
    c = cnt.cpu().numpy().reshape(-1)
    a, b = views["idx"].cpu().numpy().reshape(-1, NB), idx.cpu().numpy().reshape(-1, NB)
    assert all(np.array_equal(a[r, :c[r]], b[r, :c[r]]) for r in range(len(c)))
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)


def test_repeated_calls_are_bitwise_deterministic():
    L, hq, hkv = 2048, 4, 2
    x = _inputs(L, hq, hkv, seed=501)
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    outs = []
    for _ in range(2):
        o, lse, views = X.xattn_forward(q, k, v, causal=True, stride=8, tau=0.9, want_lse=True)
        torch.cuda.synchronize()
        outs.append((o.clone(), lse.clone(), views["scores"].clone(), views["cnt"].clone()))
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.uint8) if b.dtype == torch.bfloat16 else b)
