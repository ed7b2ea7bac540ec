"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compares the oracle with itself: each expected value comes from
a different computation (brute-force index walk over the full fp64 Q K^T,
numpy/scipy softmax, torch's fp64 CPU attention, subset enumeration, closed
forms) or from the geometry the paper draws (Fig. 1).
"""
import itertools
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def f64(u16):
    return W.bf16_bits_to_f32(u16).astype(np.float64)


def walk_scores(q, k, B, S, causal, hq_per_kv=1, mask=None):
    """Brute force: full fp64 logits Q K^T, summed over the positions (i, k)
    with (i mod S) + (k mod S) = S - 1 inside each S x S sub-block
    (Sec. 3.2), scaled by 1/(sqrt(d) S), softmaxed per reduced row over the
    valid reduced columns, block mass averaged over the block's reduced rows.
    mask (S x S, bool) replaces the antidiagonal by another sub-block pattern."""
    H, L, D = q.shape
    NB, NR, nr = L // B, L // S, B // S
    out = np.zeros((H, NB, NB))
    ii = np.arange(L)
    if mask is None:
        anti = ((ii[:, None] % S) + (ii[None, :] % S)) == S - 1
    else:
        anti = np.asarray(mask, bool)[ii[:, None] % S, ii[None, :] % S]
    for h in range(H):
        M = f64(q[h]) @ f64(k[h // hq_per_kv]).T
        Ma = np.where(anti, M, 0.0)
        X = Ma.reshape(NR, S, NR, S).sum(axis=(1, 3)) / (math.sqrt(D) * S)
        if causal:
            X = np.where(np.tril(np.ones((NR, NR), bool)), X, -np.inf)
        A = scipy.special.softmax(X, axis=1)
        out[h] = A.reshape(NB, nr, NB, nr).sum(axis=(1, 3)) / nr
    return out


def exact_block_mass(q, k, B, causal, hq_per_kv=1):
    H, L, D = q.shape
    NB = L // B
    out = np.zeros((H, NB, NB))
    for h in range(H):
        s = f64(q[h]) @ f64(k[h // hq_per_kv]).T / math.sqrt(D)
        if causal:
            s = np.where(np.tril(np.ones((L, L), bool)), s, -np.inf)
        P = scipy.special.softmax(s, axis=1)
        out[h] = P.reshape(NB, B, NB, B).sum(axis=(1, 3)) / B
    return out


# ---------------------------------------------------------------- scoring


@pytest.mark.parametrize("S,causal,D", [(2, True, 16), (4, True, 16), (8, True, 128),
                                        (16, True, 16), (4, False, 16), (8, False, 128)])
def test_score_equals_antidiagonal_index_walk(S, causal, D):
    B, L = 32, 256
    q = W.random_bf16((2, L, D), seed=11 + S, scale=1.5)
    k = W.random_bf16((1, L, D), seed=23 + S, scale=1.5)
    got = oracle.score_rows(q, k, B, S, causal).reshape(2, L // B, L // B)
    want = walk_scores(q, k, B, S, causal, hq_per_kv=2)
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-14)


@pytest.mark.parametrize("pattern", ["diagonal", "random", "antidiagonal"])
@pytest.mark.parametrize("S,causal", [(4, True), (8, False), (8, True)])
def test_score_pattern_equals_masked_index_walk(pattern, S, causal):
    # Pattern ablation (Sec. 4.5, Table 4): the S summed positions of each
    # S x S sub-block form a permutation matrix (one per row and column).
    # The oracle's pairing qsub must equal the brute-force walk over the full
    # logits masked by that matrix; the antidiagonal pairing must reproduce
    # the Algorithm 1 scores exactly.
    B, L, D = 32, 256, 16
    q = W.random_bf16((2, L, D), seed=31 + S, scale=1.5)
    k = W.random_bf16((1, L, D), seed=37 + S, scale=1.5)
    qsub = {"diagonal": np.arange(S), "antidiagonal": np.arange(S)[::-1],
            "random": np.random.default_rng(S).permutation(S)}[pattern]
    mask = np.zeros((S, S), bool)
    mask[qsub, np.arange(S)] = True
    assert np.all(mask.sum(0) == 1) and np.all(mask.sum(1) == 1)
    got = oracle.score_pattern_rows(q, k, B, S, qsub, causal).reshape(2, L // B, L // B)
    want = walk_scores(q, k, B, S, causal, hq_per_kv=2, mask=mask)
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-14)
    if pattern == "antidiagonal":
        np.testing.assert_array_equal(
            got, oracle.score_rows(q, k, B, S, causal).reshape(2, L // B, L // B))


def test_score_walk_on_clustered_inputs():
    w = W.small("pin", 512, hq=2, hkv=1, stride=8)
    x = W.generate(w)
    got = oracle.score_rows(x["q"], x["k"], 128, 8, True).reshape(2, 4, 4)
    want = walk_scores(x["q"], x["k"], 128, 8, True, hq_per_kv=2)
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-14)


@pytest.mark.parametrize("causal", [True, False])
def test_stride_one_is_exact_block_mass(causal):
    # With S = 1 the reduced product is the full Q K^T / sqrt(d), so the block
    # score is the exact softmax block mass (averaged over the block's rows).
    B, L, D = 32, 192, 64
    q = W.random_bf16((1, L, D), seed=5, scale=2.0)
    k = W.random_bf16((1, L, D), seed=6, scale=2.0)
    got = oracle.score_rows(q, k, B, 1, causal).reshape(1, L // B, L // B)
    want = exact_block_mass(q, k, B, causal)
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-14)


def test_score_rows_sum_to_one_and_causal_zeros():
    w = W.small("pin", 1024, hq=2, hkv=1, stride=16)
    x = W.generate(w)
    sc = oracle.score_rows(x["q"], x["k"], 128, 16, True).reshape(2, 8, 8)
    np.testing.assert_allclose(sc.sum(-1), 1.0, rtol=0, atol=1e-12)
    assert np.all(sc[:, np.triu_indices(8, 1)[0], np.triu_indices(8, 1)[1]] == 0.0)


def test_score_key_shift_invariance():
    # Adding one vector u to every key adds sum_t q_{RS+S-1-t}.u / (S sqrt d)
    # to every logit of reduced row R: the row softmax is unchanged.
    # Small-integer values keep every input and sum exact in bf16.
    rng = np.random.default_rng(3)
    L, D, B, S = 256, 16, 32, 4
    qf = rng.integers(-3, 4, (1, L, D)).astype(np.float32) / 4
    kf = rng.integers(-3, 4, (1, L, D)).astype(np.float32) / 4
    u = rng.integers(-2, 3, D).astype(np.float32) / 4
    q, k, k2 = W.to_bf16_bits(qf), W.to_bf16_bits(kf), W.to_bf16_bits(kf + u)
    assert np.array_equal(W.bf16_bits_to_f32(k2), kf + u)
    a = oracle.score_rows(q, k, B, S, True)
    b = oracle.score_rows(q, k2, B, S, True)
    np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-15)


@pytest.mark.parametrize("S", [1, 4, 8])
def test_zero_query_closed_form(S):
    # Q = 0: every valid reduced logit is 0, so reduced row R is uniform over
    # its R+1 valid columns (causal). Block mass = (1/nr) sum_r
    # |{c in block j : c <= R}| / (R + 1).
    L, D, B = 256, 32, 64
    q = np.zeros((1, L, D), np.uint16)
    k = W.random_bf16((1, L, D), seed=9)
    got = oracle.score_rows(q, k, B, S, True)
    NB, nr = L // B, B // S
    want = np.zeros((NB, NB))
    for b in range(NB):
        for r in range(nr):
            R = b * nr + r
            for j in range(NB):
                n_valid = max(0, min(R, (j + 1) * nr - 1) - j * nr + 1)
                want[b, j] += n_valid / (R + 1) / nr
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-15)


def _fig1_mask():
    lines = [l.strip() for l in open(os.path.join(GOLDEN, "fig1_antidiagonal_L24_B8_S4.txt"))
             if l.strip() and not l.startswith("%")]
    return np.array([[c == "X" for c in l] for l in lines])


def test_fig1_geometry():
    # Fig. 1: L = 24, 8 x 8 blocks, stride 4. A one-hot logit at (i0, k0)
    # changes the scores iff (i0, k0) lies on a strided antidiagonal.
    L, B, S, D = 24, 8, 4, 128
    alpha = W.to_bf16_bits(np.array([8.0], np.float32))[0]
    one = W.to_bf16_bits(np.array([1.0], np.float32))[0]
    base = oracle.score_rows(np.zeros((1, L, D), np.uint16),
                             np.zeros((1, L, D), np.uint16), B, S, False)
    sens = np.zeros((L, L), bool)
    for i0 in range(L):
        for k0 in range(L):
            q = np.zeros((1, L, D), np.uint16)
            k = np.zeros((1, L, D), np.uint16)
            q[0, i0, 0] = alpha
            k[0, k0, 0] = one
            sc = oracle.score_rows(q, k, B, S, False)
            sens[i0, k0] = not np.allclose(sc, base, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(sens, _fig1_mask())
    per_block = sens.reshape(3, 8, 3, 8).sum(axis=(1, 3))
    assert np.all(per_block == 16)
    # "every token contributes" (Sec. 3.1): each query row and each key column
    # of every S x S sub-block holds exactly one sampled position.
    sub = sens.reshape(6, 4, 6, 4)
    assert np.all(sub.sum(axis=1) == 1) and np.all(sub.sum(axis=3) == 1)
    # Slashes i - k = delta: with even S only odd offsets are ever sampled
    # (so the main diagonal is not), vertical lines B/S times per block.
    ii, kk = np.nonzero(sens)
    assert np.all((ii - kk) % 2 == 1)
    assert np.all(sens.reshape(3, 8, 24).sum(axis=1) == B // S)


# ---------------------------------------------------------------- selection


def _units(s):
    return np.floor(np.clip(s.astype(np.float64), 0.0, 1.0) * 2.0 ** 32).astype(np.uint64)


@pytest.mark.parametrize("seed,ties", [(1, False), (2, False), (3, True), (4, True)])
def test_select_matches_subset_enumeration(seed, ties):
    NB = 10
    s, rb = W.random_score_rows(60, NB, seed=seed, causal=True, ties=ties)
    for tau in (0.3, 0.5, 0.8, 0.9, 0.95, 0.999):
        idx, cnt = oracle.select_rows(s, rb, tau, causal=True)
        for r in range(len(rb)):
            m = rb[r] + 1
            u = _units(s[r, :m])
            target = math.ceil(float(np.float32(tau)) * float(int(u.sum())))
            best = None
            for size in range(1, m + 1):
                if any(int(u[list(c)].sum()) >= target
                       for c in itertools.combinations(range(m), size)):
                    best = size
                    break
            assert cnt[r] == best, (r, tau)
            sel = idx[r, :cnt[r]]
            assert np.all(np.diff(sel) > 0)
            assert int(u[sel].sum()) >= target
            # the selected set is the top-cnt by (mass desc, index asc)
            order = sorted(range(m), key=lambda j: (-int(u[j]), j))
            assert set(order[:cnt[r]]) == set(sel.tolist())


def test_select_small_integer_masses_match_subset_enumeration():
    # Masses of a few units each: the target ceil(tau * T) is often fractional
    # before rounding up, so "reaches tau * T" is tested at its boundary.
    rng = np.random.default_rng(12)
    NB = 9
    for tau in (0.3, 0.5, 0.6, 0.7, 0.9):
        s = (rng.integers(0, 6, (40, NB)) * 2.0 ** -32).astype(np.float32)
        rb = np.full(40, NB - 1, np.int32)
        idx, cnt = oracle.select_rows(s, rb, tau, causal=False)
        for r in range(40):
            u = [int(x) for x in _units(s[r])]
            thr = float(np.float32(tau)) * sum(u)
            best = next(size for size in range(1, NB + 1)
                        if size == NB or any(sum(u[j] for j in c) >= thr
                                             for c in itertools.combinations(range(NB), size)))
            assert cnt[r] == best, (tau, u)
            assert sum(u[j] for j in idx[r, :cnt[r]]) >= thr or cnt[r] == NB


def test_select_clamps_masses_to_unit_interval():
    # A block mass is at most 1: larger values count as 1, negative or NaN as 0.
    s = np.array([[3.0, 1.0, 0.5, -2.0, np.nan, 0.5]], np.float32)
    idx, cnt = oracle.select_rows(s, np.array([5], np.int32), 0.7, causal=False)
    # units: [2^32, 2^32, 2^31, 0, 0, 2^31], T = 3 * 2^32, target = 0.7 T
    # -> two blocks of 2^32 (2/3 of T) fall short, the third (2^31, j=2) reaches it
    assert cnt[0] == 3 and idx[0, :3].tolist() == [0, 1, 2]


def test_select_tau_one_takes_every_candidate_even_zero_mass():
    s = np.zeros((3, 6), np.float32)
    s[0, :3] = [1.0, 0.0, 0.0]
    s[1, :6] = [0.5, 0.5, 0, 0, 0, 0]
    s[2, :1] = [1.0]
    rb = np.array([2, 5, 0], np.int32)
    idx, cnt = oracle.select_rows(s, rb, 1.0, causal=True)
    assert cnt.tolist() == [3, 6, 1]
    assert idx[1, :6].tolist() == list(range(6))
    idx, cnt = oracle.select_rows(s, rb, 1.0, causal=False)
    assert cnt.tolist() == [6, 6, 6]


def test_select_monotone_in_tau_and_ties_prefer_low_index():
    s, rb = W.random_score_rows(200, 64, seed=8, causal=True)
    prev = None
    for tau in (0.1, 0.5, 0.8, 0.9, 0.95, 0.99, 1.0):
        idx, cnt = oracle.select_rows(s, rb, tau)
        sets = [set(idx[r, :cnt[r]].tolist()) for r in range(len(rb))]
        if prev is not None:
            assert all(a <= b for a, b in zip(prev, sets))
        prev = sets
    t = np.zeros((1, 8), np.float32)
    t[0, :] = 0.125
    idx, cnt = oracle.select_rows(t, np.array([7], np.int32), 0.5)
    assert cnt[0] == 4 and idx[0, :4].tolist() == [0, 1, 2, 3]


def _unit_masses(row):
    """Integer masses of a float32 score row (the find_blocks quantisation)."""
    return [int(np.floor(min(max(float(x), 0.0), 1.0) * 2.0 ** 32)) if x == x else 0
            for x in row]


@pytest.mark.parametrize("ties", [False, True])
def test_topk_is_the_upper_set_of_the_selection_order(ties):
    # Top-K (Sec. 4.5, Table 6): exactly min(k, m) blocks, and no unselected
    # candidate outranks a selected one in the (mass desc, j asc) order; the
    # two properties determine the set. Output ascending.
    s, rb = W.random_score_rows(80, 24, seed=21, causal=True, ties=ties)
    for k in (1, 2, 5, 11, 24, 100):
        idx, cnt = oracle.select_topk_rows(s, rb, k)
        for r in range(len(rb)):
            m = int(rb[r]) + 1
            sel = idx[r, :cnt[r]].tolist()
            assert cnt[r] == min(k, m) and sel == sorted(sel) and len(set(sel)) == len(sel)
            assert all(0 <= j < m for j in sel) and np.all(idx[r, cnt[r]:] == -1)
            u = _unit_masses(s[r, :m])
            rest = [j for j in range(m) if j not in sel]
            for j in sel:
                for jj in rest:
                    assert u[j] > u[jj] or (u[j] == u[jj] and j < jj), (r, k, j, jj)


def test_topk_sets_nest_and_match_threshold_selection_at_its_count():
    # Threshold selection is the shortest prefix of the same order, so Top-K
    # with k = its count returns the same set; larger k only adds blocks.
    s, rb = W.random_score_rows(150, 40, seed=22, causal=True)
    for tau in (0.3, 0.8, 0.95):
        ti, tc = oracle.select_rows(s, rb, tau)
        ki, kc = oracle.select_topk_rows(s, rb, tc)
        assert np.array_equal(tc, kc) and np.array_equal(ti, ki)
    prev = None
    for k in (1, 3, 8, 20, 40):
        idx, cnt = oracle.select_topk_rows(s, rb, k)
        sets = [set(idx[r, :cnt[r]].tolist()) for r in range(len(rb))]
        if prev is not None:
            assert all(a <= b for a, b in zip(prev, sets))
        prev = sets


def test_topk_brute_force_mass_is_maximal():
    # Among all k-subsets of the candidates, the Top-K set has the largest
    # total integer mass (enumerated on rows of at most 10 candidates).
    import itertools
    s, rb = W.random_score_rows(40, 10, seed=23, causal=True)
    for k in (1, 2, 3, 4):
        idx, cnt = oracle.select_topk_rows(s, rb, k)
        for r in range(len(rb)):
            m = int(rb[r]) + 1
            u = _unit_masses(s[r, :m])
            best = max(sum(u[j] for j in c) for c in itertools.combinations(range(m), min(k, m)))
            assert sum(u[j] for j in idx[r, :cnt[r]]) == best


@pytest.mark.parametrize("ratio,m,want", [
    (0.5, 10, 5), (0.5, 3, 2),          # exact half rounds up
    (0.27, 100, 27), (0.7, 10, 7),      # fp32 0.27 is above, fp32 0.7 below the decimal
    (0.31, 16, 5), (0.01, 3, 1),        # 4.96 -> 5; 0.03 -> at least one block
    (1.0, 9, 9), (2.0, 4, 4),           # everything, never more than the candidates
])
def test_ratio_block_count_rounds_to_nearest(ratio, m, want):
    s = np.zeros((1, m), np.float32)
    s[0] = np.arange(m, 0, -1) / np.arange(1, m + 1).sum()
    idx, cnt = oracle.select_ratio_rows(s, np.array([m - 1], np.int32), ratio)
    assert cnt[0] == want and idx[0, :want].tolist() == list(range(want))


def test_per_head_thresholds_apply_each_heads_own_tau():
    s, rb = W.random_score_rows(120, 32, seed=24, causal=True)
    rh = np.arange(120) % 6          # 3 query heads x batch 2
    tau_h = [0.5, 0.9, 0.99]
    idx, cnt = oracle.select_heads_rows(s, rh, rb, tau_h, hq=3)
    for hh, tau in enumerate(tau_h):
        rows = np.nonzero(rh % 3 == hh)[0]
        i2, c2 = oracle.select_rows(s[rows], rb[rows], tau)
        assert np.array_equal(idx[rows], i2) and np.array_equal(cnt[rows], c2)
    assert len({int(c) for c in cnt}) > 1


# ---------------------------------------------------------------- attention


def torch_attention(q, k, v, causal, hq_per_kv=1, block_mask=None, B=None):
    """torch fp64 CPU scaled_dot_product_attention (library routine)."""
    Q = torch.from_numpy(f64(q))
    K = torch.from_numpy(f64(k)).repeat_interleave(hq_per_kv, 0)
    V = torch.from_numpy(f64(v)).repeat_interleave(hq_per_kv, 0)
    L = Q.shape[1]
    mask = torch.ones(Q.shape[0], L, L, dtype=torch.bool)
    if causal:
        mask &= torch.tril(torch.ones(L, L, dtype=torch.bool))
    if block_mask is not None:
        mask &= torch.from_numpy(np.repeat(np.repeat(block_mask, B, 1), B, 2))
    return torch.nn.functional.scaled_dot_product_attention(
        Q, K, V, attn_mask=mask).numpy()


@pytest.mark.parametrize("causal", [True, False])
def test_dense_matches_torch_sdpa(causal):
    L, D, B = 384, 128, 128
    q = W.random_bf16((4, L, D), seed=31, scale=1.0)
    k = W.random_bf16((2, L, D), seed=32, scale=1.0)
    v = W.random_bf16((2, L, D), seed=33)
    o, lse = oracle.dense_attn_rows(q, k, v, B, causal)
    want = torch_attention(q, k, v, causal, hq_per_kv=2)
    np.testing.assert_allclose(o.reshape(4, L, D), want, rtol=1e-10, atol=1e-12)
    # log-sum-exp against scipy
    s = np.einsum("hid,hjd->hij", f64(q), np.repeat(f64(k), 2, 0)) / math.sqrt(D)
    if causal:
        s = np.where(np.tril(np.ones((L, L), bool)), s, -np.inf)
    np.testing.assert_allclose(lse.reshape(4, L), scipy.special.logsumexp(s, axis=-1),
                               rtol=1e-12)


@pytest.mark.parametrize("causal", [True, False])
def test_sparse_equals_block_masked_attention(causal):
    L, D, B = 512, 64, 64
    NB = L // B
    q = W.random_bf16((2, L, D), seed=41)
    k = W.random_bf16((1, L, D), seed=42)
    v = W.random_bf16((1, L, D), seed=43)
    rng = np.random.default_rng(44)
    rh, rb = oracle.all_rows(2, NB)
    idx = np.full((len(rh), NB), -1, np.int32)
    cnt = np.zeros(len(rh), np.int32)
    bm = np.zeros((2, NB, NB), bool)
    for r in range(len(rh)):
        cand = np.arange(rb[r] + 1) if causal else np.arange(NB)
        sel = np.sort(rng.choice(cand, rng.integers(1, len(cand) + 1), replace=False))
        if causal and rb[r] not in sel:      # every query must see a key
            sel = np.sort(np.append(sel, rb[r]))
        idx[r, :len(sel)] = sel
        cnt[r] = len(sel)
        bm[rh[r], rb[r], sel] = True
    o, _ = oracle.sparse_attn_rows(q, k, v, B, idx, cnt, causal)
    want = torch_attention(q, k, v, causal, hq_per_kv=2, block_mask=bm, B=B)
    np.testing.assert_allclose(o.reshape(2, L, D), want, rtol=1e-10, atol=1e-12)


def test_tau_one_forward_equals_dense_causal():
    w = W.small("pin", 512, hq=2, hkv=1, stride=8)
    x = W.generate(w)
    f = oracle.forward_rows(x["q"], x["k"], x["v"], 128, 8, 1.0, True)
    assert np.all(f["cnt"] == np.tile(np.arange(1, 5), 2))
    o, lse = oracle.dense_attn_rows(x["q"], x["k"], x["v"], 128, True)
    np.testing.assert_array_equal(f["o"], o)
    np.testing.assert_array_equal(f["lse"], lse)


def test_zero_query_attention_is_running_mean_of_values():
    L, D, B = 256, 32, 64
    q = np.zeros((1, L, D), np.uint16)
    k = W.random_bf16((1, L, D), seed=51)
    v = W.random_bf16((1, L, D), seed=52)
    o, lse = oracle.dense_attn_rows(q, k, v, B, True)
    V = f64(v[0])
    want = np.cumsum(V, 0) / np.arange(1, L + 1)[:, None]
    np.testing.assert_allclose(o.reshape(L, D), want, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(lse.reshape(L), np.log(np.arange(1, L + 1)), rtol=1e-14)


def test_block_mass_diagnostics():
    L, D, B, S = 256, 32, 64, 4
    q = W.random_bf16((1, L, D), seed=61, scale=1.5)
    k = W.random_bf16((1, L, D), seed=62, scale=1.5)
    tm, am = oracle.block_mass_rows(q, k, B, S, True)
    np.testing.assert_allclose(tm.reshape(1, 4, 4), exact_block_mass(q, k, B, True),
                               rtol=1e-10, atol=1e-14)
    s = f64(q[0]) @ f64(k[0]).T / math.sqrt(D)
    s = np.where(np.tril(np.ones((L, L), bool)), s, -np.inf)
    P = scipy.special.softmax(s, axis=1)
    ii = np.arange(L)
    P = np.where(((ii[:, None] % S) + (ii[None, :] % S)) == S - 1, P, 0.0)
    blk = P.reshape(4, B, 4, B).sum(axis=(1, 3))
    np.testing.assert_allclose(am, blk / blk.sum(1, keepdims=True), rtol=1e-10, atol=1e-14)
