"""Pins of the minimum-threshold prediction oracle (Sec. 3.3): the dynamic
program against enumeration of every adjustment assignment, against the
closed form of the one-adjustment-per-head case, boundary budgets, and the
threshold and error helpers. A planted mistake in the recurrence is caught."""
import itertools
import math

import numpy as np
import pytest

import oracle
from oracle import thresholds as T


def enumerate_best(perf, M):
    H, A = len(perf), len(perf[0]) - 1
    best = -math.inf
    for assign in itertools.product(range(A + 1), repeat=H):
        if sum(assign) == M:
            best = max(best, sum(perf[h][a] for h, a in enumerate(assign)))
    return best


@pytest.mark.parametrize("H,A,seed", [(5, 1, 0), (6, 1, 1), (4, 2, 2), (5, 3, 3), (3, 2, 4)])
def test_dp_matches_enumeration(H, A, seed):
    rng = np.random.default_rng(seed)
    perf = -np.cumsum(rng.random((H, A + 1)), axis=1)   # more adjustments, more error
    perf[rng.random(H) < 0.3] *= 0.5
    for M in range(0, H * A + 1):
        adjust, best = oracle.threshold_dp(perf, M)
        assert sum(adjust) == M and all(0 <= a <= A for a in adjust)
        assert math.isclose(sum(perf[h][a] for h, a in enumerate(adjust)), best, rel_tol=1e-12,
                            abs_tol=1e-12)
        assert math.isclose(best, enumerate_best(perf, M), rel_tol=1e-12, abs_tol=1e-12)


def test_one_adjustment_per_head_takes_the_smallest_losses():
    # With at most one adjustment per head the best M heads to adjust are the
    # M with the smallest performance loss perf[h][0] - perf[h][1].
    rng = np.random.default_rng(7)
    H = 24
    p0 = -rng.random(H)
    loss = rng.permutation(H) * 0.01 + 0.001     # distinct losses
    perf = np.stack([p0, p0 - loss], axis=1)
    for M in (0, 1, 5, 12, 23, 24):
        adjust, _ = oracle.threshold_dp(perf, M)
        chosen = {h for h in range(H) if adjust[h]}
        assert chosen == set(np.argsort(loss)[:M].tolist())


def test_budget_bounds_and_ties():
    perf = [[0.0, -1.0], [0.0, -1.0], [0.0, -1.0]]
    assert oracle.threshold_dp(perf, 0) == ([0, 0, 0], 0.0)
    assert oracle.threshold_dp(perf, 3) == ([1, 1, 1], -3.0)
    adjust, best = oracle.threshold_dp(perf, 1)
    assert best == -1.0 and sum(adjust) == 1
    with pytest.raises(ValueError):
        oracle.threshold_dp(perf, 4)


def test_thresholds_and_errors_helpers():
    t = oracle.thresholds_from_adjustments(0.9, [0, 1, 2])
    assert np.allclose(t, [0.9, 0.81, 0.729], rtol=1e-6) and t.dtype == np.float32
    o_ref = np.ones((2, 4, 2))
    o = o_ref.copy()
    o[1, 0, 0] = 3.0                     # one element off by 2 in head 1
    e = oracle.head_errors(o, o_ref)
    assert e[0] == 0.0 and math.isclose(e[1], 4.0 / 8.0)


def test_planted_mistake_in_the_recurrence_is_caught():
    # reading the previous head's row at m instead of m - a drops the budget
    import inspect
    src = inspect.getsource(T)
    bad = src.replace("prev = D[h - 1][m - a]", "prev = D[h - 1][m]")
    assert bad != src
    ns = {}
    exec(compile(bad, "mutant", "exec"), ns)
    rng = np.random.default_rng(11)
    perf = -np.cumsum(rng.random((5, 2)), axis=1)
    caught = False
    for M in range(0, 6):
        try:
            adjust, best = ns["threshold_dp"](perf, M)
            if sum(adjust) != M or not math.isclose(best, enumerate_best(perf, M)):
                caught = True
        except AssertionError:
            caught = True
    assert caught
