"""The library's minimum-threshold dynamic program (host code behind the C
ABI, no GPU) against the oracle's, and its argument checks."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2503_16428_amd as X
from paper_2503_16428_amd import binding as B


@pytest.mark.parametrize("H,A,seed", [(1, 1, 0), (7, 1, 1), (32, 1, 2), (12, 2, 3),
                                      (9, 4, 4), (64, 3, 5)])
def test_native_dp_equals_oracle(H, A, seed):
    rng = np.random.default_rng(seed)
    perf = -np.cumsum(rng.random((H, A + 1)), axis=1)
    perf[:, 1:] += (rng.random((H, A)) < 0.2) * 0.3          # some non-monotone rows
    perf[rng.integers(0, H, H // 3)] = perf[0]                # exact ties between heads
    for M in sorted({0, 1, H // 2, H, H * A // 2, H * A}):
        got, gbest = X.threshold_dp(perf, M)
        want, wbest = oracle.threshold_dp(perf, M)
        assert got.tolist() == want and gbest == wbest, (M, got.tolist(), want)


def test_native_dp_validates():
    L = X.lib()
    perf = (ctypes.c_double * 6)(0.0, -1.0, 0.0, -1.0, 0.0, -1.0)
    adj = (ctypes.c_int32 * 3)()
    best = ctypes.c_double()
    assert L.xattn_threshold_dp(perf, 3, 1, 2, adj, ctypes.byref(best)) == B.XATTN_OK
    assert list(adj) in ([0, 1, 1], [1, 0, 1], [1, 1, 0]) and best.value == -2.0
    assert L.xattn_threshold_dp(perf, 3, 1, 4, adj, None) == B.XATTN_ERR_ARG
    assert L.xattn_threshold_dp(perf, 3, 1, -1, adj, None) == B.XATTN_ERR_ARG
    assert L.xattn_threshold_dp(perf, 0, 1, 0, adj, None) == B.XATTN_ERR_ARG
    assert L.xattn_threshold_dp(None, 3, 1, 1, adj, None) == B.XATTN_ERR_ARG
    bad = (ctypes.c_double * 6)(0.0, -1.0, float("nan"), -1.0, 0.0, -1.0)
    assert L.xattn_threshold_dp(bad, 3, 1, 1, adj, None) == B.XATTN_ERR_ARG
    d = B.Dims(1, 4, 2, 1024, 128, 1)
    fake = ctypes.c_void_p(0x1000)
    n = ctypes.c_size_t(0)
    assert L.xattn_head_error_workspace_size(ctypes.byref(d), ctypes.byref(n)) == B.XATTN_OK
    assert n.value >= 4 * 16
    assert L.xattn_head_error(fake, None, ctypes.byref(d), fake, fake, n.value, None) == \
        B.XATTN_ERR_ARG
    assert L.xattn_head_error(fake, fake, ctypes.byref(d), fake, fake, 8, None) == \
        B.XATTN_ERR_WORKSPACE


def test_native_levels_equal_oracle_thresholds():
    for tau0 in (0.9, 0.95, 0.5, 1.0):
        got = X.threshold_levels(tau0, 6)
        want = oracle.thresholds_from_adjustments(tau0, range(7))
        assert got.dtype == np.float32 and np.array_equal(got, want), (tau0, got, want)


@pytest.mark.parametrize("H,A,seed", [(1, 1, 10), (8, 1, 11), (32, 1, 12), (12, 3, 13)])
def test_native_predict_equals_oracle_pipeline(H, A, seed):
    """xattn_threshold_predict on an error table = the oracle's DP on minus
    the table, then the oracle's thresholds for the chosen adjustments."""
    rng = np.random.default_rng(seed)
    err = np.cumsum(rng.random((H, A + 1)) * 0.1, axis=1)
    err[rng.integers(0, H, H // 3)] = err[0]                 # exact ties between heads
    for M in sorted({0, 1, H // 2, H * A}):
        adj, tau_h, total = X.threshold_predict(err, M, 0.9)
        want, wbest = oracle.threshold_dp(-err, M)
        assert adj.tolist() == want, (M, adj.tolist(), want)
        assert total == -wbest
        assert np.array_equal(tau_h, oracle.thresholds_from_adjustments(0.9, want))


def test_native_predict_validates():
    L = X.lib()
    err = (ctypes.c_double * 4)(0.0, 1.0, 0.0, 1.0)
    adj = (ctypes.c_int32 * 2)()
    tau = (ctypes.c_float * 2)()
    assert L.xattn_threshold_predict(err, 2, 1, 1, 0.9, adj, tau, None) == B.XATTN_OK
    assert sorted(adj) == [0, 1] and sorted(tau) == [np.float32(0.81), np.float32(0.9)]
    for t0 in (0.0, -0.5, float("nan"), float("inf")):
        assert L.xattn_threshold_predict(err, 2, 1, 1, t0, adj, tau, None) == B.XATTN_ERR_ARG
    assert L.xattn_threshold_predict(err, 2, 1, 3, 0.9, adj, tau, None) == B.XATTN_ERR_ARG
    assert L.xattn_threshold_predict(err, 2, 1, 1, 0.9, adj, None, None) == B.XATTN_ERR_ARG
    lv = (ctypes.c_float * 3)()
    assert L.xattn_threshold_levels(0.9, -1, lv) == B.XATTN_ERR_ARG
    assert L.xattn_threshold_levels(0.0, 2, lv) == B.XATTN_ERR_ARG
    assert L.xattn_threshold_levels(0.9, 2, None) == B.XATTN_ERR_ARG
    d = B.Dims(2, 4, 2, 1024, 128, 1)
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: every case fails validation
    assert L.xattn_head_error_mean(fake, None, ctypes.byref(d), fake, fake, 1 << 20, None) == \
        B.XATTN_ERR_ARG
    assert L.xattn_head_error_mean(fake, fake, ctypes.byref(d), fake, fake, 8, None) == \
        B.XATTN_ERR_WORKSPACE
