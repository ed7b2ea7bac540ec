"""Host-side sizing and validation under arbitrary shapes (no GPU): the
workspace-size and layout calls of the C ABI either reject a shape with an
error code or return sizes that hold together — the forward workspace's
four regions 256-byte aligned, in order, disjoint and inside the reported
size, each region at least as large as its array — for any int32 inputs,
including the largest accepted problems. Property-based (hypothesis)."""
import ctypes

import pytest

hyp = pytest.importorskip("hypothesis")
from hypothesis import given, settings  # noqa: E402
from hypothesis import strategies as st  # noqa: E402

import paper_2503_16428_amd as X  # noqa: E402
from paper_2503_16428_amd import binding as B  # noqa: E402

INT32 = st.integers(min_value=-2**31, max_value=2**31 - 1)
SMALLISH = st.one_of(st.integers(min_value=-4, max_value=300), INT32)
SEQ = st.one_of(st.sampled_from([128, 256, 1024, 4096, 65536, 131072, 262144, 262272]),
                st.integers(min_value=-1024, max_value=1 << 20), INT32)
STRIDE = st.one_of(st.sampled_from([1, 2, 4, 8, 16, 32, 64]), SMALLISH)
CODES = {B.XATTN_OK, B.XATTN_ERR_ARG, B.XATTN_ERR_UNSUPPORTED}


def _dims(batch, hq, hkv, seq, head_dim, causal):
    return B.Dims(batch=batch, hq=hq, hkv=hkv, seq=seq, head_dim=head_dim, causal=causal)


@settings(max_examples=400, deadline=None)
@given(batch=SMALLISH, hq=SMALLISH, hkv=SMALLISH, seq=SEQ,
       head_dim=st.one_of(st.just(128), SMALLISH), causal=st.integers(-1, 2),
       block=st.one_of(st.just(128), SMALLISH), stride=STRIDE)
def test_forward_sizing_is_consistent_or_rejected(batch, hq, hkv, seq, head_dim, causal, block,
                                                  stride):
    lib = X.lib()
    d = _dims(batch, hq, hkv, seq, head_dim, causal)
    ws = ctypes.c_size_t(0)
    rc = lib.xattn_forward_workspace_size(ctypes.byref(d), block, stride, ctypes.byref(ws))
    assert rc in CODES
    offs = [ctypes.c_size_t(0) for _ in range(4)]
    rc2 = lib.xattn_forward_layout(ctypes.byref(d), block, stride, *map(ctypes.byref, offs))
    assert rc2 == rc, "layout and size must accept the same shapes"
    sc_ws = ctypes.c_size_t(0)
    rc3 = lib.xattn_score_workspace_size(ctypes.byref(d), block, stride, ctypes.byref(sc_ws))
    assert rc3 == rc, "scoring and forward sizing must accept the same shapes"
    if rc != B.XATTN_OK:
        assert lib.xattn_last_error(), "a rejection carries a message"
        return
    H, NB = batch * hq, seq // block
    o = [x.value for x in offs]
    assert all(x % 256 == 0 for x in o)
    assert o[0] == 0 and o[0] < o[1] < o[2] < o[3]
    assert o[1] - o[0] >= H * NB * NB * 4          # scores fp32 [H][NB][NB]
    assert o[2] - o[1] >= H * NB * NB * 4          # idx int32 [H][NB][NB]
    assert o[3] - o[2] >= H * NB * 4               # cnt int32 [H][NB]
    assert ws.value >= o[3] + sc_ws.value          # the scoring scratch after them
    assert ws.value < 1 << 50


@settings(max_examples=300, deadline=None)
@given(heads=SMALLISH, max_adjust=SMALLISH, adjustments=SMALLISH)
def test_threshold_dp_rejects_or_runs(heads, max_adjust, adjustments):
    """The host DP on arbitrary sizes: rejected, or run on a small table."""
    lib = X.lib()
    small = 0 < heads <= 64 and 0 <= max_adjust <= 8 and 0 <= adjustments <= 600
    if not small:
        # only the size checks run: pass NULL tables, which must be rejected
        # whenever the sizes are accepted
        rc = lib.xattn_threshold_dp(None, heads, max_adjust, adjustments, None, None)
        assert rc in CODES and rc != B.XATTN_OK
        return
    perf = (ctypes.c_double * (heads * (max_adjust + 1)))(*[0.0] * (heads * (max_adjust + 1)))
    adj = (ctypes.c_int32 * heads)()
    total = ctypes.c_double(0.0)
    rc = lib.xattn_threshold_dp(perf, heads, max_adjust, adjustments, adj, ctypes.byref(total))
    assert rc in CODES
    # the documented contract: max_adjust >= 1 and M in [0, heads * max_adjust]
    assert (rc == B.XATTN_OK) == (max_adjust >= 1 and adjustments <= heads * max_adjust)
    if rc == B.XATTN_OK:
        assert all(0 <= a <= max_adjust for a in adj)
        assert sum(adj) == adjustments
