"""The binding rejects every shape or dtype mismatch before any kernel is
launched (CPU only: the tensors here live on the host, and a call that
passed every shape check would stop at the device check instead)."""
import pytest
import torch

import paper_2503_16428_amd as X
from paper_2503_16428_amd import binding as B


def bf(*shape):
    return torch.zeros(shape, dtype=torch.bfloat16)


H, HKV, L, D = 4, 2, 1024, 128
NB = L // 128


def good():
    return bf(H, L, D), bf(HKV, L, D), bf(HKV, L, D)


def expect(msg, fn, *a, **kw):
    with pytest.raises(B.XAttnError) as e:
        fn(*a, **kw)
    assert msg in str(e.value), str(e.value)
    assert e.value.status == B.XATTN_ERR_ARG


@pytest.mark.parametrize("fn", [X.xattn_dense_attn, X.xattn_forward])
def test_attention_inputs_are_checked(fn):
    q, k, v = good()
    expect("k must be", fn, q, bf(HKV, L // 2, D), v)
    expect("k must be", fn, q, bf(HKV, L, 64), v)
    expect("k must be", fn, q, bf(1, HKV, L, D), v)
    expect("v must have", fn, q, k, bf(HKV, L - 128, D))
    expect("must be torch.bfloat16", fn, q.float(), k, v)
    expect("must be torch.bfloat16", fn, q, k, v.half())
    expect("q must be 3-D or 4-D", fn, bf(L, D), k, v)
    # 4-D: batch must agree
    expect("k must be", fn, bf(2, H, L, D), bf(1, HKV, L, D), bf(1, HKV, L, D))
    # shapes right: stops at the device check, still before any launch
    expect("device tensor", fn, q, k, v)


@pytest.mark.parametrize("fn", [X.xattn_dense_attn, X.xattn_forward])
def test_attention_outputs_are_checked(fn):
    q, k, v = good()
    expect("o must have shape", fn, q, k, v, o=bf(H, L - 128, D))
    expect("o must be", fn, q, k, v, o=torch.zeros(H, L, D))
    expect("lse must have shape", fn, q, k, v, lse=torch.zeros(H, L + 1))
    expect("lse must be", fn, q, k, v, lse=torch.zeros(H, L, dtype=torch.float64))


def test_sparse_attention_lists_are_checked():
    q, k, v = good()
    idx = torch.zeros(H, NB, NB, dtype=torch.int32)
    cnt = torch.zeros(H, NB, dtype=torch.int32)
    f = X.xattn_block_sparse_attn
    expect("idx must have shape", f, q, k, v, idx[:, :, :-1], cnt)
    expect("idx must be", f, q, k, v, idx.long(), cnt)
    expect("cnt must have shape", f, q, k, v, idx, cnt[:-1])
    expect("cnt must be", f, q, k, v, idx, cnt.float())
    expect("v must have", f, q, k, bf(HKV, L, D // 2), idx, cnt)
    expect("device tensor", f, q, k, v, idx, cnt)


def test_selection_tensors_are_checked():
    d = B.Dims(1, H, HKV, L, D, 1)
    s = torch.zeros(H, NB, NB)
    idx = torch.zeros(H, NB, NB, dtype=torch.int32)
    cnt = torch.zeros(H, NB, dtype=torch.int32)
    for fn, arg in ((X.xattn_select, 0.9), (X.xattn_select_heads, 0.9),
                    (X.xattn_select_topk, 3), (X.xattn_select_ratio, 0.2)):
        expect("scores must have shape", fn, s[:, :-1], d, arg)
        expect("scores must be", fn, s.double(), d, arg)
        expect("idx must have shape", fn, s, d, arg, idx=idx[:-1])
        expect("cnt must have shape", fn, s, d, arg, cnt=cnt[:, :-1])
        expect("device tensor", fn, s, d, arg)


def test_scoring_tensors_are_checked():
    q, k, _ = good()
    expect("k must be", X.xattn_score, q, bf(HKV, L + 128, D))
    expect("scores must have shape", X.xattn_score, q, k, scores=torch.zeros(H, NB, NB - 1))
    expect("qsub must hold", X.xattn_score_pattern, q, k, True, 128, 8, [0, 1, 2])
    expect("workspace must be", X.xattn_score, q, k, workspace=torch.zeros(16))
    expect("device tensor", X.xattn_score, q, k)


def test_error_tensors_are_checked():
    a = bf(H, L, D)
    expect("same shape", X.head_error, a, bf(H, L - 128, D))
    expect("must be torch.bfloat16", X.head_error_mean, a, a.float())
    expect("device tensor", X.head_error_mean, a, a)


def test_forward_workspace_is_checked():
    q, k, v = good()
    expect("workspace must be", X.xattn_forward, q, k, v, workspace=torch.zeros(4, 4,
                                                                                dtype=torch.uint8))
    expect("workspace must be", X.xattn_forward_scheduled, q, k, v, 7,
           workspace=torch.zeros(16, dtype=torch.int32))
