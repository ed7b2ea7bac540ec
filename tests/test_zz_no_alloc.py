"""xattn_forward_noalloc (the forward pass on the library's static scratch,
for callers that cannot allocate) against xattn_forward with a caller
workspace, through the C ABI: two calls in a row, the second on a smaller
problem, outputs and LSE bitwise equal; and the size limit."""
import numpy as np
import pytest

import oracle
import workloads as W

from .helpers import OUT_MAX_ABS, OUT_MEAN_ABS, dev_bf16, host_f32

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2503_16428_amd as X  # noqa: E402
from paper_2503_16428_amd import binding as B  # noqa: E402


def _case(L, hq, hkv, S, causal, seed):
    w = W.small("noalloc", L, hq=hq, hkv=hkv, stride=S, causal=causal, tau=0.9, seed=seed)
    x = W.generate(w)
    return w, x, [dev_bf16(x[n]) for n in "qkv"]


def test_noalloc_equals_forward_on_two_calls_second_smaller():
    # the larger problem first, so the second call finds the first one's
    # contents in the shared scratch
    for L, hq, hkv, S, causal, seed in ((6144, 8, 2, 8, True, 61), (1536, 2, 1, 16, False, 62)):
        w, x, (q, k, v) = _case(L, hq, hkv, S, causal, seed)
        d = X.make_dims(q, k, causal)
        need = X.forward_workspace_size(d, 128, S)
        print(f"noalloc L={L} hq={hq} hkv={hkv} S={S} causal={causal}: scratch {need} B "
              f"of {64 << 20}", flush=True)
        assert need <= 64 << 20
        o_ref, l_ref, _ = X.xattn_forward(q, k, v, causal, 128, S, 0.9, want_lse=True)
        o = torch.empty_like(q)
        lse = torch.empty((d.heads, L), dtype=torch.float32, device="cuda")
        X.xattn_forward_noalloc(q, k, v, o, lse, causal, 128, S, 0.9)
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
        assert torch.equal(lse, l_ref)
        # and the oracle's bar on a few rows (the oracle run on the GPU's lists)
        _, _, views = X.xattn_forward(q, k, v, causal, 128, S, 0.9)
        NB = L // 128
        rh = np.array([0, hq - 1, hq // 2], np.int32)
        rb = np.array([0, NB - 1, NB // 2], np.int32)
        gi = views["idx"].cpu().numpy().reshape(-1, NB, NB)[rh, rb]
        gc = views["cnt"].cpu().numpy().reshape(-1, NB)[rh, rb]
        o_or, _ = oracle.sparse_attn_rows(x["q"], x["k"], x["v"], 128, gi, gc, causal,
                                          rows=(rh, rb))
        og = host_f32(o).reshape(-1, L, 128)
        got = np.stack([og[h, b * 128:(b + 1) * 128] for h, b in zip(rh, rb)])
        err = np.abs(got - o_or)
        print(f"  vs oracle: max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
        assert err.max() <= OUT_MAX_ABS and err.mean() <= OUT_MEAN_ABS


def test_noalloc_rejects_problems_beyond_the_static_scratch():
    q = torch.zeros((32, 32768, 128), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((8, 32768, 128), dtype=torch.bfloat16, device="cuda")
    o = torch.empty_like(q)
    d = X.make_dims(q, kv, True)
    assert X.forward_workspace_size(d, 128, 8) > 64 << 20
    with pytest.raises(B.XAttnError) as e:
        X.xattn_forward_noalloc(q, kv, kv, o, None, True, 128, 8, 0.9)
    assert e.value.status == B.XATTN_ERR_UNSUPPORTED and "scratch" in str(e.value)


def test_noalloc_forward_captured_in_a_graph_replays_like_eager():
    """The no-allocation forward is what code under graph capture calls: a
    captured call, replayed on new inputs copied into the captured buffers
    (eager work and synchronisation between replays), gives bitwise the
    eager xattn_forward result every time."""
    w, x, (q, k, v) = _case(4096, 4, 2, 8, True, 81)
    o = torch.empty_like(q)
    lse = torch.empty((4, 4096), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        X.xattn_forward_noalloc(q, k, v, o, lse, True, 128, 8, 0.9, stream=s)  # outside capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    print("capturing xattn_forward_noalloc", flush=True)
    with torch.cuda.graph(g):
        X.xattn_forward_noalloc(q, k, v, o, lse, True, 128, 8, 0.9)
    torch.cuda.synchronize()
    for seed in (82, 83, 84):
        _, _, (qn, kn, vn) = _case(4096, 4, 2, 8, True, seed)
        q.copy_(qn)
        k.copy_(kn)
        v.copy_(vn)
        torch.cuda.synchronize()
        print(f"replay with inputs of seed {seed}", flush=True)
        g.replay()
        torch.cuda.synchronize()
        got_o, got_lse = o.clone(), lse.clone()
        want_o, want_lse, _ = X.xattn_forward(qn, kn, vn, True, 128, 8, 0.9, want_lse=True)
        torch.cuda.synchronize()
        assert torch.equal(got_o.view(torch.int16), want_o.view(torch.int16)), seed
        assert torch.equal(got_lse, want_lse), seed
