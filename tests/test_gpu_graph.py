"""The forward path (score -> select -> sparse attention) launches kernels
only (no allocation, copy, memset or synchronisation), so it can be captured
in a HIP graph: every replay, with new inputs copied into the captured
buffers and eager work and synchronisations between replays, must give
bitwise the eager result on the same inputs."""
import pytest

import workloads as W

from .helpers import dev_bf16

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2503_16428_amd as X  # noqa: E402


def same_bits(a, b):
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


def _inputs(seed):
    w = W.small("graph", 8192, hq=4, hkv=2, stride=8, tau=0.9, seed=seed)
    x = W.generate(w)
    return w, tuple(dev_bf16(x[n]) for n in "qkv")


def test_forward_captured_in_a_graph_replays_like_eager():
    w, (q0, k0, v0) = _inputs(71)
    q, k, v = q0.clone(), k0.clone(), v0.clone()  # the captured input buffers
    dims = X.make_dims(q, k, True)
    ws = torch.empty(X.forward_workspace_size(dims, 128, w.stride), dtype=torch.uint8,
                     device="cuda")
    o = torch.empty_like(q)
    lse = torch.empty((dims.heads, dims.seq), dtype=torch.float32, device="cuda")

    def fwd(**kw):
        return X.xattn_forward(q, k, v, causal=True, stride=w.stride, tau=w.tau, o=o, lse=lse,
                               workspace=ws, want_lse=True, **kw)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fwd(stream=s)  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    print("capturing xattn_forward", flush=True)
    with torch.cuda.graph(g):
        _, _, views = fwd()
    torch.cuda.synchronize()
    for seed in (72, 73, 74):
        _, (qn, kn, vn) = _inputs(seed)
        q.copy_(qn)
        k.copy_(kn)
        v.copy_(vn)
        torch.cuda.synchronize()
        print(f"replay with inputs of seed {seed}", flush=True)
        g.replay()
        torch.cuda.synchronize()
        got_o, got_lse, got_cnt = o.clone(), lse.clone(), views["cnt"].clone()
        want_o, want_lse, want_views = X.xattn_forward(qn, kn, vn, causal=True, stride=w.stride,
                                                       tau=w.tau, want_lse=True)
        torch.cuda.synchronize()
        assert same_bits(got_o, want_o), seed
        assert torch.equal(got_lse, want_lse), seed
        assert torch.equal(got_cnt, want_views["cnt"]), seed
