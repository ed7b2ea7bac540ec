"""The C ABI launches on the stream it is given and nowhere else: the whole
path run on a side stream (inputs produced there, then overwritten there
right after the call) gives bitwise the result of the same call on the
default stream, and two layers forwarded on two streams at once give the
results of forwarding each alone."""
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


def _layer(seed):
    w = W.small("streams", 8192, hq=4, hkv=2, stride=8, tau=0.9, seed=seed)
    x = W.generate(w)
    return w, tuple(dev_bf16(x[n]) for n in "qkv")


def test_forward_on_a_side_stream_is_stream_ordered():
    w, (q, k, v) = _layer(61)
    o_ref, lse_ref, views_ref = X.xattn_forward(q, k, v, causal=True, stride=w.stride,
                                                tau=w.tau, want_lse=True)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    print("forward on a side stream", flush=True)
    with torch.cuda.stream(s):
        q2, k2, v2 = q.clone(), k.clone(), v.clone()
        o, lse, views = X.xattn_forward(q2, k2, v2, causal=True, stride=w.stride, tau=w.tau,
                                        want_lse=True, stream=s)
        # in stream order after the call: must not reach its results
        q2.zero_()
        k2.zero_()
        v2.zero_()
    s.synchronize()
    assert same_bits(o, o_ref)
    assert torch.equal(lse, lse_ref)
    assert torch.equal(views["cnt"], views_ref["cnt"])
    assert torch.equal(views["scores"], views_ref["scores"])


def test_two_layers_on_two_streams_match_each_alone():
    (w1, a), (w2, b) = _layer(62), _layer(63)
    ref = [X.xattn_forward(*t, causal=True, stride=w1.stride, tau=w1.tau)[0] for t in (a, b)]
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    print("two layers on two streams", flush=True)
    outs = []
    for t, s in ((a, s1), (b, s2)):
        with torch.cuda.stream(s):
            outs.append(X.xattn_forward(*t, causal=True, stride=w1.stride, tau=w1.tau,
                                        stream=s)[0])
    torch.cuda.synchronize()
    assert same_bits(outs[0], ref[0]) and same_bits(outs[1], ref[1])
