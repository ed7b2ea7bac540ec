"""GPU checks of the video-DiT denoising schedule (Sec. 4.2): dense attention
for the first warm-up steps, XAttention afterwards, at the video shape (115,200
tokens = 30 frames x 60 x 64, 24 heads, non-causal, S = 16) and small ones."""
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


def same_bits(a, b):
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_video_shape_schedule_switches_after_warmup():
    w = W.WORKLOADS["c5"]
    print(f"schedule at {w.name}", flush=True)
    x = W.generate(w, threads=16)
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    od, ld = X.xattn_dense_attn(q, k, v, causal=False)
    of, lf, _ = X.xattn_forward(q, k, v, causal=False, stride=w.stride, tau=w.tau,
                                want_lse=True)
    torch.cuda.synchronize()
    for step in (0, 4, 5, 49):
        o, lse = X.xattn_forward_scheduled(q, k, v, step, warmup_steps=5, causal=False,
                                           stride=w.stride, tau=w.tau, want_lse=True)
        torch.cuda.synchronize()
        ro, rl = (od, ld) if step < 5 else (of, lf)
        assert same_bits(o, ro) and torch.equal(lse, rl), step
    # the dense phase against the oracle's dense attention on sampled rows
    rows = (np.array([0, 23], np.int32), np.array([0, w.n_blocks - 1], np.int32))
    o_ref, lse_ref = oracle.dense_attn_rows(x["q"], x["k"], x["v"], w.block, False, rows=rows)
    og = host_f32(od).reshape(w.hq, w.seq, w.head_dim)
    got = np.stack([og[h, b * w.block:(b + 1) * w.block] for h, b in zip(*rows)])
    err = np.abs(got - o_ref)
    print(f"  dense phase vs oracle: max_abs={err.max():.3e} mean_abs={err.mean():.3e}")
    assert err.max() <= OUT_MAX_ABS and err.mean() <= OUT_MEAN_ABS
    lg = ld.cpu().numpy().reshape(w.hq, w.seq)
    lg = np.stack([lg[h, b * w.block:(b + 1) * w.block] for h, b in zip(*rows)])
    assert np.abs(lg - lse_ref).max() <= 1e-2


@pytest.mark.parametrize("warmup", [0, 1, 3])
def test_small_schedule_sequence(warmup):
    w = W.small("sched", 2048, hq=2, hkv=2, causal=False, stride=8, tau=0.9, seed=61)
    x = W.generate(w)
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    od, _ = X.xattn_dense_attn(q, k, v, causal=False)
    of, _, _ = X.xattn_forward(q, k, v, causal=False, stride=8, tau=0.9)
    ws = torch.empty(X.forward_workspace_size(X.make_dims(q, k, False), 128, 8),
                     dtype=torch.uint8, device="cuda")
    for step in range(6):
        o, _ = X.xattn_forward_scheduled(q, k, v, step, warmup_steps=warmup, causal=False,
                                         stride=8, tau=0.9, workspace=ws)
        torch.cuda.synchronize()
        assert same_bits(o, od if step < warmup else of), (warmup, step)
