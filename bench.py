#!/usr/bin/env python3
"""Benchmark of the XAttention prefill path on one MI355X.

One step = one full pass of the hot path over one layer of synthetic input:
antidiagonal scoring -> threshold selection -> block-sparse attention, all
heads. Default workload: 128K tokens, 32 query / 8 KV heads (GQA), head_dim
128, causal, B = 128, S = 16, tau = 0.9, clustered Q/K with a local key bias.

Prints ONE JSON line: ms per layer and dense-equivalent TFLOP/s (the value),
per-stage times, density, speedup over the library's own dense mode, the
roofline of the dominant kernel and the CPU oracle baseline on a sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads as W  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None, choices=sorted(W.WORKLOADS),
                    help="default c3 (c5 with --dit-schedule)")
    ap.add_argument("--stride", type=int, default=None)
    ap.add_argument("--seq", type=int, default=None,
                    help="override the workload's sequence length (a multiple of 128, at "
                         "most 262144); the name records it")
    ap.add_argument("--tau", type=float, default=None)
    ap.add_argument("--select-mode", default="threshold",
                    choices=["threshold", "heads", "topk", "ratio"],
                    help="block selection: one threshold (default), one threshold per query "
                         "head (--tau-heads), Top-K (--topk) or Top-Ratio (--ratio)")
    ap.add_argument("--tau-heads", default="0.8,0.95",
                    help="per-head thresholds spread linearly from the first to the second "
                         "value over the query heads")
    ap.add_argument("--topk", type=int, default=64, help="key blocks per row (Top-K)")
    ap.add_argument("--ratio", type=float, default=0.05,
                    help="fraction of each row's candidate blocks (Top-Ratio)")
    ap.add_argument("--pattern", default="antidiagonal",
                    choices=["antidiagonal", "diagonal", "random"],
                    help="sampling pattern inside each S x S sub-block of the scoring "
                         "(random: a permutation drawn from --pattern-seed)")
    ap.add_argument("--pattern-seed", type=int, default=1)
    ap.add_argument("--predict-thresholds", default=None, metavar="M[,A]",
                    help="before timing, predict per-head thresholds (Sec. 3.3): M 10 %% "
                         "reductions from tau over the query heads, at most A per head "
                         "(default 1); the step then selects with those thresholds")
    ap.add_argument("--sweep", action="store_true",
                    help="the 64K parameter sweep: tau in {0.8, 0.9, 0.95} x S in {4, 8, 16} "
                         "plus tau = 1 (S = 8); per point the layer time, stage times and "
                         "density; one JSON line with every point")
    ap.add_argument("--dit-schedule", default=None, metavar="T,W",
                    help="video-DiT denoising schedule: time T layer steps (step t uses "
                         "dense attention for t < W, XAttention afterwards); default "
                         "workload c5")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--dense-steps", type=int, default=3)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed region, copy a 256 MiB buffer once (a plain copy "
                         "kernel of known size, to scale rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    ap.add_argument("--cpu-rows", type=int, default=2048,
                    help="query-block rows the CPU oracle computes for the baseline")
    ap.add_argument("--traffic-file", default=os.path.join(ROOT, "profiles", "hbm_traffic.txt"),
                    help="HBM bytes per launch measured by rocprofv3 --pmc (if present)")
    return ap.parse_args()


def dev_bf16(u16):
    """uint16 bf16 bit patterns (host) -> torch bf16 device tensor."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).cuda()


def dense_flops(w) -> float:
    """4 L^2 d per head (QK^T and PV), halved when causal (diagonal halves)."""
    f = 4.0 * w.seq * w.seq * w.head_dim * w.hq * w.batch
    return f / 2 if w.causal else f


def cpu_baseline(w, x, n_rows: int):
    """The CPU oracle (fp64, OpenMP) on a bounded sample of query-block rows:
    score + select + sparse attention for those rows, reported as dense-
    equivalent TFLOP/s of the rows it processed."""
    import oracle
    NB = w.n_blocks
    rng = np.random.default_rng(12345)
    heads = rng.integers(0, w.hq * w.batch, n_rows).astype(np.int32)
    blocks = np.linspace(0, NB - 1, n_rows).round().astype(np.int32)
    t0 = time.perf_counter()
    f = oracle.forward_rows(x["q"], x["k"], x["v"], w.block, w.stride, w.tau, w.causal,
                            rows=(heads, blocks))
    dt = time.perf_counter() - t0
    kv = (blocks.astype(np.float64) + 1) if w.causal else np.full(n_rows, NB, np.float64)
    flops = float((4.0 * w.block * w.block * w.head_dim * kv).sum())
    if w.causal:
        flops -= 4.0 * w.block * w.block * w.head_dim * n_rows / 2   # half diagonal
    return {
        "value": flops / dt / 1e12, "unit": "TFLOP/s (dense-equivalent)",
        "cores": oracle.num_threads(), "kind": "oracle",
        "sample": f"{n_rows} query-block rows (random heads, blocks spread over 0..{NB - 1}) "
                  f"of the same layer: score+select+sparse attention in fp64, {dt:.1f} s",
        "seconds": dt, "rows_density": float(f["cnt"].sum() / kv.sum()),
    }


def read_traffic(path, w, kernel):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, calibrated against a copy
    kernel) from the profile summary: lines 'workload kernel stride tau bytes'.
    None if absent or taken for another configuration."""
    if not os.path.exists(path):
        return None
    for line in open(path):
        f = line.split()
        if len(f) == 5 and not line.startswith("#") and f[0] == w.name and f[1] == kernel \
                and int(f[2]) == w.stride and abs(float(f[3]) - w.tau) < 1e-9:
            return float(f[4])
    return None


def roofline_of(name, kd, traffic):
    """Roofline record of one kernel from its algorithmic work per launch
    (kd: ms, flops, bytes): the bound is the roof below the ridge point
    (peak FLOP/s / peak HBM B/s) at the kernel's arithmetic intensity."""
    ai = kd["flops"] / kd["bytes"]
    ridge = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    tflops = kd["flops"] / (kd["ms"] * 1e-3) / 1e12
    gbs = kd["bytes"] / (kd["ms"] * 1e-3) / 1e9
    if ai < ridge:
        r = {"bound": "hbm", "kernel": name, "achieved": round(gbs, 1),
             "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)}
    else:
        r = {"bound": "mfma", "kernel": name, "achieved": round(tflops, 2),
             "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(tflops / PEAK_BF16_TFLOPS, 4)}
    r.update({
        "traffic": traffic,
        "per_launch_bytes": kd["bytes"],
        "per_launch_flops": kd["flops"],
        "avg_launch_ms": round(kd["ms"], 4),
        "flop_per_byte": round(ai, 1), "ridge_flop_per_byte": round(ridge, 1),
        "achieved_tflops": round(tflops, 2),
        "attainable_tflops": round(min(PEAK_BF16_TFLOPS, ai * PEAK_HBM_GBS / 1e3), 1),
        "convention": ("computed 128x128 blocks x 4*B^2*d FLOPs (diagonal blocks in full); "
                       "bytes = 64 KB of K/V per computed block + Q + O; traffic = measured "
                       "L2-boundary bytes, below the algorithmic bytes where K/V hit in L2"
                       if name == "attn" else
                       "2 * (L/S)^2 * S*d FLOPs per head, halved when causal; bytes = Q + K "
                       "+ partial sums")})
    return r


def sweep_main(a, w, q, k, v, dims, stream):
    """Every (tau, S) point of the sweep on the same inputs: K timed steps of
    score -> select -> sparse attention each, HIP events per stage."""
    import torch
    import paper_2503_16428_amd as X
    NB = w.n_blocks
    scores = torch.empty((dims.heads, NB, NB), dtype=torch.float32, device=q.device)
    idx = torch.empty((dims.heads, NB, NB), dtype=torch.int32, device=q.device)
    cnt = torch.empty((dims.heads, NB), dtype=torch.int32, device=q.device)
    o = torch.empty_like(q)
    points = []
    dflops = dense_flops(w)
    for tau, S in W.C4_SWEEP:
        ws = torch.empty(X.score_workspace_size(dims, w.block, S), dtype=torch.uint8,
                         device=q.device)

        def step(ev=None):
            if ev is not None:
                ev[0].record(stream)
            X.xattn_score(q, k, w.causal, w.block, S, scores=scores, workspace=ws)
            if ev is not None:
                ev[1].record(stream)
            X.xattn_select(scores, dims, tau, w.block, idx=idx, cnt=cnt)
            if ev is not None:
                ev[2].record(stream)
            X.xattn_block_sparse_attn(q, k, v, idx, cnt, w.causal, w.block, o=o,
                                      want_lse=False)
            if ev is not None:
                ev[3].record(stream)

        for _ in range(a.warmup):
            step()
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(a.steps)]
        t0 = time.perf_counter()
        for i in range(a.steps):
            step(evs[i])
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / a.steps
        st = np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]),
                        e[2].elapsed_time(e[3])] for e in evs]).mean(0)
        c = cnt.cpu().numpy().astype(np.int64)
        dens = float(c.sum() / ((np.arange(1, NB + 1) if w.causal else np.full(NB, NB)).sum()
                               * dims.heads))
        points.append({"tau": tau, "stride": S, "ms_per_step": round(ms, 4),
                       "stages_ms": {"score": round(float(st[0]), 4),
                                     "select": round(float(st[1]), 4),
                                     "attn": round(float(st[2]), 4)},
                       "density": round(dens, 5),
                       "dense_equiv_tflops": round(dflops / (ms * 1e-3) / 1e12, 1)})
        print(f"# tau={tau} S={S}: {ms:.3f} ms, density {dens:.4f}", file=sys.stderr, flush=True)
    ref = next(p for p in points if p["tau"] == 0.9 and p["stride"] == w.stride)
    out = {
        "metric": "ms/layer + dense-equiv TFLOP/s of scored block-sparse prefill, 64K sweep",
        "value": ref["dense_equiv_tflops"], "unit": "TFLOP/s (dense-equivalent)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": ref["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic", "config": dict(w.describe(), sweep="tau x S; value at tau=0.9, S=8"),
        "sweep": points, "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


def schedule_main(a, w, q, k, v, dims, stream):
    """One video-DiT denoising run per T steps: layer step t runs dense
    attention for t < W and score -> select -> sparse attention afterwards
    (xattn_forward_scheduled). Warmup steps replay the schedule untimed."""
    import torch
    import paper_2503_16428_amd as X
    T, Wm = (int(t) for t in a.dit_schedule.split(","))
    o = torch.empty_like(q)
    ws = torch.empty(X.forward_workspace_size(dims, w.block, w.stride), dtype=torch.uint8,
                     device=q.device)

    def step(t):
        X.xattn_forward_scheduled(q, k, v, t % T, warmup_steps=Wm, causal=w.causal,
                                  block=w.block, stride=w.stride, tau=w.tau, o=o, workspace=ws)

    for i in range(a.warmup):
        step(i)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(a.steps)]
    t0 = time.perf_counter()
    for i in range(a.steps):
        evs[i][0].record(stream)
        step(i)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = np.array([e[0].elapsed_time(e[1]) for e in evs])
    is_dense = np.array([(i % T) < Wm for i in range(a.steps)])
    ms_step = wall * 1e3 / a.steps
    dense_ms = float(per[is_dense].mean()) if is_dense.any() else None
    sparse_ms = float(per[~is_dense].mean()) if (~is_dense).any() else None
    value = dense_flops(w) / (ms_step * 1e-3) / 1e12
    out = {
        "metric": "ms per denoising-step layer + dense-equiv TFLOP/s under the video-DiT "
                  "warm-up schedule",
        "value": round(value, 3), "unit": "TFLOP/s (dense-equivalent)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": dict(w.describe(), schedule={"denoising_steps": T, "dense_warmup": Wm}),
        "dense_step_ms": None if dense_ms is None else round(dense_ms, 4),
        "xattn_step_ms": None if sparse_ms is None else round(sparse_ms, 4),
        "speedup_vs_all_dense": (None if dense_ms is None else
                                 round(dense_ms / float(per.mean()), 3)),
        "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


def main():
    a = parse()
    if a.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; multi-GPU runs are "
                                   "not part of it (--gpus must be 1)"}), flush=True)
        sys.exit(2)
    import torch
    import paper_2503_16428_amd as X

    w = W.WORKLOADS[a.workload or ("c5" if a.dit_schedule else "c4" if a.sweep else "c3")]
    if a.seq is not None:
        w = w.with_(seq=a.seq, name=f"{w.name}_seq{a.seq}")
    if a.stride is not None:
        w = w.with_(stride=a.stride)
    if a.tau is not None:
        w = w.with_(tau=a.tau)
    NB = w.n_blocks
    t0 = time.perf_counter()
    x = W.generate(w, threads=16)
    gen_s = time.perf_counter() - t0
    print(f"# generated {w.name} in {gen_s:.1f} s", file=sys.stderr, flush=True)
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    dev = q.device
    dims = X.make_dims(q, k, w.causal)
    scores = torch.empty((dims.heads, NB, NB), dtype=torch.float32, device=dev)
    idx = torch.empty((dims.heads, NB, NB), dtype=torch.int32, device=dev)
    cnt = torch.empty((dims.heads, NB), dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    ws = torch.empty(X.score_workspace_size(dims, w.block, w.stride), dtype=torch.uint8,
                     device=dev)
    stream = torch.cuda.current_stream()
    if a.dit_schedule:
        schedule_main(a, w, q, k, v, dims, stream)
        return
    if a.sweep:
        sweep_main(a, w, q, k, v, dims, stream)
        return
    lo_hi = [float(t) for t in a.tau_heads.split(",")]
    tau_h = np.linspace(lo_hi[0], lo_hi[-1], w.hq).astype(np.float32)
    prediction = None
    if a.predict_thresholds:
        parts = [int(t) for t in a.predict_thresholds.split(",")]
        M, A = parts[0], (parts[1] if len(parts) > 1 else 1)
        t0 = time.perf_counter()
        res = X.predict_thresholds(q, k, v, M, tau0=w.tau, max_adjust=A, causal=w.causal,
                                   block=w.block, stride=w.stride)
        torch.cuda.synchronize()
        tau_h = res["tau_h"]
        a.select_mode = "heads"
        err = res["err"]
        prediction = {
            "adjustments": M, "max_per_head": A, "seconds": round(time.perf_counter() - t0, 3),
            "mean_tau": round(float(tau_h.mean()), 4),
            "mean_head_error_uniform_tau": round(float(err[:, 0].mean()), 6),
            "mean_head_error_predicted": round(float(np.mean(
                [err[h, j] for h, j in enumerate(res["adjust"])])), 6),
        }
        print(f"# predicted thresholds {tau_h.round(4).tolist()}", file=sys.stderr, flush=True)

    def select():
        if a.select_mode == "threshold":
            X.xattn_select(scores, dims, w.tau, w.block, idx=idx, cnt=cnt)
        elif a.select_mode == "heads":
            X.xattn_select_heads(scores, dims, tau_h, w.block, idx=idx, cnt=cnt)
        elif a.select_mode == "topk":
            X.xattn_select_topk(scores, dims, a.topk, w.block, idx=idx, cnt=cnt)
        else:
            X.xattn_select_ratio(scores, dims, a.ratio, w.block, idx=idx, cnt=cnt)

    qsub = W.sub_row_pairing(a.pattern, w.stride, seed=a.pattern_seed)

    def score():
        if a.pattern == "antidiagonal":
            X.xattn_score(q, k, w.causal, w.block, w.stride, scores=scores, workspace=ws)
        else:
            X.xattn_score_pattern(q, k, w.causal, w.block, w.stride, qsub, scores=scores,
                                  workspace=ws)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        score()
        if ev is not None:
            ev[1].record(stream)
        select()
        if ev is not None:
            ev[2].record(stream)
        X.xattn_block_sparse_attn(q, k, v, idx, cnt, w.causal, w.block, o=o, want_lse=False)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(a.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(a.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    print(f"# timed {a.steps} steps in {wall:.2f} s", file=sys.stderr, flush=True)
    st = np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3])]
                   for e in evs])
    ms_step = wall * 1e3 / a.steps
    t_score, t_select, t_attn = (float(v) for v in st.mean(0))

    c = cnt.cpu().numpy().astype(np.int64)
    cand = (np.arange(1, NB + 1) if w.causal else np.full(NB, NB)) * dims.heads
    density = float(c.sum() / cand.sum())
    computed_blocks = int(c.sum())
    attn_flops = computed_blocks * 4.0 * w.block * w.block * w.head_dim
    dflops = dense_flops(w)
    stage_sum = t_score + t_select + t_attn

    if a.copy_calibration:
        src = torch.ones(256 << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    dense_ms = None
    if not a.no_dense:
        X.xattn_dense_attn(q, k, v, w.causal, o=o, want_lse=False)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(a.dense_steps):
            X.xattn_dense_attn(q, k, v, w.causal, o=o, want_lse=False)
        e1.record(stream)
        torch.cuda.synchronize()
        dense_ms = e0.elapsed_time(e1) / a.dense_steps
        print(f"# dense mode {dense_ms:.2f} ms", file=sys.stderr, flush=True)

    # dominant kernel of the step and its roofline. Algorithmic work per launch:
    # attention = computed blocks x 4*B^2*d FLOPs over their K/V (2*B*d bf16 =
    # 64 KB per block, fetched per use) plus Q and O once; scoring = the reduced
    # GEMM over Q and K read once plus its partial sums. The bound is the
    # roof below the ridge point (peak FLOP/s / peak HBM B/s) at that
    # arithmetic intensity.
    NR = w.seq // w.stride
    score_flops = 2.0 * NR * NR * w.stride * w.head_dim * dims.heads
    if w.causal:
        score_flops /= 2
    q_bytes = dims.heads * w.seq * w.head_dim * 2.0
    k_bytes = dims.batch * dims.hkv * w.seq * w.head_dim * 2.0
    attn_bytes = computed_blocks * 2.0 * w.block * w.head_dim * 2 + 2 * q_bytes
    score_bytes = q_bytes + k_bytes + dims.heads * NR * NB * 4.0 * (0.5 if w.causal else 1.0)
    kernels = {
        "attn": {"ms": t_attn, "flops": attn_flops, "bytes": attn_bytes},
        "score": {"ms": t_score, "flops": score_flops, "bytes": score_bytes},
    }
    dom = max(kernels, key=lambda n: kernels[n]["ms"])
    traffic = read_traffic(a.traffic_file, w, dom)
    attn_traffic = read_traffic(a.traffic_file, w, "attn")
    roofline = roofline_of(dom, kernels[dom], traffic)

    cpu = None
    if not a.no_cpu_baseline:
        print("# cpu baseline (oracle) ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, x, a.cpu_rows)
        cpu["seconds"] = round(cpu["seconds"], 2)
        # the sample's rate extrapolated to the whole layer (same unit as value)
        cpu["extrapolated_s_per_layer"] = round(dflops / (cpu["value"] * 1e12), 2)
        cpu["value"] = round(cpu["value"], 6)

    value = dflops / (ms_step * 1e-3) / 1e12
    out = {
        "metric": "ms/layer + dense-equiv TFLOP/s of scored block-sparse prefill at 128K",
        "value": round(value, 3),
        "unit": "TFLOP/s (dense-equivalent)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": dict(w.describe(), **({} if a.pattern == "antidiagonal" else {
            "pattern": {"name": a.pattern, "qsub": qsub.tolist()}}), **({}
            if a.select_mode == "threshold" else {
            "select": {"heads": {"tau_h": [round(float(t), 4) for t in tau_h]},
                       "topk": {"k_blocks": a.topk},
                       "ratio": {"ratio": a.ratio}}[a.select_mode] | {"mode": a.select_mode}})),
        "stages_ms": {"score": round(t_score, 4), "select": round(t_select, 4),
                      "attn": round(t_attn, 4)},
        "score_select_share": round((t_score + t_select) / stage_sum, 4),
        "density": round(density, 5),
        "dense_ms": None if dense_ms is None else round(dense_ms, 3),
        "speedup_vs_dense": None if dense_ms is None else round(dense_ms / ms_step, 3),
        "attn_mfma_frac_computed_blocks": round(attn_flops / (t_attn * 1e-3) / 1e12 /
                                                PEAK_BF16_TFLOPS, 4),
        "score_mfma_frac": round(score_flops / (t_score * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        # K/V (+ Q, O) stream of the attention kernel: profiled HBM bytes per launch / time
        "attn_hbm_GBps": (None if attn_traffic is None else
                          round(attn_traffic / (t_attn * 1e-3) / 1e9, 1)),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if prediction is not None:
        out["threshold_prediction"] = prediction
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
