#!/usr/bin/env python3
"""Benchmark of the XAttention prefill path on one MI355X.

One step = one full pass of the hot path over one layer of synthetic input:
antidiagonal scoring -> threshold selection -> block-sparse attention, all
heads. Default workload: 128K tokens, 32 query / 8 KV heads (GQA), head_dim
128, causal, B = 128, S = 16, tau = 0.9, clustered Q/K with a local key bias.
--workload picks another of the five synthetic layers (4K single head, 32K
GQA, the 64K sweep, the 115,200-token video layer).

Timing protocol: W untimed warm-up steps; then K steps, each preceded by a
512 MB write that evicts the L2s and the Infinity Cache, each stage bracketed
by HIP events on the launch stream; the per-step and per-stage figures are
medians over the K steps. The K steps are bracketed by device synchronisation
and their wall time (flushes included) is reported beside them.

Prints ONE JSON line: ms per layer and dense-equivalent TFLOP/s (the value),
per-stage times, density, speedup over the library's own dense mode, the MFMA
roofline of the dominant kernel with its measured traffic, three probes for
context (the random-block gather rate of the attention's load pattern, a
library bf16 GEMM of the scoring's operand shapes, torch's flash attention on
the same layer), software versions, and the CPU oracle baseline on a sample.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads as W  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA (2.4 GHz)
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
FLUSH_BYTES = 512 << 20        # written before every timed step
CSRC = os.path.join(ROOT, "paper_2503_16428_amd", "csrc")
KERNEL_SOURCES = {"attn": ["attn.hip", "common.h"], "score": ["score.hip", "common.h"]}


def parse(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None, choices=sorted(W.WORKLOADS),
                    help="default c3 (c5 with --dit-schedule, c4 with --sweep)")
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
                         "plus tau = 1 (S = 8); per point the layer time, stage times, density "
                         "and MFMA rooflines; one JSON line with every point")
    ap.add_argument("--dit-schedule", default=None, metavar="T,W",
                    help="video-DiT denoising schedule: time T layer steps (step t uses "
                         "dense attention for t < W, XAttention afterwards); default "
                         "workload c5")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-flush", action="store_true",
                    help="skip the 512 MB cache-evicting write before each timed step")
    ap.add_argument("--no-probe", action="store_true",
                    help="skip the probes (random 64 KB block gather; library GEMM of the scoring "
                         "shape; the library's dense attention)")
    ap.add_argument("--dense-steps", type=int, default=3)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed region, copy a 256 MiB buffer once (a plain copy "
                         "kernel of known size, to scale rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    ap.add_argument("--cpu-rows", type=int, default=2048,
                    help="query-block rows the CPU oracle computes for the baseline")
    ap.add_argument("--traffic-file", default=os.path.join(ROOT, "profiles", "hbm_traffic.txt"),
                    help="HBM bytes per launch measured by rocprofv3 --pmc (if present)")
    return ap.parse_args(argv)


# ---------------------------------------------------------------- host logic


def dense_flops(w) -> float:
    """4 L^2 d per head (QK^T and PV), halved when causal (diagonal halves)."""
    f = 4.0 * w.seq * w.seq * w.head_dim * w.hq * w.batch
    return f / 2 if w.causal else f


def score_flops(w) -> float:
    """The reduced product of Algorithm 1: (L/S)^2 outputs of depth S*d per
    head, 2 FLOPs per multiply-add, halved when causal."""
    nr = w.seq // w.stride
    f = 2.0 * nr * nr * w.stride * w.head_dim * w.hq * w.batch
    return f / 2 if w.causal else f


def attn_flops(computed_blocks: int, w) -> float:
    """4 B^2 d per computed 128 x 128 block (QK^T and PV; diagonal blocks in full)."""
    return computed_blocks * 4.0 * w.block * w.block * w.head_dim


def source_hash(kernel: str, csrc: str = CSRC) -> str:
    """Short hash of the sources a kernel is built from: a traffic figure is
    only used while the kernel it was measured on is unchanged."""
    h = hashlib.sha1()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:12]


def read_traffic(path, w, kernel, src_hash):
    """Bytes per launch across the L2 boundary (rocprofv3 FETCH_SIZE +
    WRITE_SIZE, calibrated against a copy kernel) from the profile summary:
    lines 'workload kernel stride tau bytes source_hash'. None if absent, taken
    for another configuration, or taken on another version of the kernel."""
    if not os.path.exists(path):
        return None
    for line in open(path):
        f = line.split()
        if len(f) == 6 and not line.startswith("#") and f[0] == w.name and f[1] == kernel \
                and int(f[2]) == w.stride and abs(float(f[3]) - w.tau) < 1e-9 \
                and f[5] == src_hash:
            return float(f[4])
    return None


def roofline_of(name, flops, ms, traffic):
    """MFMA roofline record of one kernel: its algorithmic FLOPs per launch
    (computed blocks x 4 B^2 d for the attention, the reduced product for the
    scoring) over its event-timed launch duration, against the dense bf16
    peak. Beside it, the measured bytes across the L2 boundary per launch
    (rocprofv3 counters, when taken on this kernel version) as a rate and a
    fraction of the HBM peak."""
    tflops = flops / (ms * 1e-3) / 1e12
    r = {"bound": "mfma", "kernel": name, "achieved": round(tflops, 2),
         "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
         "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
         "traffic": traffic, "per_launch_flops": flops, "avg_launch_ms": round(ms, 4)}
    if traffic is not None:
        gbs = traffic / (ms * 1e-3) / 1e9
        r.update({"traffic_GBps": round(gbs, 1),
                  "traffic_frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4)})
    r["convention"] = (
        "computed 128x128 blocks x 4*B^2*d FLOPs (diagonal blocks in full); traffic = "
        "rocprofv3 FETCH_SIZE+WRITE_SIZE bytes per launch, copy-calibrated"
        if name == "attn" else
        "2*(L/S)^2*S*d FLOPs per head, halved when causal (xattn_score: partial-sum and "
        "finalize launches); traffic = rocprofv3 FETCH_SIZE+WRITE_SIZE bytes per launch")
    return r


def median(xs):
    return float(np.median(np.asarray(xs, dtype=np.float64)))


def env_info():
    """Software versions and host CPU of the run."""
    info = {}
    try:
        info["rocm"] = open("/opt/rocm/.info/version").read().strip()
    except OSError:
        info["rocm"] = None
    try:
        import torch
        info["torch"] = torch.__version__
        info["torch_hip"] = torch.version.hip
        info["device"] = torch.cuda.get_device_name(0) if torch.cuda.is_available() else None
    except Exception as e:  # noqa: BLE001
        info["torch"] = f"unavailable: {e}"
    info.update(cpu_info())
    return info


def cpu_info():
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"cpu_model": model, "affinity_cpus": len(os.sched_getaffinity(0))}


# ---------------------------------------------------------------- GPU legs


def dev_bf16(u16):
    """uint16 bf16 bit patterns (host) -> torch bf16 device tensor."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).cuda()


class Flusher:
    """A 512 MB device buffer rewritten before each timed step, so no step
    finds its inputs in the L2s or the 256 MB Infinity Cache."""

    def __init__(self, enabled):
        import torch
        self.buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.int32, device="cuda") \
            if enabled else None
        self.n = 0

    def __call__(self):
        if self.buf is not None:
            self.n += 1
            self.buf.fill_(self.n)


def time_steps(stages, steps, warmup, stream, flush):
    """Run warmup untimed steps, then `steps` timed ones (flush before each,
    HIP events around each stage on the launch stream). Returns (per-stage
    event times [steps][n_stages] in ms, wall seconds of the timed steps)."""
    import torch
    for _ in range(warmup):
        for f in stages:
            f()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)]
           for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        flush()
        evs[i][0].record(stream)
        for j, f in enumerate(stages):
            f()
            evs[i][j + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st = np.array([[e[j].elapsed_time(e[j + 1]) for j in range(len(stages))] for e in evs])
    return st, wall


def gather_probe(stream, per_wg=64, n_wg=4096, seed=7):
    """Rate of the attention kernel's K/V load pattern alone (tracked probe
    kernel, libxattn_probe.so): workgroups stream random 64 KB blocks into LDS
    with the kernel's direct-to-LDS loads. Buffers of 64 MB (one KV group's
    K+V at 128K tokens: Infinity-Cache resident) and 2 GB (HBM)."""
    import torch
    from paper_2503_16428_amd import build as B
    if not os.path.exists(B.PROBE_LIB):
        return {"error": "libxattn_probe.so not built"}
    lib = ctypes.CDLL(B.PROBE_LIB)
    lib.xattn_probe_gather.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                       ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                       ctypes.c_void_p]
    g = torch.Generator(device="cuda").manual_seed(seed)
    sink = torch.empty(n_wg, dtype=torch.int32, device="cuda")
    out = {"kernel": "gather_probe_kernel", "blocks_per_launch": per_wg * n_wg,
           "bytes_per_launch": per_wg * n_wg * 65536}
    for label, mb in (("infinity_cache_64MB", 64), ("hbm_2GB", 2048)):
        nblk = mb * 16
        buf = torch.ones(nblk * 32768, dtype=torch.bfloat16, device="cuda")
        blocks = torch.randint(0, nblk, (n_wg * per_wg,), generator=g, device="cuda",
                               dtype=torch.int32)

        def launch():
            rc = lib.xattn_probe_gather(ctypes.c_void_p(buf.data_ptr()), nblk,
                                        ctypes.c_void_p(blocks.data_ptr()), per_wg, n_wg,
                                        ctypes.c_void_p(sink.data_ptr()),
                                        ctypes.c_void_p(stream.cuda_stream))
            if rc != 0:
                raise RuntimeError(f"gather probe launch failed ({rc})")

        launch()
        torch.cuda.synchronize()
        ts = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        ms = median(ts)
        out[label] = {"ms": round(ms, 4),
                      "TBps": round(out["bytes_per_launch"] / (ms * 1e-3) / 1e12, 3)}
        del buf, blocks
    return out


def gemm_probe(stream, w, score_tflops):
    """Rate of a plain library GEMM with the reduced product's operand shapes
    (torch.matmul in bf16, served by hipBLASLt): per head, (L/S x S d) times
    (S d x L/S), the full square with a bf16 output. It measures what this
    GPU's matrix cores sustain on that shape under its power limit, as a
    practical ceiling beside the nominal peak for the scoring kernel (which
    computes the causal half and fuses the softmax epilogue instead of
    writing the product)."""
    import torch
    m, kd, heads = w.seq // w.stride, w.stride * w.head_dim, w.hq * w.batch
    g = torch.Generator(device="cuda").manual_seed(11)
    with torch.cuda.stream(stream):
        A = torch.randn((heads, m, kd), generator=g, device="cuda").to(torch.bfloat16)
        B = torch.randn((heads, kd, m), generator=g, device="cuda").to(torch.bfloat16)
        C = torch.empty((heads, m, m), device="cuda", dtype=torch.bfloat16)
        for _ in range(3):
            torch.matmul(A, B, out=C)
        torch.cuda.synchronize()
        ts = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            torch.matmul(A, B, out=C)
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
    del A, B, C
    ms = median(ts)
    tflops = 2.0 * heads * m * m * kd / (ms * 1e-3) / 1e12
    return {"op": "torch.matmul bf16 (hipBLASLt): per head (L/S x S*d) @ (S*d x L/S), "
                  "full square, bf16 output",
            "shape": [heads, m, kd, m], "ms": round(ms, 4), "TFLOPs": round(tflops, 1),
            "frac_of_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
            "score_frac_of_library": round(score_tflops / tflops, 4)}


def library_dense_probe(stream, w, q, k, v, dense_ms, ms_step, o_dense):
    """The vendor's dense attention on the same layer, for context: torch's
    scaled_dot_product_attention restricted to its flash backend (no fallback
    to the math path), K/V expanded to the query heads for GQA. Returns its
    time, rate, the speedups over it, and its largest difference from this
    library's dense output (o_dense, when given)."""
    import torch
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel
    G = w.hq // w.hkv
    try:
        with torch.cuda.stream(stream), sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
            qq = q.unsqueeze(0)
            kk = k.repeat_interleave(G, dim=0).unsqueeze(0).contiguous()
            vv = v.repeat_interleave(G, dim=0).unsqueeze(0).contiguous()
            ref = F.scaled_dot_product_attention(qq, kk, vv, is_causal=w.causal)
            torch.cuda.synchronize()
            ts = []
            for _ in range(3):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                ref = F.scaled_dot_product_attention(qq, kk, vv, is_causal=w.causal)
                e1.record(stream)
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1))
            diff = None
            if o_dense is not None:
                diff = float((ref[0].float() - o_dense.float()).abs().max().item())
            del kk, vv, ref
    except (RuntimeError, ValueError) as e:
        return {"op": "torch SDPA, flash backend", "error": f"{type(e).__name__}: {str(e)[:160]}"}
    ms = median(ts)
    tflops = dense_flops(w) / (ms * 1e-3) / 1e12
    return {"op": "torch SDPA, flash backend (K/V expanded for GQA)", "ms": round(ms, 3),
            "TFLOPs": round(tflops, 1), "frac_of_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
            "speedup_of_layer_over_it": round(ms / ms_step, 3),
            "own_dense_speedup_over_it": None if dense_ms is None else round(ms / dense_ms, 3),
            "max_abs_diff_vs_own_dense": None if diff is None else round(diff, 5)}


def cpu_baseline(w, x, n_rows: int):
    """The CPU oracle (fp64, OpenMP) on a bounded sample of query-block rows:
    score + select + sparse attention for those rows, reported as dense-
    equivalent TFLOP/s of the rows it processed."""
    import oracle
    NB = w.n_blocks
    H = w.hq * w.batch
    total = H * NB
    rng = np.random.default_rng(12345)
    if n_rows >= total:
        heads, blocks = oracle.all_rows(H, NB)
    else:
        pick = np.sort(rng.choice(total, n_rows, replace=False))
        heads, blocks = (pick // NB).astype(np.int32), (pick % NB).astype(np.int32)
    n_rows = len(heads)
    t0 = time.perf_counter()
    f = oracle.forward_rows(x["q"], x["k"], x["v"], w.block, w.stride, w.tau, w.causal,
                            rows=(heads, blocks))
    dt = time.perf_counter() - t0
    kv = (blocks.astype(np.float64) + 1) if w.causal else np.full(n_rows, NB, np.float64)
    flops = float((4.0 * w.block * w.block * w.head_dim * kv).sum())
    if w.causal:
        flops -= 4.0 * w.block * w.block * w.head_dim * n_rows / 2   # half diagonal
    ci = cpu_info()
    return {
        "value": flops / dt / 1e12, "unit": "TFLOP/s (dense-equivalent)",
        "cores": oracle.num_threads(), "kind": "oracle",
        "sample": f"{n_rows} of {total} query-block rows (distinct, seeded) of the same "
                  f"layer: score+select+sparse attention in fp64, {dt:.1f} s",
        "seconds": dt, "rows_density": float(f["cnt"].sum() / kv.sum()),
        "cpu_model": ci["cpu_model"], "affinity_cpus": ci["affinity_cpus"],
        "threads": oracle.num_threads(),
    }


def density_of(c, w, heads):
    NB = w.n_blocks
    cand = (np.arange(1, NB + 1) if w.causal else np.full(NB, NB)).sum() * heads
    return float(c.sum() / cand)


def metric_name(w):
    if w.name.startswith("c3_128k") and w.seq == 131072:
        return "ms/layer + dense-equiv TFLOP/s of scored block-sparse prefill at 128K"
    return f"ms/layer + dense-equiv TFLOP/s of scored block-sparse prefill at {w.seq} tokens"


def sweep_main(a, w, q, k, v, dims, stream, flush, x):
    """Every (tau, S) point of the sweep on the same inputs: the protocol's K
    timed steps of score -> select -> sparse attention per point, MFMA
    rooflines of both GEMM-shaped kernels per point."""
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
        wp = w.with_(tau=tau, stride=S)
        ws = torch.empty(X.score_workspace_size(dims, w.block, S), dtype=torch.uint8,
                         device=q.device)
        stages = [
            lambda: X.xattn_score(q, k, w.causal, w.block, S, scores=scores, workspace=ws),
            lambda: X.xattn_select(scores, dims, tau, w.block, idx=idx, cnt=cnt),
            lambda: X.xattn_block_sparse_attn(q, k, v, idx, cnt, w.causal, w.block, o=o,
                                              want_lse=False),
        ]
        st, wall = time_steps(stages, a.steps, a.warmup, stream, flush)
        t_score, t_select, t_attn = (median(st[:, j]) for j in range(3))
        ms = median(st.sum(1))
        c = cnt.cpu().numpy().astype(np.int64)
        blocks = int(c.sum())
        dens = density_of(c, w, dims.heads)
        tr_a = read_traffic(a.traffic_file, wp, "attn", source_hash("attn"))
        tr_s = read_traffic(a.traffic_file, wp, "score", source_hash("score"))
        points.append({
            "tau": tau, "stride": S, "ms_per_step": round(ms, 4),
            "stages_ms": {"score": round(t_score, 4), "select": round(t_select, 4),
                          "attn": round(t_attn, 4)},
            "density": round(dens, 5),
            "dense_equiv_tflops": round(dflops / (ms * 1e-3) / 1e12, 1),
            "score_select_share": round((t_score + t_select) / (t_score + t_select + t_attn), 4),
            "roofline_attn": roofline_of("attn", attn_flops(blocks, w), t_attn, tr_a),
            "roofline_score": roofline_of("score", score_flops(wp), t_score, tr_s)})
        print(f"# tau={tau} S={S}: {ms:.3f} ms, density {dens:.4f}", file=sys.stderr, flush=True)
    ref = next(p for p in points if p["tau"] == 0.9 and p["stride"] == w.stride)
    dom = "attn" if ref["stages_ms"]["attn"] >= ref["stages_ms"]["score"] else "score"
    cpu = None
    if not a.no_cpu_baseline:
        print("# cpu baseline (oracle) ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, x, a.cpu_rows)
        cpu["seconds"] = round(cpu["seconds"], 2)
        cpu["value"] = round(cpu["value"], 6)
    out = {
        "metric": "ms/layer + dense-equiv TFLOP/s of scored block-sparse prefill, 64K sweep",
        "value": ref["dense_equiv_tflops"], "unit": "TFLOP/s (dense-equivalent)",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": ref["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": dict(w.describe(), sweep="tau x S; value at tau=0.9, S=8"),
        "protocol": protocol_note(a), "env": env_info(),
        "sweep": points, "roofline": ref[f"roofline_{dom}"], "cpu_baseline": cpu,
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
    dense_ms = float(np.median(per[is_dense])) if is_dense.any() else None
    sparse_ms = float(np.median(per[~is_dense])) if (~is_dense).any() else None
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
        "env": env_info(), "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


def protocol_note(a):
    return (f"{a.warmup} untimed warm-up steps; {a.steps} timed steps, each after a "
            f"{'512 MB cache-evicting write' if not a.no_flush else 'no flush'}; HIP events "
            f"per stage on the launch stream; medians over the timed steps")


def main(argv=None):
    a = parse(argv)
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
    print(f"# generated {w.name} in {time.perf_counter() - t0:.1f} s", file=sys.stderr,
          flush=True)
    q, k, v = (dev_bf16(x[n]) for n in "qkv")
    dev = q.device
    dims = X.make_dims(q, k, w.causal)
    stream = torch.cuda.current_stream()
    flush = Flusher(not a.no_flush)
    if a.dit_schedule:
        schedule_main(a, w, q, k, v, dims, stream)
        return
    if a.sweep:
        sweep_main(a, w, q, k, v, dims, stream, flush, x)
        return
    scores = torch.empty((dims.heads, NB, NB), dtype=torch.float32, device=dev)
    idx = torch.empty((dims.heads, NB, NB), dtype=torch.int32, device=dev)
    cnt = torch.empty((dims.heads, NB), dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    ws = torch.empty(X.score_workspace_size(dims, w.block, w.stride), dtype=torch.uint8,
                     device=dev)
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

    def attend():
        X.xattn_block_sparse_attn(q, k, v, idx, cnt, w.causal, w.block, o=o, want_lse=False)

    # the step: xattn_forward (scoring, selection, attention in one call) where
    # it applies (one threshold, antidiagonal pattern); the stage times come
    # from the same kernels launched as three separate calls
    one_call = a.select_mode == "threshold" and a.pattern == "antidiagonal"
    if one_call:
        fws = torch.empty(X.forward_workspace_size(dims, w.block, w.stride), dtype=torch.uint8,
                          device=dev)
        of = torch.empty_like(q)

        def forward():
            X.xattn_forward(q, k, v, w.causal, w.block, w.stride, w.tau, o=of, workspace=fws)

    st, _ = time_steps([score, select, attend], a.steps, a.warmup, stream, flush)
    t_score, t_select, t_attn = (median(st[:, j]) for j in range(3))
    if one_call:
        stf, wall = time_steps([forward], a.steps, a.warmup, stream, flush)
        ms_step = median(stf[:, 0])
        mean_step = float(stf[:, 0].mean())
    else:
        st, wall = time_steps([score, select, attend], a.steps, 0, stream, flush)
        ms_step = median(st.sum(1))
        mean_step = float(st.sum(1).mean())
    print(f"# timed {a.steps} steps in {wall:.2f} s", file=sys.stderr, flush=True)

    c = cnt.cpu().numpy().astype(np.int64)
    density = density_of(c, w, dims.heads)
    computed_blocks = int(c.sum())
    a_flops = attn_flops(computed_blocks, w)
    s_flops = score_flops(w)
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
        dense = [lambda: X.xattn_dense_attn(q, k, v, w.causal, o=o, want_lse=False)]
        dst_, _ = time_steps(dense, a.dense_steps, 1, stream, flush)
        dense_ms = median(dst_[:, 0])
        print(f"# dense mode {dense_ms:.2f} ms", file=sys.stderr, flush=True)

    probe = gemm = libdense = None
    if not a.no_probe:
        probe = gather_probe(stream)
        gemm = gemm_probe(stream, w, s_flops / (t_score * 1e-3) / 1e12)
        libdense = library_dense_probe(stream, w, q, k, v, dense_ms, ms_step,
                                       None if dense_ms is None else o)

    # dominant kernel of the step and its MFMA roofline (both GEMM-shaped
    # kernels are priced against the bf16 peak; the measured traffic sits
    # beside the attention's)
    kernels = {"attn": (a_flops, t_attn), "score": (s_flops, t_score)}
    dom = max(kernels, key=lambda n: kernels[n][1])
    traffic = read_traffic(a.traffic_file, w, dom, source_hash(dom))
    roofline = roofline_of(dom, kernels[dom][0], kernels[dom][1], traffic)
    other = "score" if dom == "attn" else "attn"
    other_traffic = read_traffic(a.traffic_file, w, other, source_hash(other))

    cpu = None
    if not a.no_cpu_baseline:
        print("# cpu baseline (oracle) ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, x, a.cpu_rows)
        cpu["seconds"] = round(cpu["seconds"], 2)
        cpu["extrapolated_s_per_layer"] = round(dflops / (cpu["value"] * 1e12), 2)
        cpu["value"] = round(cpu["value"], 6)

    value = dflops / (ms_step * 1e-3) / 1e12
    out = {
        "metric": metric_name(w),
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
        "protocol": protocol_note(a),
        "step": ("xattn_forward" if one_call
                 else "xattn_score / xattn_select* / xattn_block_sparse_attn"),
        "wall_ms_per_step_incl_flush": round(wall * 1e3 / a.steps, 4),
        "mean_ms_per_step": round(mean_step, 4),
        "stages_ms": {"score": round(t_score, 4), "select": round(t_select, 4),
                      "attn": round(t_attn, 4)},
        "stages_sum_ms": round(stage_sum, 4),
        "score_select_share": round((t_score + t_select) / stage_sum, 4),
        "density": round(density, 5),
        "computed_blocks": computed_blocks,
        "dense_ms": None if dense_ms is None else round(dense_ms, 3),
        "speedup_vs_dense": None if dense_ms is None else round(dense_ms / ms_step, 3),
        "attn_mfma_frac_computed_blocks": round(a_flops / (t_attn * 1e-3) / 1e12 /
                                                PEAK_BF16_TFLOPS, 4),
        "score_mfma_frac": round(s_flops / (t_score * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "roofline": roofline,
        "roofline_other": roofline_of(other, kernels[other][0], kernels[other][1],
                                      other_traffic),
        "gather_probe": probe,
        "gemm_probe": gemm,
        "library_dense": libdense,
        "env": env_info(),
        "cpu_baseline": cpu,
    }
    if prediction is not None:
        out["threshold_prediction"] = prediction
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
