"""Host-side logic of bench.py (no GPU): the roofline record prices both
GEMM-shaped kernels against the bf16 MFMA peak (never above 1 for a real
kernel) with the measured traffic beside it, and the traffic summary is
matched by workload, kernel, stride, tau and the hash of the kernel's
sources."""
import importlib.util
import os
import shutil

import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_attention_roofline_is_mfma_on_computed_blocks(bench):
    blocks = 656827
    flops = bench.attn_flops(blocks, W.WORKLOADS["c3"])
    assert flops == blocks * 4.0 * 128 ** 3
    r = bench.roofline_of("attn", flops, 5.5, 3.9e10)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s" and r["peak"] == 2500.0
    assert r["achieved"] == pytest.approx(flops / 5.5e-3 / 1e12, rel=1e-4)
    assert r["frac"] == pytest.approx(r["achieved"] / 2500.0, rel=1e-3) and r["frac"] < 1
    assert r["traffic"] == 3.9e10
    assert r["traffic_GBps"] == pytest.approx(3.9e10 / 5.5e-3 / 1e9, rel=1e-3)
    assert r["traffic_frac_of_hbm_peak"] == pytest.approx(r["traffic_GBps"] / 8000.0, rel=1e-3)


def test_scoring_roofline_and_flops(bench):
    w = W.WORKLOADS["c3"]
    f = bench.score_flops(w)
    # (L/S)^2 * S * d * 2 FLOPs per head, halved when causal = L^2 d / S per head
    assert f == pytest.approx(131072 ** 2 * 128 / 16 * 32, rel=1e-12)
    r = bench.roofline_of("score", f, 4.0, None)
    assert r["bound"] == "mfma" and r["achieved"] == pytest.approx(f / 4e-3 / 1e12, rel=1e-4)
    assert r["traffic"] is None and "traffic_GBps" not in r
    assert bench.dense_flops(w) == pytest.approx(2.0 * 131072 ** 2 * 128 * 32, rel=1e-12)
    c5 = W.WORKLOADS["c5"]
    assert bench.dense_flops(c5) == pytest.approx(4.0 * 115200 ** 2 * 128 * 24, rel=1e-12)


def test_read_traffic_matches_configuration_and_kernel_version(bench, tmp_path):
    w = W.WORKLOADS["c3"]
    h = bench.source_hash("attn")
    f = tmp_path / "t.txt"
    f.write_text("# comment line\n"
                 f"{w.name} attn {w.stride} {w.tau} 123 {h}\n"
                 f"{w.name} attn {w.stride * 2} {w.tau} 456 {h}\n"
                 f"{w.name} score {w.stride} {w.tau} 789 0123456789ab\n"
                 f"{w.name} select {w.stride} {w.tau} 5\n")
    assert bench.read_traffic(str(f), w, "attn", h) == 123.0
    assert bench.read_traffic(str(f), w, "attn", "ffffffffffff") is None   # other version
    assert bench.read_traffic(str(f), w, "score", bench.source_hash("score")) is None
    assert bench.read_traffic(str(f), w, "select", h) is None
    assert bench.read_traffic(str(tmp_path / "missing.txt"), w, "attn", h) is None


def test_source_hash_follows_the_kernel_sources(bench, tmp_path):
    src = os.path.join(ROOT, "paper_2503_16428_amd", "csrc")
    for name in ("attn.hip", "score.hip", "common.h"):
        shutil.copy(os.path.join(src, name), tmp_path / name)
    a0, s0 = bench.source_hash("attn", str(tmp_path)), bench.source_hash("score", str(tmp_path))
    assert a0 == bench.source_hash("attn") and s0 == bench.source_hash("score")
    with open(tmp_path / "attn.hip", "a") as fh:
        fh.write("\n// edit\n")
    assert bench.source_hash("attn", str(tmp_path)) != a0
    assert bench.source_hash("score", str(tmp_path)) == s0


def test_metric_names_and_host_info(bench):
    assert bench.metric_name(W.WORKLOADS["c3"]) == \
        "ms/layer + dense-equiv TFLOP/s of scored block-sparse prefill at 128K"
    assert "32768 tokens" in bench.metric_name(W.WORKLOADS["c2"])
    ci = bench.cpu_info()
    assert ci["affinity_cpus"] == len(os.sched_getaffinity(0)) >= 1
    assert bench.median([3.0, 1.0, 2.0, 100.0, 0.5]) == 2.0


def test_more_than_one_gpu_is_refused(bench, capsys):
    with pytest.raises(SystemExit) as e:
        bench.main(["--gpus", "2"])
    assert e.value.code == 2
    assert "exactly one GPU" in capsys.readouterr().out
