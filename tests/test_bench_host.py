"""Host-side logic of bench.py (no GPU): the roofline record picks the roof
below the ridge point at the kernel's arithmetic intensity, and the traffic
summary is matched by workload, kernel, stride and tau."""
import importlib.util
import os

import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_gather_bound_attention_reports_hbm(bench):
    # 656827 computed 128x128 blocks of d = 128, 64 KB of K/V each, plus Q and O
    blocks = 656827
    flops = blocks * 4.0 * 128 ** 3
    nbytes = blocks * 65536.0 + 2 * 32 * 131072 * 128 * 2
    r = bench.roofline_of("attn", {"ms": 5.5, "flops": flops, "bytes": nbytes}, 3.9e10)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["flop_per_byte"] < r["ridge_flop_per_byte"] == 312.5
    assert r["achieved"] == pytest.approx(nbytes / 5.5e-3 / 1e9, rel=1e-4)
    assert r["frac"] == pytest.approx(r["achieved"] / 8000.0, rel=1e-3)
    assert r["attainable_tflops"] == pytest.approx(r["flop_per_byte"] * 8.0, rel=1e-2)
    assert r["traffic"] == 3.9e10


def test_gemm_bound_scoring_reports_mfma(bench):
    flops, nbytes = 4.4e12, 2.0e9  # reduced GEMM: far above the ridge
    r = bench.roofline_of("score", {"ms": 4.0, "flops": flops, "bytes": nbytes}, None)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s"
    assert r["achieved"] == pytest.approx(1100.0, rel=1e-3)
    assert r["frac"] == pytest.approx(0.44, rel=1e-3)
    assert r["attainable_tflops"] == 2500.0 and r["traffic"] is None


def test_read_traffic_matches_the_configuration(bench, tmp_path):
    w = W.WORKLOADS["c3"]
    f = tmp_path / "t.txt"
    f.write_text("# comment line\n"
                 f"{w.name} attn {w.stride} {w.tau} 123\n"
                 f"{w.name} attn {w.stride * 2} {w.tau} 456\n"
                 f"{w.name} score {w.stride} {w.tau} 789\n")
    assert bench.read_traffic(str(f), w, "attn") == 123.0
    assert bench.read_traffic(str(f), w, "score") == 789.0
    assert bench.read_traffic(str(f), w, "select") is None
    assert bench.read_traffic(str(tmp_path / "missing.txt"), w, "attn") is None
