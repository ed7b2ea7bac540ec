"""Seeded synthetic inputs for the XAttention prefill path.

This module only draws numbers. It holds none of the method's arithmetic
(no scoring, selection or attention) and is the one piece of code that both
the GPU path's tests/benchmark and the CPU oracle consume.

The paper measures on RULER, LongBench, Video-MME and VBench with real model
activations (Sec. 4.1); none of that is available here, so five synthetic
workloads stand in for it, shaped like the paper's prefill settings:

* ``c1`` 4K tokens, one head, causal, S=8        (clustered Q/K)
* ``c2`` 32K tokens, 32 q / 8 kv heads, S=8      (clustered Q/K, Llama-3-8B GQA)
* ``c3`` 128K tokens, 32 q / 8 kv heads, S=16    (clustered Q/K + local key bias)
* ``c4`` 64K tokens, 32 q / 8 kv heads, sweep of tau x S
* ``c5`` 115,200 tokens (30 frames x 60 x 64), 24 heads, non-causal, S=16
  (Q/K = noise + a smooth 3-D positional field, video-DiT shaped)

All tensors are drawn in float32 and rounded once to bfloat16 with
round-to-nearest-even; they are returned as ``uint16`` bit patterns laid out
``[heads][seq][head_dim]`` (batch 1).

Random streams: ``numpy.random.default_rng([base, head, stream])`` with
stream 0 = cluster centres / positional field, 1 = keys, 2 = queries,
3 = values. Keys, centres and values are drawn per KV head; queries per query
head, using the centres of their KV group ``g(h) = h // (hq // hkv)``.
"""
from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HEAD_DIM = 128
BLOCK = 128
N_CENTRES = 64
CENTRE_SCALE = 3.0


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and hyper-parameters of one synthetic prefill layer."""

    name: str
    seq: int
    hq: int
    hkv: int
    causal: bool
    stride: int
    tau: float
    base_seed: int
    kind: str = "clustered"      # "clustered" | "clustered_local" | "video"
    head_dim: int = HEAD_DIM
    block: int = BLOCK
    batch: int = 1
    frames: tuple = ()           # (F, Y, X) for kind == "video"

    @property
    def n_blocks(self) -> int:
        return self.seq // self.block

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def describe(self) -> dict:
        return {
            "workload": self.name, "seq": self.seq, "hq": self.hq,
            "hkv": self.hkv, "head_dim": self.head_dim, "causal": self.causal,
            "block": self.block, "stride": self.stride, "tau": self.tau,
            "batch": self.batch, "inputs": self.kind, "seed": self.base_seed,
        }


WORKLOADS = {
    "c1": Workload("c1_4k_1h_s8", 4096, 1, 1, True, 8, 0.9, 1001),
    "c2": Workload("c2_32k_gqa32x8_s8", 32768, 32, 8, True, 8, 0.9, 2001),
    "c3": Workload("c3_128k_gqa32x8_s16_local", 131072, 32, 8, True, 16, 0.9,
                   3001, kind="clustered_local"),
    "c4": Workload("c4_64k_gqa32x8_sweep", 65536, 32, 8, True, 8, 0.9, 4001),
    "c5": Workload("c5_video_115200_24h_s16", 115200, 24, 24, False, 16, 0.9,
                   5001, kind="video", frames=(30, 60, 64)),
}

C4_SWEEP = [(tau, s) for tau in (0.8, 0.9, 0.95) for s in (4, 8, 16)] + [(1.0, 8)]


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even) -> uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(u: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(base: int, head: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([base, head, stream])


def _centres(w: Workload, g: int) -> np.ndarray:
    return (CENTRE_SCALE * _rng(w.base_seed, g, 0).standard_normal(
        (N_CENTRES, w.head_dim), dtype=np.float32)).astype(np.float32)


def _clustered_rows(w: Workload, centres: np.ndarray, head: int, stream: int) -> np.ndarray:
    rng = _rng(w.base_seed, head, stream)
    z = rng.integers(0, N_CENTRES, w.seq)
    x = rng.standard_normal((w.seq, w.head_dim), dtype=np.float32)
    x += centres[z]
    return x


def _local_bias(k: np.ndarray, window: int = 4, weight: float = 0.5) -> np.ndarray:
    """k'_j = k_j + weight * mean(k_{max(0,j-window)} .. k_{j-1}); k'_0 = k_0.

    The mean is taken over the un-biased keys."""
    L = k.shape[0]
    c = np.zeros((L + 1, k.shape[1]), dtype=np.float64)
    np.cumsum(k, axis=0, dtype=np.float64, out=c[1:])
    j = np.arange(L)
    lo = np.maximum(0, j - window)
    n = (j - lo).astype(np.float64)
    s = c[j] - c[lo]
    mean = np.zeros_like(s)
    nz = n > 0
    mean[nz] = s[nz] / n[nz, None]
    return (k + weight * mean).astype(np.float32)


def _video_field(w: Workload, head: int) -> np.ndarray:
    """Smooth 3-D positional field: sum of 16 random sinusoids over
    (frame, row, col), per-component unit variance."""
    F, Y, X = w.frames
    assert F * Y * X == w.seq
    rng = _rng(w.base_seed, head, 0)
    n_sin = 16
    amp = rng.standard_normal((n_sin, w.head_dim))
    freq = rng.uniform(0.0, 4.0, (n_sin, 3))
    phase = rng.uniform(0.0, 2.0 * math.pi, n_sin)
    f, y, x = np.meshgrid(np.arange(F) / F, np.arange(Y) / Y, np.arange(X) / X,
                          indexing="ij")
    pos = np.stack([f.ravel(), y.ravel(), x.ravel()], axis=1)       # [L, 3]
    s = np.sin(2.0 * math.pi * pos @ freq.T + phase)                # [L, 16]
    return ((s @ amp) / math.sqrt(8.0)).astype(np.float32)


def generate(w: Workload, threads: int = 8, want=("q", "k", "v")) -> dict:
    """Draw Q [hq][L][d], K and V [hkv][L][d] as bf16 bit patterns (uint16)."""
    assert w.batch == 1, "synthetic workloads are batch 1"
    group = w.hq // w.hkv
    out = {}
    if w.kind == "video":
        fields = {}

        def field(h):
            if h not in fields:
                fields[h] = _video_field(w, h)
            return fields[h]

        def qk_head(h, stream):
            x = _rng(w.base_seed, h, stream).standard_normal(
                (w.seq, w.head_dim), dtype=np.float32)
            x += 2.0 * field(h)
            return to_bf16_bits(x)

        # MHA: one field per head shared by its Q and K.
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(field, range(w.hq)))
            if "q" in want:
                out["q"] = np.stack(list(ex.map(lambda h: qk_head(h, 2), range(w.hq))))
            if "k" in want:
                out["k"] = np.stack(list(ex.map(lambda h: qk_head(h, 1), range(w.hkv))))
    else:
        with ThreadPoolExecutor(threads) as ex:
            cents = list(ex.map(lambda g: _centres(w, g), range(w.hkv)))

            def k_head(g):
                k = _clustered_rows(w, cents[g], g, 1)
                if w.kind == "clustered_local":
                    k = _local_bias(k)
                return to_bf16_bits(k)

            def q_head(h):
                return to_bf16_bits(_clustered_rows(w, cents[h // group], h, 2))

            if "q" in want:
                out["q"] = np.stack(list(ex.map(q_head, range(w.hq))))
            if "k" in want:
                out["k"] = np.stack(list(ex.map(k_head, range(w.hkv))))
    if "v" in want:
        def v_head(g):
            return to_bf16_bits(_rng(w.base_seed, g, 3).standard_normal(
                (w.seq, w.head_dim), dtype=np.float32))
        with ThreadPoolExecutor(threads) as ex:
            out["v"] = np.stack(list(ex.map(v_head, range(w.hkv))))
    return out


def small(name: str, seq: int, hq: int = 2, hkv: int = 1, causal: bool = True,
          stride: int = 8, tau: float = 0.9, seed: int = 7, kind: str = "clustered",
          frames: tuple = ()) -> Workload:
    """A reduced-size workload of the same construction (for parity tests)."""
    return Workload(name, seq, hq, hkv, causal, stride, tau, seed, kind=kind, frames=frames)


def random_bf16(shape, seed: int, scale: float = 1.0) -> np.ndarray:
    """Plain N(0, scale^2) tensor as bf16 bits (for edge-case tests)."""
    x = np.random.default_rng(seed).standard_normal(shape, dtype=np.float32) * scale
    return to_bf16_bits(x)


def random_score_rows(n_rows: int, n_blocks: int, seed: int, causal: bool = True,
                      ties: bool = False) -> tuple[np.ndarray, np.ndarray]:
    """Random non-negative float32 block-score rows, each row normalised to sum 1
    over its candidates (j <= b when causal). Returns (scores[n_rows][n_blocks],
    row_block_index[n_rows]). With ``ties`` many scores repeat exactly."""
    rng = np.random.default_rng(seed)
    b = rng.integers(0, n_blocks, n_rows) if causal else np.full(n_rows, n_blocks - 1)
    s = np.zeros((n_rows, n_blocks), dtype=np.float64)
    for r in range(n_rows):
        m = b[r] + 1 if causal else n_blocks
        if ties:
            x = rng.integers(1, 5, m).astype(np.float64)
        else:
            x = rng.gamma(0.3, 1.0, m)
        s[r, :m] = x / x.sum()
    return s.astype(np.float32), b.astype(np.int32)


def sub_row_pairing(pattern: str, stride: int, seed: int = 0) -> np.ndarray:
    """Sampling pattern inside each S x S sub-block as the query sub-row paired
    with key sub-row t: 'antidiagonal' (S-1-t), 'diagonal' (t) or 'random' (a
    permutation drawn from seed), int32."""
    if pattern == "antidiagonal":
        return np.arange(stride - 1, -1, -1, dtype=np.int32)
    if pattern == "diagonal":
        return np.arange(stride, dtype=np.int32)
    if pattern == "random":
        return np.random.default_rng(seed).permutation(stride).astype(np.int32)
    raise ValueError(f"unknown pattern {pattern!r}")
