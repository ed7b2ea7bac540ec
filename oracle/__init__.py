"""XAttention CPU oracle -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import this package. The GPU library never uses it:
the oracle is an independent fp64 C implementation of the paper's definitions
(Sec. 3.2, Algorithm 1, Fig. 1), see ``xattn_oracle.c`` for the readings it
takes where the paper is silent.

Pins (checked by the CPU tests against brute force, closed forms, invariants
and library routines, never against the oracle itself):
  score_rows      -- antidiagonal index walk over the full fp64 Q K^T, S=1 ==
                     exact block mass of softmax(QK^T/sqrt d), key-shift
                     invariance, zero-query closed form, Fig. 1 geometry.
  select_rows     -- subset enumeration of find_blocks, tau monotonicity,
                     tau=1 selects every candidate.
  sparse/dense    -- textbook masked softmax attention (torch fp64 CPU SDPA and
                     numpy), zero-query closed form.
  block_mass_rows -- (diagnostic) numpy softmax block sums.
  select_topk/ratio_rows -- upper set of the find_blocks order, brute-force
                     maximal mass, equality with find_blocks at its count,
                     hand-derived ratio counts.
  score_pattern_rows -- brute-force walk over the logits masked by the
                     sub-block permutation; antidiagonal == score_rows.
  threshold_dp    -- (thresholds.py) enumeration of every adjustment
                     assignment, top-M gains for one adjustment per head.

Array conventions: bf16 tensors are uint16 bit patterns [heads][seq][d];
a "row" is one (query head, query block) pair.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None


class _Dims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("hq", ctypes.c_int32),
                ("hkv", ctypes.c_int32), ("seq", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("causal", ctypes.c_int32)]


def lib():
    """Load liboracle.so (built by ``oracle/build.py``; built here if absent)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        P = ctypes.c_void_p
        i = ctypes.c_int
        L.oracle_num_threads.restype = i
        L.oracle_score_rows.argtypes = [P, P, P, i, i, i, P, P, P]
        L.oracle_select_rows.argtypes = [P, i, i, i, P, ctypes.c_float, P, P]
        L.oracle_select_topk_rows.argtypes = [P, i, i, i, P, P, P, P]
        L.oracle_score_pattern_rows.argtypes = [P, P, P, i, i, P, i, P, P, P]
        L.oracle_select_ratio_rows.argtypes = [P, i, i, i, P, P, P, P]
        L.oracle_sparse_attn_rows.argtypes = [P, P, P, P, i, i, P, P, P, i, P, P, P]
        L.oracle_dense_attn_rows.argtypes = [P, P, P, P, i, i, P, P, P, P]
        L.oracle_block_mass_rows.argtypes = [P, P, P, i, i, i, P, P, P, P]
        _LIB = L
    return _LIB


def num_threads() -> int:
    return lib().oracle_num_threads()


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    assert a.dtype == np.uint16, "bf16 tensors are passed as uint16 bit patterns"
    return a


def _dims(q, k, causal, batch=1):
    hq, L, D = q.shape[0] // batch, q.shape[1], q.shape[2]
    hkv = k.shape[0] // batch
    return _Dims(batch, hq, hkv, L, D, 1 if causal else 0)


def all_rows(n_heads: int, n_blocks: int):
    h, b = np.meshgrid(np.arange(n_heads), np.arange(n_blocks), indexing="ij")
    return h.ravel().astype(np.int32), b.ravel().astype(np.int32)


def _rows(rows, q, B):
    if rows is None:
        return all_rows(q.shape[0], q.shape[1] // B)
    rh, rb = rows
    return (np.ascontiguousarray(rh, dtype=np.int32),
            np.ascontiguousarray(rb, dtype=np.int32))


def score_rows(q, k, B, S, causal=True, rows=None, batch=1):
    """Antidiagonal block scores (fp64) of the given (head, query block) rows."""
    q, k = _u16(q), _u16(k)
    d = _dims(q, k, causal, batch)
    assert d.seq % B == 0 and B % S == 0
    rh, rb = _rows(rows, q, B)
    out = np.zeros((len(rh), d.seq // B), dtype=np.float64)
    lib().oracle_score_rows(_ptr(q), _ptr(k), ctypes.byref(d), B, S, len(rh),
                            _ptr(rh), _ptr(rb), _ptr(out))
    return out


def score_pattern_rows(q, k, B, S, qsub, causal=True, rows=None, batch=1):
    """Block scores with the sub-block positions (qsub[t], t) instead of the
    antidiagonal (qsub = S-1-t reproduces score_rows)."""
    q, k = _u16(q), _u16(k)
    d = _dims(q, k, causal, batch)
    assert d.seq % B == 0 and B % S == 0
    qs = np.ascontiguousarray(qsub, dtype=np.int32)
    assert sorted(qs.tolist()) == list(range(S)), "qsub must be a permutation of 0..S-1"
    rh, rb = _rows(rows, q, B)
    out = np.zeros((len(rh), d.seq // B), dtype=np.float64)
    lib().oracle_score_pattern_rows(_ptr(q), _ptr(k), ctypes.byref(d), B, S, _ptr(qs),
                                    len(rh), _ptr(rh), _ptr(rb), _ptr(out))
    return out


def select_rows(scores, row_b, tau, causal=True):
    """find_blocks on score rows. Returns (idx [n][NB] int32, -1 padded; cnt [n])."""
    s = np.ascontiguousarray(scores, dtype=np.float64)
    rb = np.ascontiguousarray(row_b, dtype=np.int32)
    n, NB = s.shape
    idx = np.full((n, NB), -1, dtype=np.int32)
    cnt = np.zeros(n, dtype=np.int32)
    lib().oracle_select_rows(_ptr(s), NB, 1 if causal else 0, n, _ptr(rb),
                             ctypes.c_float(tau), _ptr(idx), _ptr(cnt))
    return idx, cnt


def select_heads_rows(scores, row_h, row_b, tau_h, hq, causal=True):
    """find_blocks with a threshold per query head: row i uses tau_h[row_h[i] % hq]."""
    s = np.ascontiguousarray(scores, dtype=np.float64)
    row_h = np.asarray(row_h)
    n, NB = s.shape
    idx = np.full((n, NB), -1, dtype=np.int32)
    cnt = np.zeros(n, dtype=np.int32)
    for hh in np.unique(row_h % hq):
        sel = np.nonzero(row_h % hq == hh)[0]
        i2, c2 = select_rows(s[sel], np.asarray(row_b)[sel], float(np.float32(tau_h[hh])), causal)
        idx[sel], cnt[sel] = i2, c2
    return idx, cnt


def select_topk_rows(scores, row_b, k_row, causal=True):
    """The k_row[i] first candidates of row i in (mass desc, j asc) order."""
    s = np.ascontiguousarray(scores, dtype=np.float64)
    rb = np.ascontiguousarray(row_b, dtype=np.int32)
    n, NB = s.shape
    kr = np.ascontiguousarray(np.broadcast_to(np.asarray(k_row, dtype=np.int32), (n,)))
    idx = np.full((n, NB), -1, dtype=np.int32)
    cnt = np.zeros(n, dtype=np.int32)
    lib().oracle_select_topk_rows(_ptr(s), NB, 1 if causal else 0, n, _ptr(rb), _ptr(kr),
                                  _ptr(idx), _ptr(cnt))
    return idx, cnt


def select_ratio_rows(scores, row_b, ratio_row, causal=True):
    """Top-Ratio: round(ratio * candidates) blocks per row (at least one)."""
    s = np.ascontiguousarray(scores, dtype=np.float64)
    rb = np.ascontiguousarray(row_b, dtype=np.int32)
    n, NB = s.shape
    rr = np.ascontiguousarray(np.broadcast_to(np.asarray(ratio_row, dtype=np.float32), (n,)))
    idx = np.full((n, NB), -1, dtype=np.int32)
    cnt = np.zeros(n, dtype=np.int32)
    lib().oracle_select_ratio_rows(_ptr(s), NB, 1 if causal else 0, n, _ptr(rb), _ptr(rr),
                                   _ptr(idx), _ptr(cnt))
    return idx, cnt


def sparse_attn_rows(q, k, v, B, idx, cnt, causal=True, rows=None, batch=1):
    """Attention of query blocks over their selected key blocks (fp64)."""
    q, k, v = _u16(q), _u16(k), _u16(v)
    d = _dims(q, k, causal, batch)
    rh, rb = _rows(rows, q, B)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    cnt = np.ascontiguousarray(cnt, dtype=np.int32)
    assert idx.shape[0] == len(rh) and cnt.shape[0] == len(rh)
    o = np.zeros((len(rh), B, d.head_dim), dtype=np.float64)
    lse = np.zeros((len(rh), B), dtype=np.float64)
    lib().oracle_sparse_attn_rows(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(d), B,
                                  len(rh), _ptr(rh), _ptr(rb), _ptr(idx),
                                  idx.shape[1], _ptr(cnt), _ptr(o), _ptr(lse))
    return o, lse


def dense_attn_rows(q, k, v, B, causal=True, rows=None, batch=1):
    """Full causal (or bidirectional) attention of query blocks (fp64)."""
    q, k, v = _u16(q), _u16(k), _u16(v)
    d = _dims(q, k, causal, batch)
    rh, rb = _rows(rows, q, B)
    o = np.zeros((len(rh), B, d.head_dim), dtype=np.float64)
    lse = np.zeros((len(rh), B), dtype=np.float64)
    lib().oracle_dense_attn_rows(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(d), B,
                                 len(rh), _ptr(rh), _ptr(rb), _ptr(o), _ptr(lse))
    return o, lse


def block_mass_rows(q, k, B, S, causal=True, rows=None, batch=1):
    """Diagnostics: exact softmax block mass and antidiagonal probability mass."""
    q, k = _u16(q), _u16(k)
    d = _dims(q, k, causal, batch)
    rh, rb = _rows(rows, q, B)
    tm = np.zeros((len(rh), d.seq // B), dtype=np.float64)
    am = np.zeros_like(tm)
    lib().oracle_block_mass_rows(_ptr(q), _ptr(k), ctypes.byref(d), B, S, len(rh),
                                 _ptr(rh), _ptr(rb), _ptr(tm), _ptr(am))
    return tm, am


def forward_rows(q, k, v, B, S, tau, causal=True, rows=None, batch=1):
    """Score -> select -> sparse attention for the given rows, all in fp64."""
    rh, rb = _rows(rows, q, B)
    sc = score_rows(q, k, B, S, causal, (rh, rb), batch)
    idx, cnt = select_rows(sc, rb, tau, causal)
    o, lse = sparse_attn_rows(q, k, v, B, idx, cnt, causal, (rh, rb), batch)
    return {"scores": sc, "idx": idx, "cnt": cnt, "o": o, "lse": lse}


from .thresholds import (  # noqa: E402,F401
    head_errors, threshold_dp, thresholds_from_adjustments,
)
