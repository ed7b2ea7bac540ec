"""Thin ctypes binding of libxattn.so (the C ABI declared in include/xattn.h).

Argument marshalling only: tensors are torch device tensors (torch supplies
device memory and the current HIP stream); every step of the computation runs
in the library's HIP kernels. There is no fallback: if the library is missing
or no GPU is present, calls raise.

Tensor layouts (batch folded into heads when 3-D tensors are given):
  q      bf16 [batch, hq, seq, 128]  or [hq, seq, 128]
  k, v   bf16 [batch, hkv, seq, 128] or [hkv, seq, 128]
  scores fp32 [batch*hq, NB, NB]; idx int32 [batch*hq, NB, NB]; cnt int32 [batch*hq, NB]
  o      bf16 like q; lse fp32 [batch*hq, seq]
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

from . import build as _build

XATTN_OK = 0
XATTN_ERR_ARG = 1
XATTN_ERR_UNSUPPORTED = 2
XATTN_ERR_WORKSPACE = 3
XATTN_ERR_HIP = 4
BLOCK = 128

_LIB = None


class XAttnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"xattn status {status}: {msg}")
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("hq", ctypes.c_int32), ("hkv", ctypes.c_int32),
                ("seq", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("causal", ctypes.c_int32)]

    def __repr__(self):
        return (f"Dims(batch={self.batch}, hq={self.hq}, hkv={self.hkv}, seq={self.seq}, "
                f"head_dim={self.head_dim}, causal={self.causal})")

    @property
    def n_blocks(self) -> int:
        return self.seq // BLOCK

    @property
    def heads(self) -> int:
        return self.batch * self.hq


EXPORTS = [
    "xattn_score_workspace_size", "xattn_score", "xattn_score_pattern", "xattn_select",
    "xattn_select_heads",
    "xattn_select_topk", "xattn_select_ratio", "xattn_block_sparse_attn",
    "xattn_dense_attn", "xattn_forward_workspace_size", "xattn_forward_layout",
    "xattn_forward", "xattn_forward_noalloc", "xattn_forward_scheduled", "xattn_threshold_dp",
    "xattn_threshold_levels", "xattn_threshold_predict",
    "xattn_head_error_workspace_size", "xattn_head_error", "xattn_head_error_mean",
    "xattn_strerror", "xattn_last_error", "xattn_version",
]


def lib_path() -> str:
    return _build.LIB


def lib() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            raise XAttnError(XATTN_ERR_HIP, f"{_build.LIB} not built; run __graft_entry__.build()")
        L = ctypes.CDLL(_build.LIB)
        P, I, F, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        PD = ctypes.POINTER(Dims)
        PSZ = ctypes.POINTER(SZ)
        L.xattn_score_workspace_size.argtypes = [PD, I, I, PSZ]
        L.xattn_score.argtypes = [P, P, PD, I, I, P, P, SZ, P]
        L.xattn_score_pattern.argtypes = [P, P, PD, I, I, P, P, P, SZ, P]
        L.xattn_select.argtypes = [P, PD, I, F, P, P, P]
        L.xattn_select_heads.argtypes = [P, PD, I, P, P, P, P]
        L.xattn_select_topk.argtypes = [P, PD, I, P, P, P, P]
        L.xattn_select_ratio.argtypes = [P, PD, I, P, P, P, P]
        L.xattn_block_sparse_attn.argtypes = [P, P, P, PD, I, P, P, P, P, P]
        L.xattn_dense_attn.argtypes = [P, P, P, PD, P, P, P]
        L.xattn_forward_workspace_size.argtypes = [PD, I, I, PSZ]
        L.xattn_forward_layout.argtypes = [PD, I, I, PSZ, PSZ, PSZ, PSZ]
        L.xattn_forward.argtypes = [P, P, P, PD, I, I, F, P, P, P, SZ, P]
        L.xattn_forward_noalloc.argtypes = [P, P, P, PD, I, I, F, P, P, P]
        L.xattn_forward_scheduled.argtypes = [P, P, P, PD, I, I, F, I, I, P, P, P, SZ, P]
        L.xattn_threshold_dp.argtypes = [P, I, I, I, P, P]
        L.xattn_threshold_levels.argtypes = [ctypes.c_double, I, P]
        L.xattn_threshold_predict.argtypes = [P, I, I, I, ctypes.c_double, P, P, P]
        L.xattn_head_error_workspace_size.argtypes = [PD, PSZ]
        L.xattn_head_error.argtypes = [P, P, PD, P, P, SZ, P]
        L.xattn_head_error_mean.argtypes = [P, P, PD, P, P, SZ, P]
        L.xattn_strerror.argtypes = [I]
        L.xattn_strerror.restype = ctypes.c_char_p
        L.xattn_last_error.restype = ctypes.c_char_p
        L.xattn_version.restype = I
        for name in EXPORTS:
            if name not in ("xattn_strerror", "xattn_last_error", "xattn_version"):
                getattr(L, name).restype = I
        _LIB = L
    return _LIB


def _check(status: int):
    if status != XATTN_OK:
        L = lib()
        raise XAttnError(status, f"{L.xattn_strerror(status).decode()}: "
                                 f"{L.xattn_last_error().decode()}")


def make_dims(q: torch.Tensor, k: torch.Tensor, causal: bool) -> Dims:
    if q.dim() == 3:
        batch, hq, seq, d = 1, q.shape[0], q.shape[1], q.shape[2]
        hkv = k.shape[0] if k.dim() == 3 else -1
    elif q.dim() == 4:
        batch, hq, seq, d = q.shape
        hkv = k.shape[1] if k.dim() == 4 else -1
    else:
        raise XAttnError(XATTN_ERR_ARG, f"q must be 3-D or 4-D, got {tuple(q.shape)}")
    want_k = (hkv, seq, d) if q.dim() == 3 else (batch, hkv, seq, d)
    if k.dim() != q.dim() or tuple(k.shape) != want_k:
        raise XAttnError(XATTN_ERR_ARG, f"k must be [{'batch, ' if q.dim() == 4 else ''}hkv, "
                                        f"seq, head_dim] matching q {tuple(q.shape)}, got "
                                        f"{tuple(k.shape)}")
    return Dims(batch, hq, hkv, seq, d, 1 if causal else 0)


def _check_shape(t, shape, dtype, name):
    """Shape and dtype of a tensor the kernels read or write, checked before
    the device check so that a mismatch never reaches a launch."""
    if t is None:
        return
    if tuple(t.shape) != tuple(shape):
        raise XAttnError(XATTN_ERR_ARG, f"{name} must have shape {tuple(shape)}, got "
                                        f"{tuple(t.shape)}")
    if t.dtype != dtype:
        raise XAttnError(XATTN_ERR_ARG, f"{name} must be {dtype}, got {t.dtype}")


def _qkv_dims(q, k, v, causal):
    """Dims of an attention call: q, k, v bf16 with k.shape == v.shape."""
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        if t.dtype != torch.bfloat16:
            raise XAttnError(XATTN_ERR_ARG, f"{n} must be torch.bfloat16, got {t.dtype}")
    d = make_dims(q, k, causal)
    if tuple(v.shape) != tuple(k.shape):
        raise XAttnError(XATTN_ERR_ARG, f"v must have k's shape {tuple(k.shape)}, got "
                                        f"{tuple(v.shape)}")
    return d


def _on_device(**tensors):
    """Device and layout checks, after every shape check of the call."""
    for n, t in tensors.items():
        if t is not None:
            _need(t, t.dtype, n)


def _check_select_shapes(dims: Dims, block: int, scores=None, idx=None, cnt=None):
    nb = dims.seq // block if block > 0 else 0
    _check_shape(scores, (dims.heads, nb, nb), torch.float32, "scores")
    _check_shape(idx, (dims.heads, nb, nb), torch.int32, "idx")
    _check_shape(cnt, (dims.heads, nb), torch.int32, "cnt")


def _check_outputs(q, dims: Dims, o=None, lse=None):
    _check_shape(o, tuple(q.shape), torch.bfloat16, "o")
    _check_shape(lse, (dims.heads, dims.seq), torch.float32, "lse")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t: torch.Tensor, dtype, name: str):
    if not t.is_cuda:
        raise XAttnError(XATTN_ERR_ARG, f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise XAttnError(XATTN_ERR_ARG, f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise XAttnError(XATTN_ERR_ARG, f"{name} must be contiguous")


def score_workspace_size(dims: Dims, block: int, stride: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().xattn_score_workspace_size(ctypes.byref(dims), block, stride, ctypes.byref(n)))
    return n.value


def forward_workspace_size(dims: Dims, block: int, stride: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().xattn_forward_workspace_size(ctypes.byref(dims), block, stride, ctypes.byref(n)))
    return n.value


def forward_layout(dims: Dims, block: int, stride: int) -> dict:
    v = [ctypes.c_size_t(0) for _ in range(4)]
    _check(lib().xattn_forward_layout(ctypes.byref(dims), block, stride,
                                      *[ctypes.byref(x) for x in v]))
    return dict(zip(("scores", "idx", "cnt", "scratch"), (x.value for x in v)))


def _qk_dims(q, k, causal):
    for t, n in ((q, "q"), (k, "k")):
        if t.dtype != torch.bfloat16:
            raise XAttnError(XATTN_ERR_ARG, f"{n} must be torch.bfloat16, got {t.dtype}")
    return make_dims(q, k, causal)


def _check_workspace(workspace):
    if workspace is not None and (workspace.dtype != torch.uint8 or workspace.dim() != 1):
        raise XAttnError(XATTN_ERR_ARG, "workspace must be a 1-D torch.uint8 tensor")


def _workspace(workspace, nbytes, device):
    if workspace is None:
        return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)
    _check_workspace(workspace)
    _need(workspace, torch.uint8, "workspace")
    return workspace


def xattn_score(q, k, causal=True, block=BLOCK, stride=8, scores=None, workspace=None,
                stream=None):
    """Antidiagonal block scores [batch*hq, NB, NB] (fp32)."""
    d = _qk_dims(q, k, causal)
    _check_select_shapes(d, block, scores=scores)
    _check_workspace(workspace)
    _on_device(q=q, k=k, scores=scores, workspace=workspace)
    nb = d.seq // block if block > 0 else 0
    if scores is None:
        scores = torch.empty((d.heads, nb, nb), dtype=torch.float32, device=q.device)
    _need(scores, torch.float32, "scores")
    workspace = _workspace(workspace, score_workspace_size(d, block, stride), q.device)
    _check(lib().xattn_score(_ptr(q), _ptr(k), ctypes.byref(d), block, stride, _ptr(scores),
                             _ptr(workspace), workspace.numel(), _stream(stream)))
    return scores


def xattn_score_pattern(q, k, causal, block, stride, qsub, scores=None, workspace=None,
                        stream=None):
    """Block scores with the sub-block positions (qsub[t], t): qsub a permutation of
    0..stride-1 (stride-1-t is the antidiagonal of xattn_score, t the diagonal)."""
    d = _qk_dims(q, k, causal)
    _check_select_shapes(d, block, scores=scores)
    qs = np.ascontiguousarray(qsub, dtype=np.int32)
    if qs.shape != (stride,):
        raise XAttnError(XATTN_ERR_ARG, f"qsub must hold {stride} entries, got {qs.shape}")
    _check_workspace(workspace)
    _on_device(q=q, k=k, scores=scores, workspace=workspace)
    nb = d.seq // block
    if scores is None:
        scores = torch.empty((d.heads, nb, nb), dtype=torch.float32, device=q.device)
    _need(scores, torch.float32, "scores")
    workspace = _workspace(workspace, score_workspace_size(d, block, stride), q.device)
    _check(lib().xattn_score_pattern(_ptr(q), _ptr(k), ctypes.byref(d), block, stride,
                                     qs.ctypes.data_as(ctypes.c_void_p), _ptr(scores),
                                     _ptr(workspace), workspace.numel(), _stream(stream)))
    return scores


def _select_outputs(scores, dims, block, idx, cnt):
    _check_select_shapes(dims, block, scores=scores, idx=idx, cnt=cnt)
    _need(scores, torch.float32, "scores")
    nb = dims.seq // block
    if idx is None:
        idx = torch.full((dims.heads, nb, nb), -1, dtype=torch.int32, device=scores.device)
    if cnt is None:
        cnt = torch.empty((dims.heads, nb), dtype=torch.int32, device=scores.device)
    _need(idx, torch.int32, "idx")
    _need(cnt, torch.int32, "cnt")
    return idx, cnt


def xattn_select(scores, dims: Dims, tau: float, block=BLOCK, idx=None, cnt=None, stream=None):
    """find_blocks per row: (idx [H, NB, NB] int32, cnt [H, NB] int32)."""
    idx, cnt = _select_outputs(scores, dims, block, idx, cnt)
    _check(lib().xattn_select(_ptr(scores), ctypes.byref(dims), block, float(tau), _ptr(idx),
                              _ptr(cnt), _stream(stream)))
    return idx, cnt


def _per_head(values, dims, dtype):
    """Host array of dims.hq values (a scalar is repeated for every head)."""
    a = np.ascontiguousarray(np.broadcast_to(np.asarray(values, dtype=dtype), (dims.hq,)))
    return a, a.ctypes.data_as(ctypes.c_void_p)


def xattn_select_heads(scores, dims: Dims, tau_h, block=BLOCK, idx=None, cnt=None,
                       stream=None):
    """find_blocks with one threshold per query head (tau_h: dims.hq values)."""
    idx, cnt = _select_outputs(scores, dims, block, idx, cnt)
    a, p = _per_head(tau_h, dims, np.float32)
    _check(lib().xattn_select_heads(_ptr(scores), ctypes.byref(dims), block, p, _ptr(idx),
                                    _ptr(cnt), _stream(stream)))
    return idx, cnt


def xattn_select_topk(scores, dims: Dims, k_h, block=BLOCK, idx=None, cnt=None, stream=None):
    """Top-K key blocks per row (k_h: dims.hq block counts, or one for all heads)."""
    idx, cnt = _select_outputs(scores, dims, block, idx, cnt)
    a, p = _per_head(k_h, dims, np.int32)
    _check(lib().xattn_select_topk(_ptr(scores), ctypes.byref(dims), block, p, _ptr(idx),
                                   _ptr(cnt), _stream(stream)))
    return idx, cnt


def xattn_select_ratio(scores, dims: Dims, ratio_h, block=BLOCK, idx=None, cnt=None,
                       stream=None):
    """Top-Ratio: round(ratio * candidates) key blocks per row (at least one)."""
    idx, cnt = _select_outputs(scores, dims, block, idx, cnt)
    a, p = _per_head(ratio_h, dims, np.float32)
    _check(lib().xattn_select_ratio(_ptr(scores), ctypes.byref(dims), block, p, _ptr(idx),
                                    _ptr(cnt), _stream(stream)))
    return idx, cnt


def _attn_outputs(q, d, o, lse, want_lse):
    _check_outputs(q, d, o, lse)
    if o is None:
        o = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((d.heads, d.seq), dtype=torch.float32, device=q.device)
    return o, lse


def xattn_block_sparse_attn(q, k, v, idx, cnt, causal=True, block=BLOCK, o=None, lse=None,
                            want_lse=True, stream=None):
    """Attention over the listed key blocks: (o bf16 like q, lse fp32 [H, seq] or None)."""
    d = _qkv_dims(q, k, v, causal)
    _check_select_shapes(d, block, idx=idx, cnt=cnt)
    _check_outputs(q, d, o, lse)
    _on_device(q=q, k=k, v=v, idx=idx, cnt=cnt, o=o, lse=lse)
    o, lse = _attn_outputs(q, d, o, lse, want_lse)
    _check(lib().xattn_block_sparse_attn(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(d), block,
                                         _ptr(idx), _ptr(cnt), _ptr(o), _ptr(lse),
                                         _stream(stream)))
    return o, lse


def xattn_dense_attn(q, k, v, causal=True, o=None, lse=None, want_lse=True, stream=None):
    """Dense (all candidate blocks) attention, same kernel as the sparse mode."""
    d = _qkv_dims(q, k, v, causal)
    _check_outputs(q, d, o, lse)
    _on_device(q=q, k=k, v=v, o=o, lse=lse)
    o, lse = _attn_outputs(q, d, o, lse, want_lse)
    _check(lib().xattn_dense_attn(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(d), _ptr(o),
                                  _ptr(lse), _stream(stream)))
    return o, lse


def _forward_views(workspace, d, block, stride):
    lay = forward_layout(d, block, stride)
    nb = d.seq // block
    return {
        "scores": workspace[lay["scores"]:lay["scores"] + d.heads * nb * nb * 4]
        .view(torch.float32).view(d.heads, nb, nb),
        "idx": workspace[lay["idx"]:lay["idx"] + d.heads * nb * nb * 4]
        .view(torch.int32).view(d.heads, nb, nb),
        "cnt": workspace[lay["cnt"]:lay["cnt"] + d.heads * nb * 4]
        .view(torch.int32).view(d.heads, nb),
    }


def xattn_forward(q, k, v, causal=True, block=BLOCK, stride=8, tau=0.9, o=None, lse=None,
                  workspace=None, want_lse=False, stream=None):
    """score -> select -> sparse attention. Returns (o, lse, workspace views dict)."""
    d = _qkv_dims(q, k, v, causal)
    _check_outputs(q, d, o, lse)
    _check_workspace(workspace)
    _on_device(q=q, k=k, v=v, o=o, lse=lse, workspace=workspace)
    o, lse = _attn_outputs(q, d, o, lse, want_lse)
    workspace = _workspace(workspace, forward_workspace_size(d, block, stride), q.device)
    _check(lib().xattn_forward(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(d), block, stride,
                               float(tau), _ptr(o), _ptr(lse), _ptr(workspace),
                               workspace.numel(), _stream(stream)))
    return o, lse, _forward_views(workspace, d, block, stride)


def xattn_forward_noalloc(q, k, v, o, lse=None, causal=True, block=BLOCK, stride=8, tau=0.9,
                          stream=None):
    """score -> select -> sparse attention with the library's static scratch
    (no allocation by the call): the caller passes the output o (bf16 like q)
    and optionally lse (fp32 [H, seq]). Returns (o, lse)."""
    d = _qkv_dims(q, k, v, causal)
    if o is None:
        raise XAttnError(XATTN_ERR_ARG, "o must be given (the call allocates nothing)")
    _check_outputs(q, d, o, lse)
    _on_device(q=q, k=k, v=v, o=o, lse=lse)
    _check(lib().xattn_forward_noalloc(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(d), block,
                                       stride, float(tau), _ptr(o), _ptr(lse), _stream(stream)))
    return o, lse


def xattn_forward_scheduled(q, k, v, step, warmup_steps=5, causal=False, block=BLOCK,
                            stride=16, tau=0.9, o=None, lse=None, workspace=None,
                            want_lse=False, stream=None):
    """Dense attention for steps < warmup_steps, XAttention afterwards (video
    DiT schedule). Returns (o, lse); the workspace is allocated only when needed."""
    d = _qkv_dims(q, k, v, causal)
    _check_outputs(q, d, o, lse)
    _check_workspace(workspace)
    _on_device(q=q, k=k, v=v, o=o, lse=lse, workspace=workspace)
    o, lse = _attn_outputs(q, d, o, lse, want_lse)
    if workspace is not None or step >= warmup_steps:
        workspace = _workspace(workspace, forward_workspace_size(d, block, stride), q.device)
    _check(lib().xattn_forward_scheduled(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(d), block,
                                         stride, float(tau), int(step), int(warmup_steps),
                                         _ptr(o), _ptr(lse), _ptr(workspace),
                                         0 if workspace is None else workspace.numel(),
                                         _stream(stream)))
    return o, lse


def threshold_dp(perf, adjustments: int):
    """Minimum-threshold dynamic program over a per-head performance table
    perf [heads][max_adjust + 1] (host). Returns (adjust int32 [heads], best)."""
    p = np.ascontiguousarray(perf, dtype=np.float64)
    if p.ndim != 2 or p.shape[1] < 2:
        raise XAttnError(XATTN_ERR_ARG, f"perf must be [heads][max_adjust + 1], got {p.shape}")
    adj = np.zeros(p.shape[0], dtype=np.int32)
    best = ctypes.c_double(0.0)
    _check(lib().xattn_threshold_dp(p.ctypes.data_as(ctypes.c_void_p), p.shape[0],
                                    p.shape[1] - 1, int(adjustments),
                                    adj.ctypes.data_as(ctypes.c_void_p), ctypes.byref(best)))
    return adj, best.value


def threshold_levels(tau0: float, max_adjust: int) -> np.ndarray:
    """The thresholds after 0 .. max_adjust reductions of 10 % from tau0 (float32)."""
    out = np.zeros(max(int(max_adjust), 0) + 1, dtype=np.float32)
    _check(lib().xattn_threshold_levels(ctypes.c_double(tau0), int(max_adjust),
                                        out.ctypes.data_as(ctypes.c_void_p)))
    return out


def threshold_predict(err, adjustments: int, tau0: float):
    """Per-head thresholds from a per-head error table err [heads][max_adjust + 1]
    (host): the assignment of exactly `adjustments` reductions with the least
    total error. Returns (adjust int32 [heads], tau_h float32 [heads], total error)."""
    e = np.ascontiguousarray(err, dtype=np.float64)
    if e.ndim != 2 or e.shape[1] < 2:
        raise XAttnError(XATTN_ERR_ARG, f"err must be [heads][max_adjust + 1], got {e.shape}")
    adj = np.zeros(e.shape[0], dtype=np.int32)
    tau_h = np.zeros(e.shape[0], dtype=np.float32)
    best = ctypes.c_double(0.0)
    _check(lib().xattn_threshold_predict(e.ctypes.data_as(ctypes.c_void_p), e.shape[0],
                                         e.shape[1] - 1, int(adjustments), ctypes.c_double(tau0),
                                         adj.ctypes.data_as(ctypes.c_void_p),
                                         tau_h.ctypes.data_as(ctypes.c_void_p),
                                         ctypes.byref(best)))
    return adj, tau_h, best.value


def _error_dims(o, o_ref, causal):
    if o.dtype != torch.bfloat16 or o_ref.dtype != torch.bfloat16:
        raise XAttnError(XATTN_ERR_ARG, "o and o_ref must be torch.bfloat16")
    if tuple(o.shape) != tuple(o_ref.shape):
        raise XAttnError(XATTN_ERR_ARG, f"o and o_ref must have the same shape, got "
                                        f"{tuple(o.shape)} and {tuple(o_ref.shape)}")
    d = make_dims(o, o, causal)
    _need(o, torch.bfloat16, "o")
    _need(o_ref, torch.bfloat16, "o_ref")
    return d


def head_error(o, o_ref, causal=True, workspace=None, stream=None):
    """Per-head relative squared error of o against o_ref (float64 [heads] on the device)."""
    d = _error_dims(o, o_ref, causal)
    n = ctypes.c_size_t(0)
    _check(lib().xattn_head_error_workspace_size(ctypes.byref(d), ctypes.byref(n)))
    workspace = _workspace(workspace, n.value, o.device)
    err = torch.empty(d.heads, dtype=torch.float64, device=o.device)
    _check(lib().xattn_head_error(_ptr(o), _ptr(o_ref), ctypes.byref(d), _ptr(err),
                                  _ptr(workspace), workspace.numel(), _stream(stream)))
    return err


def head_error_mean(o, o_ref, causal=True, workspace=None, stream=None):
    """Per-query-head relative squared error averaged over the batch (float64 [hq])."""
    d = _error_dims(o, o_ref, causal)
    n = ctypes.c_size_t(0)
    _check(lib().xattn_head_error_workspace_size(ctypes.byref(d), ctypes.byref(n)))
    workspace = _workspace(workspace, n.value, o.device)
    err = torch.empty(d.hq, dtype=torch.float64, device=o.device)
    _check(lib().xattn_head_error_mean(_ptr(o), _ptr(o_ref), ctypes.byref(d), _ptr(err),
                                       _ptr(workspace), workspace.numel(), _stream(stream)))
    return err


def version() -> int:
    return lib().xattn_version()
