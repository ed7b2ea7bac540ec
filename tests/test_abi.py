"""C ABI checks that need no GPU: the library loads, exports every entry point
include/xattn.h declares, and rejects bad arguments on the host before any
HIP call is made."""
import ctypes
import os
import re

import pytest

import paper_2503_16428_amd as X
from paper_2503_16428_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "xattn.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(xattn_[a-z_0-9]+)\s*\(", src)))


def test_header_and_binding_agree():
    decl = declared_functions()
    assert "xattn_score" in decl and "xattn_block_sparse_attn" in decl
    assert sorted(B.EXPORTS) == decl


def test_library_exports_every_declared_symbol():
    L = ctypes.CDLL(X.lib_path())
    for name in declared_functions():
        assert hasattr(L, name), name
    assert X.version() == 10100


def test_nm_shows_exports():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", X.lib_path()], capture_output=True,
                         text=True, check=True).stdout
    syms = set(re.findall(r"\bT (xattn_\w+)", out))
    assert set(declared_functions()) <= syms


def _dims(**kw):
    d = dict(batch=1, hq=4, hkv=2, seq=1024, head_dim=128, causal=1)
    d.update(kw)
    return B.Dims(**d)


def _score_ws(d, block=128, stride=8):
    n = ctypes.c_size_t(0)
    rc = X.lib().xattn_score_workspace_size(ctypes.byref(d), block, stride, ctypes.byref(n))
    return rc, n.value


@pytest.mark.parametrize("kw,code", [
    (dict(seq=1000), B.XATTN_ERR_ARG),
    (dict(hq=3, hkv=2), B.XATTN_ERR_ARG),
    (dict(hkv=0), B.XATTN_ERR_ARG),
    (dict(batch=0), B.XATTN_ERR_ARG),
    (dict(causal=2), B.XATTN_ERR_ARG),
    (dict(head_dim=64), B.XATTN_ERR_UNSUPPORTED),
    (dict(seq=128 * 2049), B.XATTN_ERR_UNSUPPORTED),
])
def test_bad_dims_are_rejected(kw, code):
    rc, _ = _score_ws(_dims(**kw))
    assert rc == code
    assert X.lib().xattn_last_error().decode()


@pytest.mark.parametrize("block,stride,code", [
    (64, 8, B.XATTN_ERR_UNSUPPORTED), (0, 8, B.XATTN_ERR_ARG), (128, 3, B.XATTN_ERR_ARG),
    (128, 0, B.XATTN_ERR_ARG), (128, 128, B.XATTN_ERR_UNSUPPORTED), (128, 256, B.XATTN_ERR_ARG),
])
def test_bad_block_or_stride(block, stride, code):
    rc, _ = _score_ws(_dims(), block, stride)
    assert rc == code


def test_workspace_sizes_cover_partials():
    d = _dims(hq=32, hkv=8, seq=131072)
    rc, n = _score_ws(d, 128, 16)
    assert rc == 0
    NR, NB, nrb, NT = 131072 // 16, 1024, 8, 131072 // 16 // 128
    # causal: partial sums for key blocks j <= b only (a packed triangle) and
    # row stats for sub-tiles starting at or before the row
    part = 32 * NB * (NB + 1) // 2 * nrb * 4
    stats = 32 * (NT * NR - 128 * NT * (NT - 1) // 2) * 8
    assert n == (part + 255) // 256 * 256 + stats
    assert n < 0.52 * (32 * NR * NB * 4 + 32 * NR * NT * 8)   # about half the square
    rc, n_full = _score_ws(_dims(hq=32, hkv=8, seq=131072, causal=0), 128, 16)
    assert rc == 0 and n_full == 32 * NR * NB * 4 + 32 * NR * NT * 8
    lay = B.forward_layout(d, 128, 16)
    assert lay["scores"] == 0 and lay["idx"] >= 32 * NB * NB * 4
    assert all(v % 256 == 0 for v in lay.values())
    assert B.forward_workspace_size(d, 128, 16) == lay["scratch"] + n


def test_calls_validate_before_launch():
    L = X.lib()
    d = _dims()
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: every case fails validation
    assert L.xattn_score(None, fake, ctypes.byref(d), 128, 8, fake, fake, 1 << 40, None) == \
        B.XATTN_ERR_ARG
    assert L.xattn_score(fake, fake, ctypes.byref(d), 128, 8, fake, None, 0, None) == \
        B.XATTN_ERR_WORKSPACE
    assert L.xattn_score(fake, fake, ctypes.byref(d), 128, 8, fake, fake, 16, None) == \
        B.XATTN_ERR_WORKSPACE
    for tau in (0.0, -1.0, float("nan")):
        assert L.xattn_select(fake, ctypes.byref(d), 128, tau, fake, fake, None) == \
            B.XATTN_ERR_ARG
    assert L.xattn_select(None, ctypes.byref(d), 128, 0.9, fake, fake, None) == B.XATTN_ERR_ARG
    assert L.xattn_block_sparse_attn(fake, fake, fake, ctypes.byref(d), 128, None, fake, fake,
                                     None, None) == B.XATTN_ERR_ARG
    assert L.xattn_dense_attn(fake, fake, None, ctypes.byref(d), fake, None, None) == \
        B.XATTN_ERR_ARG
    assert L.xattn_forward(fake, fake, fake, ctypes.byref(d), 128, 8, 0.9, fake, None, fake, 8,
                           None) == B.XATTN_ERR_WORKSPACE
    assert L.xattn_dense_attn(fake, fake, fake, None, fake, None, None) == B.XATTN_ERR_ARG
    assert L.xattn_strerror(99) == b"unknown status"


def test_per_head_selection_validates_before_launch():
    L = X.lib()
    d = _dims()                      # hq = 4
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: every case fails validation

    def arr(vals, ct):
        a = (ct * len(vals))(*vals)
        return ctypes.cast(a, ctypes.c_void_p), a

    for fn, ct, bad in ((L.xattn_select_heads, ctypes.c_float, [0.9, 0.9, 0.0, 0.9]),
                        (L.xattn_select_heads, ctypes.c_float, [0.9, float("nan"), 0.9, 0.9]),
                        (L.xattn_select_topk, ctypes.c_int32, [4, 0, 4, 4]),
                        (L.xattn_select_topk, ctypes.c_int32, [4, 4, 4, -3]),
                        (L.xattn_select_ratio, ctypes.c_float, [0.3, 0.3, -0.1, 0.3]),
                        (L.xattn_select_ratio, ctypes.c_float, [float("inf"), 0.3, 0.3, 0.3])):
        p, keep = arr(bad, ct)
        assert fn(fake, ctypes.byref(d), 128, p, fake, fake, None) == B.XATTN_ERR_ARG
        assert b"[" in L.xattn_last_error()          # names the offending head
    for fn in (L.xattn_select_heads, L.xattn_select_topk, L.xattn_select_ratio):
        assert fn(fake, ctypes.byref(d), 128, None, fake, fake, None) == B.XATTN_ERR_ARG
    big = _dims(hq=512, hkv=512)
    p, keep = arr([0.5] * 512, ctypes.c_float)
    assert L.xattn_select_heads(fake, ctypes.byref(big), 128, p, fake, fake, None) == \
        B.XATTN_ERR_UNSUPPORTED
    p, keep = arr([0.5] * 4, ctypes.c_float)
    assert L.xattn_select_ratio(None, ctypes.byref(d), 128, p, fake, fake, None) == \
        B.XATTN_ERR_ARG


def test_scheduled_forward_validates_before_launch():
    L = X.lib()
    d = _dims()
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: every case fails validation
    assert L.xattn_forward_scheduled(fake, fake, fake, ctypes.byref(d), 128, 8, 0.9, -1, 5,
                                     fake, None, None, 0, None) == B.XATTN_ERR_ARG
    assert L.xattn_forward_scheduled(fake, fake, fake, ctypes.byref(d), 128, 8, 0.9, 0, -2,
                                     fake, None, None, 0, None) == B.XATTN_ERR_ARG
    # a dense step still checks every argument of the later sparse steps
    assert L.xattn_forward_scheduled(fake, fake, fake, ctypes.byref(d), 128, 3, 0.9, 0, 5,
                                     fake, None, None, 0, None) == B.XATTN_ERR_ARG
    assert L.xattn_forward_scheduled(fake, fake, fake, ctypes.byref(d), 128, 8, 0.0, 0, 5,
                                     fake, None, None, 0, None) == B.XATTN_ERR_ARG
    assert L.xattn_forward_scheduled(fake, fake, None, ctypes.byref(d), 128, 8, 0.9, 0, 5,
                                     fake, None, None, 0, None) == B.XATTN_ERR_ARG
    # a sparse step needs the workspace
    assert L.xattn_forward_scheduled(fake, fake, fake, ctypes.byref(d), 128, 8, 0.9, 5, 5,
                                     fake, None, None, 0, None) == B.XATTN_ERR_WORKSPACE


def test_pattern_scoring_validates_before_launch():
    L = X.lib()
    d = _dims()
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: every case fails validation
    for bad in ([0, 1, 2, 3, 4, 5, 6, 6], [0, 1, 2, 3, 4, 5, 6, 8], [-1, 1, 2, 3, 4, 5, 6, 7]):
        a = (ctypes.c_int32 * 8)(*bad)
        assert L.xattn_score_pattern(fake, fake, ctypes.byref(d), 128, 8, a, fake, fake,
                                     1 << 40, None) == B.XATTN_ERR_ARG
    assert L.xattn_score_pattern(fake, fake, ctypes.byref(d), 128, 8, None, fake, fake,
                                 1 << 40, None) == B.XATTN_ERR_ARG
    a = (ctypes.c_int32 * 8)(*range(8))
    assert L.xattn_score_pattern(fake, fake, ctypes.byref(d), 128, 8, a, fake, None, 0,
                                 None) == B.XATTN_ERR_WORKSPACE


def test_noalloc_forward_validates_before_any_hip_call():
    L = X.lib()
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: every case fails validation
    d = _dims()
    assert L.xattn_forward_noalloc(fake, fake, None, ctypes.byref(d), 128, 8, 0.9, fake, None,
                                   None) == B.XATTN_ERR_ARG
    assert L.xattn_forward_noalloc(fake, fake, fake, ctypes.byref(d), 128, 8, 0.0, fake, None,
                                   None) == B.XATTN_ERR_ARG
    assert L.xattn_forward_noalloc(fake, fake, fake, ctypes.byref(d), 128, 3, 0.9, fake, None,
                                   None) == B.XATTN_ERR_ARG
    big = _dims(hq=32, hkv=8, seq=32768)
    assert L.xattn_forward_noalloc(fake, fake, fake, ctypes.byref(big), 128, 8, 0.9, fake, None,
                                   None) == B.XATTN_ERR_UNSUPPORTED
    assert b"scratch" in L.xattn_last_error()
