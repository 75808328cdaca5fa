"""The C-ABI library loads and exports what include/*.h declare (no GPU).

Only host-side argument validation is exercised here: every call below
returns before any HIP runtime call is made.
"""
import ctypes
import glob
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def declared_functions():
    names = []
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names += re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "while")))


@pytest.fixture(scope="module")
def L():
    import paper_2604_22312_amd as g
    if not os.path.exists(g.library_path()):
        from paper_2604_22312_amd import build
        build.build()
    return g.lib()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("gvr_topk", "radix_topk", "gvr_topk_ex", "radix_topk_ex", "gvr_topk_ex_noalloc",
              "gvr_workspace_size", "gvr_topk_ex_ws", "radix_topk_ex_ws", "gvr_status_string", "gvr_version", "gvr_rope_params_default", "gvr_rope_g",
              "gvr_rope_prior", "gvr_indexer_scores", "gvr_indexer_topk"):
        assert n in names, n


def test_every_declared_symbol_is_exported(L):
    for n in declared_functions():
        assert hasattr(L, n), "symbol %s missing from libgvr_topk.so" % n


def test_status_strings(L):
    import paper_2604_22312_amd as g
    for code in (0, -1, -2, -3, -4, -5):
        assert g.status_string(code) and "unknown" not in g.status_string(code)
    assert "unknown" in g.status_string(-99)
    assert "gfx950" in g.version()


def _call(L, B, ld, K, scores=1, out=1):
    vp = ctypes.c_void_p
    return L.gvr_topk(vp(scores) if scores else None, B, ld, None, None, K,
                      vp(out) if out else None, None)


def test_host_side_validation(L):
    # K out of range -> UNSUPPORTED_K (checked first)
    assert _call(L, 4, 100, 0) == -2
    assert _call(L, 4, 100, 2049) == -2
    assert L.radix_topk(None, 4, 100, None, None, 0, None, None) == -2
    # negative sizes -> INVALID_ARG
    assert _call(L, -1, 100, 16) == -1
    assert _call(L, 4, -1, 16) == -1
    # NULL required pointers with B > 0 -> INVALID_ARG
    assert _call(L, 4, 100, 16, scores=0) == -1
    assert _call(L, 4, 100, 16, out=0) == -1
    # B == 0 is a no-op (nothing touched, not even the pointers)
    assert _call(L, 0, 100, 16, scores=0, out=0) == 0
    # absurd stride -> TOO_LONG
    assert _call(L, 1, 1 << 40, 16) == -5


def test_options_validation(L):
    import paper_2604_22312_amd as g
    vp = ctypes.c_void_p
    bad = [g.Options(capacity=100, flags=0, parts=0, reserved1=0),      # capacity < K
           g.Options(capacity=0, flags=48, parts=0, reserved1=0),       # two workgroup shapes forced
           g.Options(capacity=0, flags=80, parts=0, reserved1=0),       # two workgroup shapes forced
           g.Options(capacity=0, flags=96, parts=0, reserved1=0),       # two workgroup shapes forced
           g.Options(capacity=0, flags=112, parts=0, reserved1=0),      # three workgroup shapes forced
           g.Options(capacity=0, flags=256, parts=0, reserved1=0),      # unknown flag bit
           g.Options(capacity=0, flags=0, parts=0, reserved1=1),        # reserved field set
           g.Options(capacity=0, flags=0, parts=17, reserved1=0),       # too many parts
           g.Options(capacity=0, flags=0, parts=-1, reserved1=0),       # negative parts
           g.Options(capacity=20000, flags=0, parts=0, reserved1=0)]    # capacity > max
    for opt in bad:
        assert L.gvr_topk_ex(vp(1), 2, 100, None, None, 128, vp(1), None, ctypes.byref(opt), None) == -1
        assert L.radix_topk_ex(vp(1), 2, 100, None, 128, vp(1), None, ctypes.byref(opt), None) == -1
        assert L.gvr_topk_ex_noalloc(vp(1), 2, 100, None, None, 128, vp(1), None, ctypes.byref(opt), None) == -1
    # the allocation-free entry point checks its arguments like gvr_topk_ex
    assert L.gvr_topk_ex_noalloc(vp(1), 2, 100, None, None, 0, vp(1), None, None, None) == -2
    assert L.gvr_topk_ex_noalloc(None, 2, 100, None, None, 16, vp(1), None, None, None) == -1
    assert L.gvr_topk_ex_noalloc(None, 0, 100, None, None, 16, None, None, None, None) == 0


def test_caller_workspace_validation(L):
    """The caller-workspace calls check sizes and options like gvr_topk_ex,
    then the workspace pointer, all before touching the device."""
    import paper_2604_22312_amd as g
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    ok = g.Options(capacity=0, flags=0, parts=0, reserved1=0)
    bad = g.Options(capacity=0, flags=0, parts=17, reserved1=0)
    for f in (lambda *a: L.gvr_topk_ex_ws(vp(1), 2, 100, None, None, *a),
              lambda *a: L.radix_topk_ex_ws(vp(1), 2, 100, None, *a)):
        assert f(0, vp(1), None, None, None, None, 0) == -2                     # K out of range
        assert f(16, vp(1), None, ctypes.byref(bad), None, None, 0) == -1      # bad option
        assert f(16, vp(1), None, ctypes.byref(ok), None, None, 4096) == -1    # NULL workspace, bytes > 0
        assert f(16, vp(1), None, ctypes.byref(ok), None, vp(4100), 4096) == -1   # misaligned workspace
    assert L.gvr_topk_ex_ws(None, 2, 100, None, None, 16, vp(1), None, None, None, None, 0) == -1
    assert L.gvr_topk_ex_ws(None, 0, 100, None, None, 16, None, None, None, None, None, 0) == 0
    n = sz(123)
    assert L.gvr_workspace_size(0, 100, 16, 1, None, ctypes.byref(n)) == 0 and n.value == 0
    assert L.gvr_workspace_size(2, 100, 16, 1, None, None) == -1
    assert L.gvr_workspace_size(2, 100, 0, 1, None, ctypes.byref(n)) == -2
    assert L.gvr_workspace_size(-1, 100, 16, 1, None, ctypes.byref(n)) == -1
    assert L.gvr_workspace_size(2, 1 << 40, 16, 0, None, ctypes.byref(n)) == -5
    assert L.gvr_workspace_size(2, 100, 16, 1, ctypes.byref(bad), ctypes.byref(n)) == -1


def test_read_floor_validation(L):
    vp = ctypes.c_void_p
    assert L.gvr_read_floor(None, 0, 100, None, None, None) == 0
    assert L.gvr_read_floor(vp(1), -1, 100, None, vp(1), None) == -1
    assert L.gvr_read_floor(vp(1), 2, -1, None, vp(1), None) == -1
    assert L.gvr_read_floor(None, 2, 100, None, vp(1), None) == -1
    assert L.gvr_read_floor(vp(1), 2, 100, None, None, None) == -1
    assert L.gvr_read_floor(vp(1), 2, 1 << 40, None, vp(1), None) == -5


def test_python_binding_refuses_cpu_tensors():
    import torch
    import paper_2604_22312_amd as g
    with pytest.raises(ValueError):
        g.gvr_topk(torch.zeros(2, 10), None, None, 4)


def test_rope_defaults_and_validation(L):
    import paper_2604_22312_amd as g
    vp = ctypes.c_void_p
    p = g.gvr_rope_params()
    assert (p.d_rope, p.orig_ctx, p.base, p.scale, p.beta_fast, p.beta_slow) == (64, 4096, 1e4, 40.0, 32.0, 1.0)
    bad = [dict(d_rope=63), dict(d_rope=0), dict(d_rope=514), dict(orig_ctx=0), dict(base=1.0),
           dict(base=math.inf), dict(scale=0.0), dict(scale=math.nan), dict(beta_fast=-1.0),
           dict(beta_slow=0.0)]
    for kw in bad:
        q = g.gvr_rope_params(**kw)
        assert L.gvr_rope_g(10, ctypes.byref(q), vp(1), None, None) == -1, kw
        assert L.gvr_rope_prior(10, 16, ctypes.byref(q), vp(1), vp(1), None) == -1, kw
    assert L.gvr_rope_g(-1, None, vp(1), None, None) == -1
    assert L.gvr_rope_g(10, None, None, None, None) == -1          # g NULL with n > 0
    assert L.gvr_rope_g(0, None, None, None, None) == 0            # nothing to do
    assert L.gvr_rope_g(1 << 31, None, vp(1), None, None) == -5
    assert L.gvr_rope_prior(10, 0, None, vp(1), vp(1), None) == -2
    assert L.gvr_rope_prior(10, 2049, None, vp(1), vp(1), None) == -2
    assert L.gvr_rope_prior(10, 16, None, vp(1), None, None) == -1  # out NULL
    assert L.gvr_rope_prior(1 << 31, 16, None, vp(1), vp(1), None) == -5


def test_rope_binding_refuses_cpu_device():
    import paper_2604_22312_amd as g
    with pytest.raises(ValueError):
        g.gvr_rope_prior(100, 16, device="cpu")


def test_indexer_validation(L):
    vp = ctypes.c_void_p
    a = vp(256)   # 16-byte aligned stand-in; no call below reaches the GPU
    def call(B=4, H=64, D=128, group=2, ld=100, q=a, k=a, out=a):
        return L.gvr_indexer_scores(q, a, k, a, B, H, D, group, ld, None, out, None)
    assert call(B=-1) == -1 and call(ld=-1) == -1
    assert call(H=48) == -1 and call(H=256) == -1 and call(D=96) == -1
    assert call(group=0) == -1 and call(group=5) == -1 and call(B=5, group=2) == -1
    assert call(q=None) == -1 and call(out=None) == -1
    assert call(q=vp(257)) == -1 and call(k=vp(264)) == -1      # not 16-byte aligned
    assert call(ld=1 << 31) == -5
    assert call(B=0) == 0 and call(ld=0) == 0
    # the combined call checks K and the Top-K options first
    assert L.gvr_indexer_topk(a, a, a, a, 4, 64, 128, 2, 100, None, a, None, 0, a, None, None, None) == -2
    assert L.gvr_indexer_topk(a, a, a, a, 4, 64, 128, 2, 100, None, a, None, 2049, a, None, None, None) == -2
    import paper_2604_22312_amd as g
    bad = g.Options(capacity=0, flags=256, parts=0, reserved1=0)
    assert L.gvr_indexer_topk(a, a, a, a, 4, 64, 128, 2, 100, None, a, None, 16, a, None, ctypes.byref(bad),
                              None) == -1
    assert L.gvr_indexer_topk(a, a, a, a, 4, 64, 128, 2, 100, None, a, None, 16, None, None, None, None) == -1
