"""The C-ABI library loads and exports what include/gvr_topk.h declares (no GPU).

Only host-side argument validation is exercised here: every call below
returns before any HIP runtime call is made.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gvr_topk.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
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
    for n in ("gvr_topk", "radix_topk", "gvr_topk_ex", "radix_topk_ex",
              "gvr_status_string", "gvr_version"):
        assert n in names, n


def test_every_declared_symbol_is_exported(L):
    for n in declared_functions():
        assert hasattr(L, n), "symbol %s missing from libgvr_topk.so" % n


def test_status_strings(L):
    import paper_2604_22312_amd as g
    for code in (0, -1, -2, -4, -5):
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
           g.Options(capacity=0, flags=8, parts=0, reserved1=0),        # unknown flag bit
           g.Options(capacity=0, flags=16, parts=0, reserved1=0),       # unknown flag bit
           g.Options(capacity=0, flags=0, parts=0, reserved1=1),        # reserved field set
           g.Options(capacity=0, flags=0, parts=17, reserved1=0),       # too many parts
           g.Options(capacity=0, flags=0, parts=-1, reserved1=0),       # negative parts
           g.Options(capacity=20000, flags=0, parts=0, reserved1=0)]    # capacity > max
    for opt in bad:
        assert L.gvr_topk_ex(vp(1), 2, 100, None, None, 128, vp(1), None, ctypes.byref(opt), None) == -1
        assert L.radix_topk_ex(vp(1), 2, 100, None, 128, vp(1), None, ctypes.byref(opt), None) == -1


def test_python_binding_refuses_cpu_tensors():
    import torch
    import paper_2604_22312_amd as g
    with pytest.raises(ValueError):
        g.gvr_topk(torch.zeros(2, 10), None, None, 4)
