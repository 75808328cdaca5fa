"""CPU oracle for exact per-row Top-K -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The GPU product path
(``paper_2604_22312_amd``) never imports it, and the two share no code.

The arithmetic lives in ``oracle_topk.c`` (plain C, built with gcc); this
module only builds/loads it and marshals numpy arrays. What it computes:

* ``topk``     -- the exact Top-K of each row (Sec. 4.1, problem statement),
                  larger key first, lower index first among equal keys, answer
                  listed in ascending index order, ``-1`` padding when n <= K.
* ``count_ge`` -- the threshold count f(T) = |{i : x_i >= T}| (Sec. 4.1),
                  with ">=" taken on sortable keys.
* ``key``      -- the sortable 32-bit key of each fp32 value (the "sortable
                  FP32 score key" the radix baseline ranks, Sec. 2.2).

The oracle of the static RoPE/YaRN prior (g(Delta), P_static; Sec. 3.2,
3.3) is the numpy module ``oracle/rope_prior.py``.

Parity status: ``topk``, ``count_ge`` and ``key`` are pinned by
``tests/test_oracle_pins.py`` (brute force, closed forms, invariants, numpy
cross-checks and planted mistakes).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "oracle_topk.c")
LIBRARY = os.path.join(_HERE, "liboracle_topk.so")


def compile_library(src: str, out: str) -> str:
    """gcc -O2 ``src`` into the shared library ``out`` (atomic replace)."""
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall",
                           "-Wextra", "-o", tmp, src])
    os.replace(tmp, out)
    return out


def build(force: bool = True) -> str:
    """Compile ``oracle_topk.c`` into ``liboracle_topk.so``."""
    if force or not os.path.exists(LIBRARY):
        compile_library(SOURCE, LIBRARY)
    return LIBRARY


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """ctypes front end of one build of ``oracle_topk.c``."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        lib.oracle_key.restype = ctypes.c_uint32
        lib.oracle_key.argtypes = [ctypes.c_float]
        lib.oracle_keys.restype = None
        lib.oracle_keys.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_count_ge.restype = ctypes.c_int64
        lib.oracle_count_ge.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32]
        lib.oracle_topk_row.restype = ctypes.c_int
        lib.oracle_topk_row.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        self.lib = lib
        self.path = path

    def key(self, x) -> np.ndarray:
        """Sortable uint32 key of every fp32 value in ``x``."""
        shape = np.shape(x)
        x = np.ascontiguousarray(np.asarray(x, dtype=np.float32)).reshape(-1)
        out = np.empty(x.shape, dtype=np.uint32)
        self.lib.oracle_keys(_ptr(x), x.size, _ptr(out))
        return out.reshape(shape)

    def count_ge(self, row, tkey: int, n: int | None = None) -> int:
        """f(T): number of i < n with key(row[i]) >= tkey."""
        row = np.ascontiguousarray(np.asarray(row, dtype=np.float32))
        n = row.size if n is None else int(n)
        assert 0 <= n <= row.size
        return int(self.lib.oracle_count_ge(_ptr(row), n, ctypes.c_uint32(int(tkey))))

    def topk(self, scores, K: int, row_len=None, threads: int = 1):
        """Exact Top-K of each row of ``scores`` ([B][ld] fp32, or one row).

        Returns ``(idx [B][K] int32, kth_key [B] uint32, n_gt [B] int32)``.
        ``row_len`` ([B] ints) is clamped to [0, ld]; ``None`` means full rows.
        ``threads`` > 1 spreads rows over Python threads (the C call releases
        the GIL); the per-row computation is unchanged.
        """
        s = np.ascontiguousarray(np.asarray(scores, dtype=np.float32))
        if s.ndim == 1:
            s = s[None, :]
        B, ld = s.shape
        K = int(K)
        if K < 1:
            raise ValueError("K must be >= 1")
        if row_len is None:
            rl = np.full(B, ld, dtype=np.int64)
        else:
            rl = np.asarray(row_len, dtype=np.int64).reshape(B)
        out = np.empty((B, K), dtype=np.int32)
        kth = np.zeros(B, dtype=np.uint32)
        ngt = np.zeros(B, dtype=np.int32)
        lib = self.lib

        def one(b):
            n = min(max(int(rl[b]), 0), ld)
            rc = lib.oracle_topk_row(
                ctypes.c_void_p(s.ctypes.data + b * ld * 4), n, K,
                ctypes.c_void_p(out.ctypes.data + b * K * 4),
                ctypes.c_void_p(kth.ctypes.data + b * 4),
                ctypes.c_void_p(ngt.ctypes.data + b * 4))
            if rc != 0:
                raise MemoryError("oracle_topk_row failed (%d)" % rc)

        if threads <= 1 or B <= 1:
            for b in range(B):
                one(b)
        else:
            with ThreadPoolExecutor(max_workers=threads) as ex:
                list(ex.map(one, range(B)))
        return out, kth, ngt


_default = None
_lock = threading.Lock()


def default() -> Oracle:
    global _default
    with _lock:
        if _default is None:
            if not os.path.exists(LIBRARY):
                build(force=True)
            _default = Oracle(LIBRARY)
    return _default


def key(x) -> np.ndarray:
    return default().key(x)


def count_ge(row, tkey: int, n: int | None = None) -> int:
    return default().count_ge(row, tkey, n)


def topk(scores, K: int, row_len=None, threads: int = 1):
    return default().topk(scores, K, row_len=row_len, threads=threads)
