"""ctypes marshalling for ``libgvr_topk.so`` (argument checks and pointers only)."""
from __future__ import annotations

import ctypes
import os

import torch

GVR_MAX_K = 2048
GVR_MAX_CANDIDATES = 16384
PATH_NAMES = {0: "trivial", 1: "all", 2: "guess", 3: "narrowed", 4: "ties", 5: "no_guess", 6: "secant", -1: "error"}

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libgvr_topk.so")
_lib = None

STATS_INTS = 22   # sizeof(gvr_row_stats) / 4


class GvrError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__("%s failed: %s (%d)" % (fn, status_string(status), status))
        self.status = status


class Options(ctypes.Structure):
    """Mirror of ``gvr_options``: capacity C, flags (bit 0: ignore the guess;
    bit 1: scatter a row's parts over XCDs; bit 2: the paper's secant
    threshold search; bit 3: the paper's snap-iteration selection; bit 4 /
    5 / 6: force the 4-wave / 16-wave / 8-wave workgroup shape), parts
    (workgroups per row, 0 = automatic)."""
    _fields_ = [("capacity", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("parts", ctypes.c_int32), ("reserved1", ctypes.c_int32)]


class RopeParams(ctypes.Structure):
    """Mirror of ``gvr_rope_params`` (RoPE/YaRN angles of the static prior)."""
    _fields_ = [("d_rope", ctypes.c_int32), ("orig_ctx", ctypes.c_int32), ("base", ctypes.c_double),
                ("scale", ctypes.c_double), ("beta_fast", ctypes.c_double), ("beta_slow", ctypes.c_double)]


def library_path() -> str:
    return _LIB_PATH


def lib():
    """Load the HIP library; raise loudly if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError("libgvr_topk.so not built: run `python -m paper_2604_22312_amd.build` "
                              "(or __graft_entry__.build())")
        L = ctypes.CDLL(_LIB_PATH)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        for name in ("gvr_topk", "radix_topk"):
            f = getattr(L, name)
            f.restype = ctypes.c_int
            f.argtypes = [vp, i64, i64, vp, vp, i32, vp, vp]
        for name in ("gvr_topk_ex", "gvr_topk_ex_noalloc"):
            f = getattr(L, name)
            f.restype = ctypes.c_int
            f.argtypes = [vp, i64, i64, vp, vp, i32, vp, vp, ctypes.POINTER(Options), vp]
        L.radix_topk_ex.restype = ctypes.c_int
        L.radix_topk_ex.argtypes = [vp, i64, i64, vp, i32, vp, vp, ctypes.POINTER(Options), vp]
        L.gvr_workspace_size.restype = ctypes.c_int
        L.gvr_workspace_size.argtypes = [i64, i64, i32, ctypes.c_int, ctypes.POINTER(Options),
                                         ctypes.POINTER(ctypes.c_size_t)]
        L.gvr_topk_ex_ws.restype = ctypes.c_int
        L.gvr_topk_ex_ws.argtypes = [vp, i64, i64, vp, vp, i32, vp, vp, ctypes.POINTER(Options), vp, vp,
                                     ctypes.c_size_t]
        L.radix_topk_ex_ws.restype = ctypes.c_int
        L.radix_topk_ex_ws.argtypes = [vp, i64, i64, vp, i32, vp, vp, ctypes.POINTER(Options), vp, vp,
                                       ctypes.c_size_t]
        L.gvr_rope_params_default.restype = None
        L.gvr_rope_params_default.argtypes = [ctypes.POINTER(RopeParams)]
        L.gvr_rope_g.restype = ctypes.c_int
        L.gvr_rope_g.argtypes = [i64, ctypes.POINTER(RopeParams), vp, vp, vp]
        L.gvr_rope_prior.restype = ctypes.c_int
        L.gvr_rope_prior.argtypes = [i64, i32, ctypes.POINTER(RopeParams), vp, vp, vp]
        L.gvr_indexer_scores.restype = ctypes.c_int
        L.gvr_indexer_scores.argtypes = [vp, vp, vp, vp, i64, i32, i32, i32, i64, vp, vp, vp]
        L.gvr_indexer_topk.restype = ctypes.c_int
        L.gvr_indexer_topk.argtypes = [vp, vp, vp, vp, i64, i32, i32, i32, i64, vp, vp, vp, i32, vp, vp,
                                       ctypes.POINTER(Options), vp]
        L.gvr_read_floor.restype = ctypes.c_int
        L.gvr_read_floor.argtypes = [vp, i64, i64, vp, vp, vp]
        L.gvr_status_string.restype = ctypes.c_char_p
        L.gvr_status_string.argtypes = [ctypes.c_int]
        L.gvr_version.restype = ctypes.c_char_p
        L.gvr_version.argtypes = []
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().gvr_status_string(int(status)).decode()


def version() -> str:
    return lib().gvr_version().decode()


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream, device):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _on_device(dev):
    """The tensors' device made current for the call (a no-op context when it
    already is, which skips the device switch and restore)."""
    idx = dev.index if isinstance(dev, torch.device) else int(dev)
    if idx is None or torch.cuda.current_device() == idx:
        return _NO_SWITCH
    return torch.cuda.device(idx)


class _NoSwitch:
    def __enter__(self):
        return self

    def __exit__(self, *exc):
        return False


_NO_SWITCH = _NoSwitch()


def _check(scores, row_len, prev_topk, K, out_idx):
    if not isinstance(scores, torch.Tensor) or scores.dtype != torch.float32 or scores.dim() != 2:
        raise ValueError("scores must be a float32 tensor [B][ld]")
    if not scores.is_cuda:
        raise ValueError("scores must be on a GPU (there is no CPU path)")
    if not scores.is_contiguous():
        raise ValueError("scores must be contiguous (row stride = ld)")
    B, ld = scores.shape
    dev = scores.device
    K = int(K)
    if row_len is not None:
        if row_len.dtype != torch.int32 or row_len.shape != (B,) or row_len.device != dev or not row_len.is_contiguous():
            raise ValueError("row_len must be a contiguous int32 tensor [B] on the scores' device")
    if prev_topk is not None:
        if (prev_topk.dtype != torch.int32 or prev_topk.shape != (B, K) or prev_topk.device != dev
                or not prev_topk.is_contiguous()):
            raise ValueError("prev_topk must be a contiguous int32 tensor [B][K] on the scores' device")
    if out_idx is None:
        out_idx = torch.empty((B, max(K, 0)), dtype=torch.int32, device=dev)
    elif (out_idx.dtype != torch.int32 or out_idx.shape != (B, K) or out_idx.device != dev
          or not out_idx.is_contiguous()):
        raise ValueError("out_idx must be a contiguous int32 tensor [B][K] on the scores' device")
    return B, ld, K, out_idx


def _call(fn_name, scores, row_len, prev_topk, K, out_idx, stream):
    B, ld, K, out_idx = _check(scores, row_len, prev_topk, K, out_idx)
    with _on_device(scores.device):
        st = getattr(lib(), fn_name)(_ptr(scores), B, ld, _ptr(row_len), _ptr(prev_topk), K,
                                     _ptr(out_idx), _stream(stream, scores.device))
    if st != 0:
        raise GvrError(fn_name, st)
    return out_idx


def gvr_topk(scores, row_len, prev_topk, K, out_idx=None, stream=None):
    """Guess-Verify-Refine Top-K; returns ``out_idx`` [B][K] int32 (ascending indices)."""
    return _call("gvr_topk", scores, row_len, prev_topk, K, out_idx, stream)


def radix_topk(scores, row_len, prev_topk, K, out_idx=None, stream=None):
    """Radix-select Top-K (``prev_topk`` accepted and ignored); same result as ``gvr_topk``."""
    return _call("radix_topk", scores, row_len, prev_topk, K, out_idx, stream)


def _call_ex(radix, scores, row_len, prev_topk, K, out_idx, stream, options, stats, fn="gvr_topk_ex"):
    B, ld, K, out_idx = _check(scores, row_len, prev_topk, K, out_idx)
    if stats is not None and (stats.dtype != torch.int32 or stats.shape != (B, STATS_INTS)
                              or stats.device != scores.device or not stats.is_contiguous()):
        raise ValueError("stats must be a contiguous int32 tensor [B][%d] on the scores' device" % STATS_INTS)
    opt = None
    if options is not None:
        opt = Options(**options) if isinstance(options, dict) else options
    optp = ctypes.byref(opt) if opt is not None else None
    with _on_device(scores.device):
        L = lib()
        if radix:
            st = L.radix_topk_ex(_ptr(scores), B, ld, _ptr(row_len), K, _ptr(out_idx),
                                 _stream(stream, scores.device), optp, _ptr(stats))
        else:
            st = getattr(L, fn)(_ptr(scores), B, ld, _ptr(row_len), _ptr(prev_topk), K, _ptr(out_idx),
                                _stream(stream, scores.device), optp, _ptr(stats))
    if st != 0:
        raise GvrError("radix_topk_ex" if radix else fn, st)
    return out_idx


def gvr_topk_ex(scores, row_len, prev_topk, K, out_idx=None, stream=None, options=None, stats=None):
    """``gvr_topk`` with options (dict or ``Options``) and an optional stats
    tensor ([B][22] int32, see ``decode_stats``)."""
    return _call_ex(False, scores, row_len, prev_topk, K, out_idx, stream, options, stats)


def gvr_topk_ex_noalloc(scores, row_len, prev_topk, K, out_idx=None, stream=None, options=None, stats=None):
    """``gvr_topk_ex`` taking its split-row workspace from the library's static
    device array (no allocation inside the call). ``out_idx`` is allocated
    here when it is None, before the call."""
    return _call_ex(False, scores, row_len, prev_topk, K, out_idx, stream, options, stats, fn="gvr_topk_ex_noalloc")


def radix_topk_ex(scores, row_len, K, out_idx=None, stream=None, options=None, stats=None):
    return _call_ex(True, scores, row_len, None, K, out_idx, stream, options, stats)


def _options(options):
    if options is None:
        return None
    return Options(**options) if isinstance(options, dict) else options


def gvr_workspace_size(B, ld, K, use_guess=True, options=None, device=None) -> int:
    """Bytes of caller workspace a ``gvr_topk_ex_ws`` (``use_guess``, with a
    guess) or ``radix_topk_ex_ws`` call of this shape and these options needs
    on ``device`` (default: the current device); 0 when it does not split."""
    opt = _options(options)
    n = ctypes.c_size_t(0)
    dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
    with _on_device(dev):
        st = lib().gvr_workspace_size(int(B), int(ld), int(K), 1 if use_guess else 0,
                                      ctypes.byref(opt) if opt is not None else None, ctypes.byref(n))
    if st != 0:
        raise GvrError("gvr_workspace_size", st)
    return int(n.value)


def new_workspace(B, ld, K, use_guess=True, options=None, device=None):
    """A zero-filled uint8 device tensor of ``gvr_workspace_size`` bytes (at
    least one byte, so that its pointer is never NULL)."""
    n = gvr_workspace_size(B, ld, K, use_guess, options, device)
    dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
    return torch.zeros(max(n, 1), dtype=torch.uint8, device=dev)


def _call_ws(radix, scores, row_len, prev_topk, K, workspace, out_idx, stream, options, stats):
    B, ld, K, out_idx = _check(scores, row_len, None if radix else prev_topk, K, out_idx)
    if stats is not None and (stats.dtype != torch.int32 or stats.shape != (B, STATS_INTS)
                              or stats.device != scores.device or not stats.is_contiguous()):
        raise ValueError("stats must be a contiguous int32 tensor [B][%d] on the scores' device" % STATS_INTS)
    if workspace is not None and (workspace.device != scores.device or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous tensor on the scores' device")
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    opt = _options(options)
    optp = ctypes.byref(opt) if opt is not None else None
    with _on_device(scores.device):
        L = lib()
        if radix:
            st = L.radix_topk_ex_ws(_ptr(scores), B, ld, _ptr(row_len), K, _ptr(out_idx),
                                    _stream(stream, scores.device), optp, _ptr(stats), _ptr(workspace), nbytes)
        else:
            st = L.gvr_topk_ex_ws(_ptr(scores), B, ld, _ptr(row_len), _ptr(prev_topk), K, _ptr(out_idx),
                                  _stream(stream, scores.device), optp, _ptr(stats), _ptr(workspace), nbytes)
    if st != 0:
        raise GvrError("radix_topk_ex_ws" if radix else "gvr_topk_ex_ws", st)
    return out_idx


def gvr_topk_ex_ws(scores, row_len, prev_topk, K, workspace, out_idx=None, stream=None, options=None,
                   stats=None):
    """``gvr_topk_ex`` with the split-row workspace supplied by the caller
    (``workspace``: a contiguous device tensor, zero-filled before its first
    use, e.g. from ``new_workspace``; its size in bytes is passed as
    ws_bytes; None = no workspace). ``out_idx`` is allocated here when it is
    None, before the call."""
    return _call_ws(False, scores, row_len, prev_topk, K, workspace, out_idx, stream, options, stats)


def radix_topk_ex_ws(scores, row_len, K, workspace, out_idx=None, stream=None, options=None, stats=None):
    """``radix_topk_ex`` with a caller workspace (as ``gvr_topk_ex_ws``)."""
    return _call_ws(True, scores, row_len, None, K, workspace, out_idx, stream, options, stats)


class PreparedCall:
    """One Top-K call whose tensors were checked and whose pointers were
    marshalled once: calling the object enqueues the same call again, on the
    same stream, and returns its ``out_idx``. The tensors must stay alive and
    keep their shapes; their contents may change between calls. For loops over
    fixed buffers, where the per-call checks would take more host time than
    the kernel takes on the device."""
    __slots__ = ("_f", "_args", "_name", "_dev", "out_idx", "_keep")

    def __call__(self):
        if torch.cuda.current_device() != self._dev:
            with torch.cuda.device(self._dev):
                st = self._f(*self._args)
        else:
            st = self._f(*self._args)
        if st != 0:
            raise GvrError(self._name, st)
        return self.out_idx


def _prepare(radix, scores, row_len, prev_topk, K, out_idx, stream, options, workspace=None):
    B, ld, K, out_idx = _check(scores, row_len, None if radix else prev_topk, K, out_idx)
    L = lib()
    opt = None
    if options is not None:
        opt = Options(**options) if isinstance(options, dict) else options
    pc = PreparedCall()
    pc._dev = scores.device.index if scores.device.index is not None else torch.cuda.current_device()
    sp = _stream(stream, scores.device)
    if workspace is not None:
        if workspace.device != scores.device or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on the scores' device")
        nbytes = workspace.numel() * workspace.element_size()
        optp = ctypes.byref(opt) if opt is not None else None
        if radix:
            pc._name, pc._f = "radix_topk_ex_ws", L.radix_topk_ex_ws
            pc._args = (_ptr(scores), B, ld, _ptr(row_len), K, _ptr(out_idx), sp, optp, None, _ptr(workspace), nbytes)
        else:
            pc._name, pc._f = "gvr_topk_ex_ws", L.gvr_topk_ex_ws
            pc._args = (_ptr(scores), B, ld, _ptr(row_len), _ptr(prev_topk), K, _ptr(out_idx), sp, optp, None,
                        _ptr(workspace), nbytes)
    elif opt is None and not radix:
        pc._name, pc._f = "gvr_topk", L.gvr_topk
        pc._args = (_ptr(scores), B, ld, _ptr(row_len), _ptr(prev_topk), K, _ptr(out_idx), sp)
    elif opt is None:
        pc._name, pc._f = "radix_topk", L.radix_topk
        pc._args = (_ptr(scores), B, ld, _ptr(row_len), None, K, _ptr(out_idx), sp)
    elif radix:
        pc._name, pc._f = "radix_topk_ex", L.radix_topk_ex
        pc._args = (_ptr(scores), B, ld, _ptr(row_len), K, _ptr(out_idx), sp, ctypes.byref(opt), None)
    else:
        pc._name, pc._f = "gvr_topk_ex", L.gvr_topk_ex
        pc._args = (_ptr(scores), B, ld, _ptr(row_len), _ptr(prev_topk), K, _ptr(out_idx), sp, ctypes.byref(opt), None)
    pc.out_idx = out_idx
    pc._keep = (scores, row_len, prev_topk, opt, stream, workspace)
    return pc


def prepare_gvr_topk(scores, row_len, prev_topk, K, out_idx=None, stream=None, options=None, workspace=None):
    """A ``PreparedCall`` of ``gvr_topk`` (``gvr_topk_ex`` with options;
    ``gvr_topk_ex_ws`` with a caller ``workspace``, see ``new_workspace``)."""
    return _prepare(False, scores, row_len, prev_topk, K, out_idx, stream, options, workspace)


def prepare_radix_topk(scores, row_len, K, out_idx=None, stream=None, options=None, workspace=None):
    """A ``PreparedCall`` of ``radix_topk`` (``radix_topk_ex`` with options;
    ``radix_topk_ex_ws`` with a caller ``workspace``)."""
    return _prepare(True, scores, row_len, None, K, out_idx, stream, options, workspace)


def new_stats(B, device):
    """A zeroed stats tensor for ``*_ex`` calls."""
    return torch.zeros((B, STATS_INTS), dtype=torch.int32, device=device)


def decode_stats(stats: torch.Tensor) -> dict:
    """Split a [B][22] int32 stats tensor (``gvr_row_stats``) into named columns."""
    s = stats.detach().cpu()
    i32 = s[:, :12]
    i64 = s[:, 12:22].contiguous().view(torch.int64)
    u32 = lambda c: (i32[:, c].to(torch.int64) & 0xFFFFFFFF)  # noqa: E731
    return {
        "n": i32[:, 0].clone(), "path": i32[:, 1].clone(), "passes": i32[:, 2].clone(),
        "candidates": i32[:, 3].clone(), "threshold": u32(4), "kth_key": u32(5),
        "n_gt": i32[:, 6].clone(), "guess_valid": i32[:, 7].clone(),
        "spec_threshold": u32(8), "spec_count": i32[:, 9].clone(),
        "pmean": i32[:, 10].clone().view(torch.float32), "refine_iters": i32[:, 11].clone(),
        "t_start": i64[:, 0].clone(), "t_guess": i64[:, 1].clone(), "t_search": i64[:, 2].clone(),
        "t_collect": i64[:, 3].clone(), "t_refine": i64[:, 4].clone(),
    }


def gvr_rope_params(**kw) -> RopeParams:
    """``gvr_rope_params`` holding the library defaults, with ``kw`` overrides."""
    p = RopeParams()
    lib().gvr_rope_params_default(ctypes.byref(p))
    for k, v in kw.items():
        if not hasattr(p, k):
            raise ValueError("unknown RoPE parameter %r" % k)
        setattr(p, k, v)
    return p


def _rope_args(params, device):
    if params is None:
        params = gvr_rope_params()
    elif isinstance(params, dict):
        params = gvr_rope_params(**params)
    if device is None:
        raise ValueError("device must be given")
    dev = torch.device(device)
    if dev.type != "cuda":
        raise ValueError("the RoPE prior runs on a GPU (there is no CPU path)")
    if dev.index is None:
        dev = torch.device("cuda", torch.cuda.current_device())
    return params, dev


def gvr_rope_g(n, params=None, device="cuda", g=None, theta=None, stream=None):
    """g(Delta), Delta = 0..n-1, as a float64 tensor on ``device``; ``theta``
    (float64 [d/2], optional) receives the YaRN angles."""
    params, dev = _rope_args(params, device)
    n = int(n)
    if g is None:
        g = torch.empty(max(n, 0), dtype=torch.float64, device=dev)
    for t, size in ((g, n), (theta, params.d_rope // 2)):
        if t is not None and (t.dtype != torch.float64 or t.numel() != size or t.device != dev
                              or not t.is_contiguous()):
            raise ValueError("g / theta must be contiguous float64 tensors of n / d/2 elements on the device")
    with _on_device(dev):
        st = lib().gvr_rope_g(n, ctypes.byref(params), _ptr(g), _ptr(theta), _stream(stream, dev))
    if st != 0:
        raise GvrError("gvr_rope_g", st)
    return g


def gvr_rope_prior(n, K, params=None, device="cuda", out=None, g=None, stream=None):
    """P_static (int32 [K], ascending) of the RoPE/YaRN prior over Delta = 0..n-1;
    ``g`` (float64 [n], optional) receives g(Delta)."""
    params, dev = _rope_args(params, device)
    n, K = int(n), int(K)
    if g is None:
        g = torch.empty(max(n, 0), dtype=torch.float64, device=dev)
    elif g.dtype != torch.float64 or g.numel() != n or g.device != dev or not g.is_contiguous():
        raise ValueError("g must be a contiguous float64 tensor of n elements on the device")
    if out is None:
        out = torch.empty(max(K, 0), dtype=torch.int32, device=dev)
    elif out.dtype != torch.int32 or out.numel() != K or out.device != dev or not out.is_contiguous():
        raise ValueError("out must be a contiguous int32 tensor of K elements on the device")
    with _on_device(dev):
        st = lib().gvr_rope_prior(n, K, ctypes.byref(params), _ptr(g), _ptr(out), _stream(stream, dev))
    if st != 0:
        raise GvrError("gvr_rope_prior", st)
    return out


def _check_indexer(q, w, k, k_scale, row_len, scores):
    for name, t, dt in (("q", q, torch.uint8), ("w", w, torch.float32), ("k", k, torch.uint8),
                        ("k_scale", k_scale, torch.float32)):
        if not isinstance(t, torch.Tensor) or t.dtype != dt or not t.is_cuda or not t.is_contiguous():
            raise ValueError("%s must be a contiguous %s tensor on a GPU (there is no CPU path)" % (name, dt))
    if q.dim() != 3 or w.dim() != 2 or k.dim() != 3 or k_scale.dim() != 2:
        raise ValueError("shapes: q [B][H][D], w [B][H], k [C][ld][D], k_scale [C][ld]")
    B, H, D = q.shape
    C, ld, Dk = k.shape
    dev = q.device
    if w.shape != (B, H) or Dk != D or k_scale.shape != (C, ld) or C == 0 or B % C != 0:
        raise ValueError("inconsistent indexer shapes: q %s w %s k %s k_scale %s"
                         % (tuple(q.shape), tuple(w.shape), tuple(k.shape), tuple(k_scale.shape)))
    for t in (w, k, k_scale):
        if t.device != dev:
            raise ValueError("indexer tensors must be on one device")
    if row_len is not None and (row_len.dtype != torch.int32 or row_len.shape != (B,) or row_len.device != dev
                                or not row_len.is_contiguous()):
        raise ValueError("row_len must be a contiguous int32 tensor [B] on the device")
    if scores is None:
        scores = torch.empty((B, ld), dtype=torch.float32, device=dev)
    elif (scores.dtype != torch.float32 or scores.shape != (B, ld) or scores.device != dev
          or not scores.is_contiguous()):
        raise ValueError("scores must be a contiguous float32 tensor [B][ld] on the device")
    return B, H, D, B // C, ld, scores


def gvr_indexer_scores(q, w, k, k_scale, row_len=None, scores=None, stream=None):
    """Indexer scores I [B][ld] (float32; entries s >= n_b are not written)
    from FP8 E4M3 bytes q [B][H][D], key cache k [C][ld][D] shared by B / C
    consecutive rows, k_scale [C][ld] and head weights w [B][H]."""
    B, H, D, group, ld, scores = _check_indexer(q, w, k, k_scale, row_len, scores)
    with _on_device(q.device):
        st = lib().gvr_indexer_scores(_ptr(q), _ptr(w), _ptr(k), _ptr(k_scale), B, H, D, group, ld,
                                      _ptr(row_len), _ptr(scores), _stream(stream, q.device))
    if st != 0:
        raise GvrError("gvr_indexer_scores", st)
    return scores


def gvr_indexer_topk(q, w, k, k_scale, row_len, prev_topk, K, scores=None, out_idx=None, stream=None,
                     options=None, stats=None):
    """The indexer, then gvr_topk_ex on its scores; returns (out_idx [B][K], scores [B][ld])."""
    B, H, D, group, ld, scores = _check_indexer(q, w, k, k_scale, row_len, scores)
    _, _, K, out_idx = _check(scores, row_len, prev_topk, K, out_idx)
    opt = None
    if options is not None:
        opt = Options(**options) if isinstance(options, dict) else options
    with _on_device(q.device):
        st = lib().gvr_indexer_topk(_ptr(q), _ptr(w), _ptr(k), _ptr(k_scale), B, H, D, group, ld,
                                    _ptr(row_len), _ptr(scores), _ptr(prev_topk), K, _ptr(out_idx),
                                    _stream(stream, q.device), ctypes.byref(opt) if opt is not None else None,
                                    _ptr(stats))
    if st != 0:
        raise GvrError("gvr_indexer_topk", st)
    return out_idx, scores


def gvr_read_floor(scores, row_len=None, out_words=None, stream=None):
    """Measurement helper: read every element of each row once (the plain
    read rate of the rows). Returns ``out_words`` [B][16] uint32 as int32;
    the xor of a row's 16 words is the xor of its elements' bits."""
    if not isinstance(scores, torch.Tensor) or scores.dtype != torch.float32 or scores.dim() != 2:
        raise ValueError("scores must be a float32 tensor [B][ld]")
    if not scores.is_cuda or not scores.is_contiguous():
        raise ValueError("scores must be a contiguous tensor on a GPU (there is no CPU path)")
    B, ld = scores.shape
    if row_len is not None and (row_len.dtype != torch.int32 or row_len.shape != (B,)
                                or row_len.device != scores.device or not row_len.is_contiguous()):
        raise ValueError("row_len must be a contiguous int32 tensor [B] on the scores' device")
    if out_words is None:
        out_words = torch.empty((B, 16), dtype=torch.int32, device=scores.device)
    elif (out_words.dtype != torch.int32 or out_words.shape != (B, 16) or out_words.device != scores.device
          or not out_words.is_contiguous()):
        raise ValueError("out_words must be a contiguous int32 tensor [B][16] on the scores' device")
    with _on_device(scores.device):
        st = lib().gvr_read_floor(_ptr(scores), B, ld, _ptr(row_len), _ptr(out_words), _stream(stream, scores.device))
    if st != 0:
        raise GvrError("gvr_read_floor", st)
    return out_words
