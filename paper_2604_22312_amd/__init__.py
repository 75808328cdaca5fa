"""Exact decode-time Top-K for MI355X (gfx950): Guess-Verify-Refine and radix select.

Thin Python binding over the C ABI of ``include/gvr_topk.h`` (library
``libgvr_topk.so`` built in-tree by ``paper_2604_22312_amd.build``). This module
only validates tensors and marshals pointers; every step of the Top-K runs in
the HIP kernels of ``csrc/gvr_topk.hip``, ``csrc/rope_prior.hip`` and
``csrc/indexer.hip``. There is no CPU fallback: if the
library is missing, importing the functions raises.

Functions mirror the C entry points:

* ``gvr_topk(scores, row_len, prev_topk, K, out_idx=None, stream=None)``
* ``radix_topk(scores, row_len, prev_topk, K, out_idx=None, stream=None)``
* ``gvr_topk_ex`` / ``radix_topk_ex`` (options, per-row stats)
* ``gvr_topk_ex_noalloc`` -- ``gvr_topk_ex`` with no allocation inside the
  call (split-row workspace in a static device array)
* ``gvr_workspace_size`` / ``gvr_topk_ex_ws`` / ``radix_topk_ex_ws`` /
  ``new_workspace`` -- the split-row workspace owned by the caller (nothing
  allocated inside the call)
* ``prepare_gvr_topk`` / ``prepare_radix_topk`` -- a call checked and
  marshalled once, re-enqueued by calling it (loops over fixed buffers; with
  ``workspace=``, on a caller workspace)
* ``gvr_rope_g(n, params=None, device=...)`` -- g(Delta) of the RoPE/YaRN prior
* ``gvr_rope_prior(n, K, params=None, device=...)`` -- its static index set
  (``include/gvr_rope_prior.h``)
* ``gvr_indexer_scores(q, w, k, k_scale, ...)`` / ``gvr_indexer_topk(...)`` --
  the FP8 indexer scores, and the indexer followed by gvr_topk
  (``include/gvr_indexer.h``)
"""
from .binding import (  # noqa: F401
    GVR_MAX_CANDIDATES,
    GVR_MAX_K,
    PATH_NAMES,
    GvrError,
    Options,
    PreparedCall,
    RopeParams,
    decode_stats,
    gvr_indexer_scores,
    gvr_indexer_topk,
    gvr_rope_g,
    gvr_rope_params,
    gvr_read_floor,
    gvr_rope_prior,
    gvr_topk,
    gvr_topk_ex,
    gvr_topk_ex_noalloc,
    gvr_topk_ex_ws,
    gvr_workspace_size,
    lib,
    library_path,
    new_stats,
    new_workspace,
    prepare_gvr_topk,
    prepare_radix_topk,
    radix_topk,
    radix_topk_ex,
    radix_topk_ex_ws,
    status_string,
    version,
)
