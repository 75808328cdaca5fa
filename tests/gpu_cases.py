"""Shared helpers of the GPU parity tests: a decode-loop driver against the oracle."""
from __future__ import annotations

import functools
import sys

import numpy as np
import torch

import oracle
import workloads

K_TOPK = 2048


def note(msg: str) -> None:
    """Name the case before a GPU step (flushed, so it survives a crash)."""
    sys.stdout.write("[gpu-case] %s\n" % msg)
    sys.stdout.flush()


@functools.lru_cache(maxsize=16)
def workload(cfg: int, nsteps: int, queries: int, sub: str | None = None):
    return workloads.generate(cfg, steps=list(range(nsteps)), queries=queries, sub=sub)


def oracle_step(w, i, threads=8):
    return oracle.topk(w.scores[i].numpy(), w.K, row_len=w.row_len[i].numpy(), threads=threads)


def next_prev(exp: np.ndarray, B: int, nn: int) -> np.ndarray:
    """Every draft row of a query reuses the last draft row's exact output."""
    K = exp.shape[1]
    last = exp.reshape(B, nn, K)[:, nn - 1, :]
    return np.ascontiguousarray(np.repeat(last, nn, axis=0))


def assert_rows_equal(got: np.ndarray, exp: np.ndarray, what: str) -> None:
    if np.array_equal(got, exp):
        return
    bad = np.nonzero((got != exp).any(axis=1))[0]
    r = int(bad[0])
    diff = np.nonzero(got[r] != exp[r])[0][:5]
    raise AssertionError("%s: %d rows differ; first row %d at positions %s: got %s expected %s"
                         % (what, len(bad), r, diff.tolist(), got[r][diff].tolist(), exp[r][diff].tolist()))


def run_decode(fn, cfg, nsteps, queries, sub=None, dev="cuda", stats_check=False):
    """Run ``fn`` over the decode steps of a workload; compare every step with the oracle."""
    import paper_2604_22312_amd as gvr

    w = workload(cfg, nsteps, queries, sub)
    K, nn, B = w.K, w.next_n, w.B
    S = w.scores.to(dev)
    RL = w.row_len.to(dev)
    prev = None
    results = []
    for i, t in enumerate(w.steps):
        exp, kth, ngt = oracle_step(w, i)
        if sub == "a":
            pd = w.random_prev[i].to(dev)
        else:
            pd = None if prev is None else torch.from_numpy(prev).to(dev)
        note("%s cfg=%s sub=%s step=%d rows=%d ld=%d" % (fn.__name__, cfg, sub, t, w.rows, w.ld))
        if stats_check:
            st = gvr.new_stats(w.rows, dev)
            out = fn(S[i], RL[i], pd, K, stats=st)
        else:
            out = fn(S[i], RL[i], pd, K)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert_rows_equal(got, exp, "%s cfg %s%s step %d" % (fn.__name__, cfg, "" if sub is None else sub, t))
        if stats_check:
            results.append((i, gvr.decode_stats(st), kth, ngt))
        prev = next_prev(exp, B, nn)
    return w, results
