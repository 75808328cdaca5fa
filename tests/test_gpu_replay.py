"""Pass-count parity: the GPU's per-row stats (path, full-row passes,
speculative threshold and count, accepted threshold and candidates) equal the
CPU replay of the control flow (tests/replay.py) on the same fp32 rows, for
the decode workloads (the previous step's Top-K as the guess, a random guess,
bf16 ties, ragged rows, rows of at most K) and for the guess-free kernel."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from tests import replay as R
from tests.gpu_cases import K_TOPK, next_prev, note

pytestmark = pytest.mark.gpu

DEV = "cuda"
FIELDS = ("path", "passes", "spec_threshold", "spec_count", "threshold", "candidates")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2604_22312_amd as g
    g.lib()


def _compare(w, i, S, RL, pv, st, parts, what):
    import paper_2604_22312_amd as g
    d = g.decode_stats(st)
    s = w.scores[i].numpy()
    rl = w.row_len[i].numpy()
    base = S.data_ptr()
    bad = []
    for r in range(w.rows):
        aoff = ((base + 4 * r * w.ld) >> 2) & 31
        pred = R.replay_row(s[r], int(rl[r]), None if pv is None else pv[r], K_TOPK, parts, aoff)
        for f in FIELDS:
            if f in pred and int(d[f][r]) != int(pred[f]):
                bad.append((r, f, int(d[f][r]), int(pred[f])))
    assert not bad, "%s: %d mismatches, first %s" % (what, len(bad), bad[:5])
    return d


@pytest.mark.parametrize("cfg,sub,steps,queries", [(2, None, 3, 64), (1, None, 3, 32), (3, "a", 2, 8),
                                                   (3, "b", 2, 8), (3, "c", 2, 8), (3, "d", 2, 8),
                                                   (4, None, 2, 16), (0, None, 4, 1)],
                         ids=["c2", "c1", "c3a", "c3b", "c3c", "c3d", "c4", "c0"])
def test_row_stats_match_the_replay(cfg, sub, steps, queries):
    import paper_2604_22312_amd as g
    w = workloads.generate(cfg, steps=list(range(steps)), queries=queries, sub=sub)
    parts = R.choose_parts(w.rows, w.ld)
    prev = None
    passes = []
    for i in range(steps):
        S = w.scores[i].to(DEV)
        RL = w.row_len[i].to(DEV)
        exp, _, _ = oracle.topk(w.scores[i].numpy(), K_TOPK, row_len=w.row_len[i].numpy(), threads=8)
        pv = w.random_prev[i].numpy() if sub == "a" else prev
        note("replay cfg=%d sub=%s step=%d rows=%d parts=%d" % (cfg, sub, i, w.rows, parts))
        st = g.new_stats(w.rows, DEV)
        g.gvr_topk_ex(S, RL, None if pv is None else torch.from_numpy(np.ascontiguousarray(pv)).to(DEV), K_TOPK,
                      stats=st)
        torch.cuda.synchronize()
        d = _compare(w, i, S, RL, pv, st, parts if pv is not None else 1, "gvr cfg %d%s step %d" % (cfg, sub or "", i))
        passes += d["passes"].tolist()
        # the guess-free kernel on the same rows
        st = g.new_stats(w.rows, DEV)
        g.radix_topk_ex(S, RL, K_TOPK, stats=st)
        torch.cuda.synchronize()
        _compare(w, i, S, RL, None, st, 1, "radix cfg %d%s step %d" % (cfg, sub or "", i))
        prev = next_prev(exp, w.B, w.next_n)
    note("  passes per row: mean %.3f max %d" % (float(np.mean(passes)), int(np.max(passes))))
