"""The CPU replay of gvr_topk's control flow (tests/replay.py), checked
against the oracle and the definitions it restates (no GPU): whatever path it
predicts ends at a threshold T with K <= f(T) <= C at or below the K-th key
(Lemma 1, Sec. 4.1), or at the K-th key itself (ties); on the 100K decode
rows the guess of the previous step holds the answer in one pass; a random
guess does not. The GPU's row stats are compared with it in
tests/test_gpu_replay.py."""
import numpy as np
import pytest

import oracle
import workloads
from tests import replay as R
from tests.gpu_cases import next_prev

K = 2048


def _check_row(x, n, pred, kth):
    xk = R.keys(x[:n])
    if pred["path"] == R.PATH["trivial"]:
        assert n <= K
        return
    if pred["path"] == R.PATH["ties"]:
        assert pred["threshold"] == kth
        return
    T = pred["threshold"] if "threshold" in pred else None
    if pred["path"] == R.PATH["all"]:
        assert pred["candidates"] == n
        return
    assert K <= pred["candidates"] <= R.CAP
    assert R.count_ge(xk, T) == pred["candidates"] == oracle.count_ge(x, T, n=n)
    assert T <= kth


@pytest.mark.parametrize("cfg,sub,steps,queries", [(2, None, 3, 4), (3, "a", 2, 8), (3, "b", 2, 8),
                                                   (3, "c", 2, 8), (3, "d", 2, 8), (0, None, 3, 1)],
                         ids=["c2", "c3a", "c3b", "c3c", "c3d", "c0"])
def test_replay_reaches_a_valid_threshold(cfg, sub, steps, queries):
    w = workloads.generate(cfg, steps=list(range(steps)), queries=queries, sub=sub)
    parts = R.choose_parts(w.rows, w.ld)
    prev = None
    for i in range(steps):
        s = w.scores[i].numpy()
        rl = w.row_len[i].numpy()
        exp, kth, _ = oracle.topk(s, K, row_len=rl)
        pv = w.random_prev[i].numpy() if sub == "a" else prev
        for r in range(w.rows):
            pred = R.replay_row(s[r], int(rl[r]), None if pv is None else pv[r], K, parts, (r * w.ld) & 31)
            _check_row(s[r], int(rl[r]), pred, int(kth[r]))
            if i > 0 and cfg == 2:
                assert pred["path"] == R.PATH["guess"] and pred["passes"] == 1
            if i > 0 and sub == "a" and int(rl[r]) > 2 * K:
                assert pred["passes"] >= 2   # a random guess leaves far too many candidates
        prev = next_prev(exp, w.B, w.next_n)


def test_replay_spec_threshold_definition():
    """Phase 1 on a hand-made guess: the sampled keys sit in known bins."""
    x = np.arange(10000, dtype=np.float32) / 100.0
    prev = np.arange(2048, dtype=np.int32) * 4          # samples 0, 32, 64, ... of the guess
    t, cnt = R.spec_threshold(R.keys(x), 10000, prev, K)
    assert cnt == 256
    # rank ceil(65 * 256 / 2048) = 9 from the bottom: the 9th sampled element, index 8 * 32
    assert t <= int(R.keys(x[256:257])[0]) and t > int(R.keys(x[224:225])[0])
    assert R.spec_threshold(R.keys(x), 100, np.full(2048, 5000, np.int32), K) == (None, 0)
