"""Shape and determinism checks of the seeded decode workloads (no GPU)."""
import numpy as np
import pytest
import torch

import workloads


def test_config0_shapes_and_lengths():
    w = workloads.generate(0)
    assert w.scores.shape == (16, 1, 8207) and w.scores.dtype == torch.float32
    assert w.row_len[:, 0].tolist() == list(range(8192, 8208))
    assert torch.isfinite(w.scores).all() and (w.scores >= 0).all()


def test_step_subset_matches_full_run():
    full = workloads.generate(1, steps=[0, 1, 2, 3], queries=2)
    part = workloads.generate(1, steps=[3], queries=2)
    assert torch.equal(full.scores[3], part.scores[0])
    assert torch.equal(full.row_len[3], part.row_len[0])


def test_mtp_rows_and_lengths():
    w = workloads.generate(2, steps=[0, 5], queries=2)
    assert w.scores.shape == (2, 4, 102463)
    # row = b * next_n + r ; n = L0 + t * next_n + r
    assert w.row_len[1].tolist() == [102410, 102411, 102410, 102411]


def test_config3_subcases():
    a = workloads.generate(3, steps=[0], sub="a", queries=2)
    assert a.random_prev.shape == (1, 2, 2048)
    for r in range(2):
        p = a.random_prev[0, r].numpy()
        assert len(np.unique(p)) == 2048 and p.min() >= 0 and p.max() < int(a.row_len[0, r])
    b = workloads.generate(3, steps=[0], sub="b", queries=1)
    s = b.scores[0, 0]
    assert torch.equal(s, s.to(torch.bfloat16).to(torch.float32))
    c = workloads.generate(3, steps=[0], sub="c", queries=3)
    for r in range(3):
        n = int(c.row_len[0, r])
        assert 4096 <= n <= 131079
        assert torch.isinf(c.scores[0, r, n:]).all() and (c.scores[0, r, n:] < 0).all()
    d = workloads.generate(3, steps=[0], sub="d")
    assert d.row_len[0].tolist()[:4] == [0, 1, 2047, 2048]
    assert all(1 <= v <= 2048 for v in d.row_len[0].tolist()[4:])


def test_config4_lengths_fit_stride():
    spec = workloads.spec(4)
    assert spec["ld"] == 262144
    lo, hi = spec["L0"]
    assert hi + (spec["steps"] - 1) * spec["next_n"] + spec["next_n"] - 1 < spec["ld"]


def test_l0_override():
    w = workloads.generate(1, steps=[0, 1], queries=3, L0=5000)
    assert w.ld == 5000 + 63 and w.name == "c1_L5000"
    assert w.row_len.tolist() == [[5000] * 3, [5001] * 3]
    assert w.scores.shape == (2, 3, 5063)
    assert torch.isfinite(w.scores).all() and (w.scores >= 0).all()
    with pytest.raises(ValueError):
        workloads.generate(4, steps=[0], queries=1, L0=5000)
    with pytest.raises(ValueError):
        workloads.generate(3, steps=[0], queries=1, sub="a", L0=5000)
