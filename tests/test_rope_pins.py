"""Pins for the RoPE/YaRN prior oracle (no GPU).

The oracle (``oracle/rope_prior.py``) computes g(Delta) of Sec. 3.2 and the
static index set P_static of Sec. 3.3. These tests tie it to things other than
its own formulas:

* closed forms: plain RoPE angles at pairs 0, 8, 16, 24 of d = 64 are
  1, 0.1, 0.01, 0.001; g(0) = d; one rotary pair with angle 1 gives
  g(Delta) = 2 cos(Delta);
* hand-worked YaRN ramp bounds (10 and 23 for DeepSeek-V3.2's values);
* YaRN's wavelength criterion, checked pair by pair: a pair turning more than
  beta_fast times over the original context keeps its angle, one turning
  less than beta_slow times is divided by the scale, the rest lie between;
* the rotation-matrix form of g: 1^T R_Delta 1 with R_Delta built as a
  block-diagonal matrix of 2x2 rotations (the sine terms cancel), evaluated
  with a matrix product;
* brute force: the selection rule on tiny vectors full of ties, and P_static
  on a short range with g summed by ``math.cos`` in pure Python;
* invariants of P_static at full length (distinct, ascending, every selected
  g >= every unselected g, value multiset = the K largest);
* the synthetic workload at zero noise equals g rounded to float32 (an
  independent implementation of the same angles and rotations);
* planted mistakes: mutated copies of the oracle must fail a pin.
"""
import importlib.util
import math
import re

import numpy as np
import pytest

from oracle import rope_prior as RP
from workloads import rope as WR

OTHER = dict(d=128, base=500000.0, scale=8.0, orig_ctx=8192, beta_fast=32.0, beta_slow=1.0)


def check_plain_angles(m):
    th = m.rope_theta(64, 10000.0)
    assert th.shape == (32,)
    for i, v in ((0, 1.0), (8, 0.1), (16, 0.01), (24, 0.001)):
        assert abs(th[i] - v) <= 1e-15 * v, (i, th[i])
    # scale 1 turns YaRN off
    assert np.allclose(m.yarn_theta(scale=1.0), th, rtol=1e-15, atol=0)


def check_bounds(m):
    # 64 ln(4096 / (64 pi)) / (2 ln 1e4) = 10.47..., 64 ln(4096 / (2 pi)) / (2 ln 1e4) = 22.51...
    assert m.yarn_bounds(64, 10000.0, 4096, 32.0, 1.0) == (10, 23)
    # 128 ln(8192 / (64 pi)) / (2 ln 5e5) = 128 * 3.707 / 26.245 = 18.08...,
    # 128 ln(8192 / (2 pi)) / (2 ln 5e5) = 128 * 7.173 / 26.245 = 34.98...
    assert m.yarn_bounds(128, 500000.0, 8192, 32.0, 1.0) == (18, 35)


def check_wavelength_rule(m):
    for p in (RP.DEFAULTS, OTHER):
        th = m.yarn_theta(**p)
        base_th = np.array([p["base"] ** (-2.0 * i / p["d"]) for i in range(p["d"] // 2)])
        turns = p["orig_ctx"] * base_th / (2.0 * math.pi)
        kept = turns > p["beta_fast"]
        slowed = turns < p["beta_slow"]
        assert kept.any() and slowed.any()
        assert np.allclose(th[kept], base_th[kept], rtol=1e-14, atol=0)
        assert np.allclose(th[slowed], base_th[slowed] / p["scale"], rtol=1e-14, atol=0)
        assert np.all(th <= base_th * (1 + 1e-14)) and np.all(th >= base_th / p["scale"] * (1 - 1e-14))
        assert np.all(np.diff(th) < 0), "angles must decrease with the pair index"


def check_g_rotation_form(m):
    rng = np.random.default_rng(3)
    for p in (RP.DEFAULTS, OTHER):
        th = m.yarn_theta(**p)
        d = p["d"]
        n = 140000
        g = m.g_delta(n, th)
        ones = np.ones(d)
        for delta in [0, 1, 2, 7, 4095, 4096, 70689, n - 1] + list(rng.integers(0, n, 6)):
            R = np.zeros((d, d))
            for i, t in enumerate(th):
                c, s = math.cos(delta * t), math.sin(delta * t)
                R[2 * i:2 * i + 2, 2 * i:2 * i + 2] = [[c, -s], [s, c]]
            ref = ones @ R @ ones
            assert abs(g[delta] - ref) <= 1e-9, (delta, g[delta], ref)


def check_g_closed_forms(m):
    th = m.yarn_theta()
    g = m.g_delta(100000, th)
    assert g[0] == 64.0
    assert np.all(np.abs(g) <= 64.0 + 1e-12)
    one = m.g_delta(1000, np.array([1.0]))
    assert np.allclose(one, [2.0 * math.cos(k) for k in range(1000)], rtol=0, atol=1e-13)


def brute_topk(vals, K):
    n = len(vals)
    if n <= K:
        return list(range(n)) + [-1] * (K - n)
    order = sorted(range(n), key=lambda i: (-vals[i], i))
    return sorted(order[:K])


def check_argtopk_ties(m):
    rng = np.random.default_rng(5)
    for case in range(200):
        n = int(rng.integers(0, 30))
        levels = rng.standard_normal(int(rng.integers(1, 4)))
        v = levels[rng.integers(0, len(levels), n)] if n else np.zeros(0)
        for K in {1, 3, max(n - 1, 1), max(n, 1), n + 2}:
            got = m.argtopk(v, K).tolist()
            assert got == brute_topk(v.tolist(), K), (case, v.tolist(), K, got)


def check_prior_small(m):
    th = m.yarn_theta()
    for n, K in ((50, 10), (300, 64), (9, 20)):
        g = [2.0 * sum(math.cos(delta * t) for t in th) for delta in range(n)]
        assert m.static_prior(n, K, th).tolist() == brute_topk(g, K), (n, K)


def check_prior_invariants(m, n=131072, K=2048):
    th = m.yarn_theta()
    g = m.g_delta(n, th)
    P = m.static_prior(n, K, th)
    assert P.shape == (K,) and P.dtype == np.int32
    assert np.all(np.diff(P) > 0) and P[0] >= 0 and P[-1] < n
    mask = np.zeros(n, bool)
    mask[P] = True
    assert g[mask].min() >= g[~mask].max()
    assert np.array_equal(np.sort(g[mask]), np.sort(g)[-K:])


ALL_CHECKS = [check_plain_angles, check_bounds, check_wavelength_rule, check_g_rotation_form,
              check_g_closed_forms, check_argtopk_ties, check_prior_small, check_prior_invariants]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=[c.__name__ for c in ALL_CHECKS])
def test_oracle_pin(check):
    check(RP)


def test_synthetic_rows_at_zero_noise_are_g():
    """Independent implementations: workload rotations with amp = 0 vs oracle g."""
    th = RP.yarn_theta()
    assert np.allclose(WR.angles(), th, rtol=1e-15, atol=0)
    for n in (1, 5000, 70690):
        s = WR.row_scores(n, amp=0.0)
        assert s.dtype == np.float32 and s.shape == (n,)
        assert np.max(np.abs(s.astype(np.float64) - RP.g_delta(n, th))) <= 2.0 ** -18


def test_synthetic_rows_seeded_and_correlated_with_prior():
    a = WR.row_scores(8192, row=2)
    assert np.array_equal(a, WR.row_scores(8192, row=2))
    assert not np.array_equal(a, WR.row_scores(8192, row=3))
    th = RP.yarn_theta()
    P = RP.static_prior(8192, 2048, th)
    top = RP.argtopk(a.astype(np.float64), 2048)
    # the prior is a guess, not the answer: large overlap, not equality
    overlap = len(np.intersect1d(P, top)) / 2048
    assert 0.5 < overlap < 1.0, overlap


MUTATIONS = [
    ("factor 2 dropped", r"return 2\.0 \* np\.cos", "return np.cos"),
    ("ramp reversed", r"theta \* \(1\.0 - gamma\) \+ \(theta / scale\) \* gamma",
     "theta * gamma + (theta / scale) * (1.0 - gamma)"),
    ("lower bound rounded up", r"lo = max\(math\.floor\(", "lo = max(math.ceil("),
    ("exponent without the 2", r"-2\.0 \* i / d", "-i / d"),
    ("ties to the higher index", r'np\.argsort\(-v, kind="stable"\)', 'np.argsort(v, kind="stable")[::-1]'),
    ("sine for cosine", r"np\.cos\(np\.outer", "np.sin(np.outer"),
    ("first element dropped", r"np\.sort\(order\[:K\]\)", "np.sort(order[1:K + 1])"),
]


@pytest.mark.parametrize("name,pattern,repl", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(tmp_path, name, pattern, repl):
    src = open(RP.__file__).read()
    mutated, nsub = re.subn(pattern, repl, src)
    assert nsub >= 1, "mutation pattern no longer matches the oracle source"
    path = tmp_path / "mutant_rope_prior.py"
    path.write_text(mutated)
    spec = importlib.util.spec_from_file_location("mutant_rope_prior", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    caught = 0
    for check in ALL_CHECKS:
        try:
            check(mod)
        except AssertionError:
            caught += 1
    assert caught, "mutation '%s' was not caught by any pin" % name
