"""Seeded synthetic indexer rows built from random queries and keys under
YaRN-scaled RoPE (the paper's synthetic single-operator benchmark, Sec. 6.3.1
and the synthetic-data appendix).

Each row is one query scoring keys j = 0 .. n-1 that sit j positions away
from it, on the rotary dimensions only (d = 64): the query and every key are
1 + amp * N(0, 1) per dimension (amp = 0.1), rotary pair i rotates by the
angle j * theta'_i between the query and key j, and the score is the dot
product of the rotated vectors,

    s_j = sum_i (q_a k_a + q_b k_b) cos(j theta'_i) + (q_b k_a - q_a k_b) sin(j theta'_i),

with pair i made of dimensions a = i and b = i + d/2. With amp = 0 every
score is g(j) of Sec. 3.2, so the static prior P_static of Sec. 3.3 is a good
(not exact) guess of each row's Top-K. The angles follow DeepSeek-V3.2's YaRN
setting (base 1e4, scale 40, original context 4096, ramp 32 .. 1 rotations);
this module computes them itself for the data only. Scores are formed in
float64 and rounded once to float32.

Random numbers: ``numpy.random.default_rng((61, n, row))``, drawn as the
query (d values) then the keys (n x d values).
"""
from __future__ import annotations

import math

import numpy as np

K_TOPK = 2048
# The sequence lengths of the paper's synthetic latency table (Sec. 6.3.1).
N_LIST = (8192, 16384, 32768, 65536, 70690, 131072)
AMP = 0.1
ROPE = dict(d=64, base=10000.0, scale=40.0, orig_ctx=4096, beta_fast=32.0, beta_slow=1.0)


def angles(d=64, base=10000.0, scale=40.0, orig_ctx=4096, beta_fast=32.0, beta_slow=1.0) -> np.ndarray:
    """Per-pair rotation rate of the model (YaRN: fast pairs kept, slow pairs
    divided by ``scale``, a linear ramp over the pair index in between)."""
    half = d // 2
    log_base = math.log(base)

    def edge(rotations):
        # pair index at which a pair turns `rotations` times over orig_ctx
        return d * math.log(orig_ctx / (rotations * 2.0 * math.pi)) / (2.0 * log_base)

    first = max(math.floor(edge(beta_fast)), 0)
    last = min(math.ceil(edge(beta_slow)), d - 1)
    span = max(last - first, 1e-3)
    out = np.empty(half, dtype=np.float64)
    for i in range(half):
        rate = base ** (-2.0 * i / d)
        w = min(max((i - first) / span, 0.0), 1.0)
        out[i] = rate * (1.0 - w) + (rate / scale) * w
    return out


def row_scores(n: int, row: int = 0, amp: float = AMP, rope=None) -> np.ndarray:
    """float32 [n] scores of one synthetic row (see the module docstring)."""
    r = dict(ROPE if rope is None else rope)
    d = r["d"]
    half = d // 2
    rng = np.random.default_rng((61, int(n), int(row)))
    q = 1.0 + amp * rng.standard_normal(d)
    k = 1.0 + amp * rng.standard_normal((n, d))
    theta = angles(**r)
    j = np.arange(n, dtype=np.float64)[:, None]
    phase = j * theta[None, :]
    qa, qb = q[:half], q[half:]
    ka, kb = k[:, :half], k[:, half:]
    s = ((ka * qa + kb * qb) * np.cos(phase) + (ka * qb - kb * qa) * np.sin(phase)).sum(axis=1)
    return s.astype(np.float32)


def batch_scores(n: int, rows: int, amp: float = AMP, rope=None) -> np.ndarray:
    """float32 [rows][n]: ``rows`` independent synthetic rows of length n."""
    return np.stack([row_scores(n, r, amp, rope) for r in range(rows)])
