"""CPU oracle for the static RoPE/YaRN prior -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module; the GPU product path never does, and the
two share no code. Everything here is plain numpy in float64.

What it computes (Sec. 3.2 "Theoretical Basis", Sec. 3.3 "Pre-Computed
Candidate Indices"):

* ``rope_theta``   -- the RoPE angle of rotary pair i: theta_i = base^(-2i/d)
                      (Sec. 3.2, the equation defining g).
* ``yarn_bounds``  -- the first and last pair index of YaRN's interpolation
                      ramp for an original context L and the two ramp
                      parameters (rotations over L) beta_fast > beta_slow.
* ``yarn_theta``   -- the YaRN-scaled angles theta'_i: pairs that turn many
                      times over L keep theta_i, pairs that turn less than
                      once are divided by the scale s, and a linear ramp in i
                      blends the two in between (Sec. 3.2 "YaRN extension";
                      the parameter values d = 64, base = 1e4, s = 40,
                      L = 4096, beta_fast = 32, beta_slow = 1 are the ones
                      the synthetic-data appendix uses for DeepSeek-V3.2).
* ``g_delta``      -- g(Delta) = 2 sum_i cos(Delta theta'_i) for
                      Delta = 0 .. n-1 (Sec. 3.2, equation for g).
* ``argtopk``      -- the K largest values of a float64 vector, the lower
                      index first among equal values, returned in ascending
                      index order; 0..n-1 then -1 when n <= K.
* ``static_prior`` -- P_static = argtopk over Delta in [0, n) of g(Delta)
                      (Sec. 3.3, equation for the static index set).

Readings where the paper leaves a choice (each listed in the design notes):

* the ramp bounds are lo = max(floor(x(beta_fast)), 0) and
  hi = min(ceil(x(beta_slow)), d - 1) with
  x(beta) = d ln(L / (2 pi beta)) / (2 ln base), and the ramp is
  clamp((i - lo) / max(hi - lo, 1e-3), 0, 1) -- the synthetic-data
  appendix's frequency rule;
* angles, g and the selection are all float64 (the definition; the kernel
  decides in float64 too);
* Delta = j is the distance of key j from the query, so P_static holds key
  indices directly, as in the paper's synthetic benchmark.

Parity status: pinned by ``tests/test_rope_pins.py`` (hand-worked ramp
bounds, the wavelength criterion of YaRN, the rotation-matrix form of g,
closed forms for one pair, brute-force selection with ties, the synthetic
workload at zero noise, planted mistakes).
"""
from __future__ import annotations

import math

import numpy as np

# DeepSeek-V3.2 indexer RoPE (synthetic-data appendix; Sec. 3.2, 3.3).
DEFAULTS = dict(d=64, base=10000.0, scale=40.0, orig_ctx=4096, beta_fast=32.0, beta_slow=1.0)


def rope_theta(d: int, base: float) -> np.ndarray:
    """theta_i = base ** (-2 i / d), i = 0 .. d/2 - 1 (Sec. 3.2, equation for g)."""
    i = np.arange(d // 2, dtype=np.float64)
    return np.power(float(base), -2.0 * i / d)


def yarn_bounds(d: int, base: float, orig_ctx: int, beta_fast: float, beta_slow: float):
    """Ramp bounds (lo, hi) in pair indices (reading stated in the module header)."""
    def x(beta):
        return d * math.log(orig_ctx / (2.0 * math.pi * beta)) / (2.0 * math.log(base))
    lo = max(math.floor(x(beta_fast)), 0)
    hi = min(math.ceil(x(beta_slow)), d - 1)
    return lo, hi


def yarn_theta(d: int = 64, base: float = 10000.0, scale: float = 40.0, orig_ctx: int = 4096,
               beta_fast: float = 32.0, beta_slow: float = 1.0) -> np.ndarray:
    """theta'_i = (1 - gamma_i) theta_i + gamma_i theta_i / s (Sec. 3.2, YaRN)."""
    theta = rope_theta(d, base)
    lo, hi = yarn_bounds(d, base, orig_ctx, beta_fast, beta_slow)
    i = np.arange(d // 2, dtype=np.float64)
    gamma = np.clip((i - lo) / max(hi - lo, 1e-3), 0.0, 1.0)
    return theta * (1.0 - gamma) + (theta / scale) * gamma


def g_delta(n: int, theta: np.ndarray) -> np.ndarray:
    """g(Delta) = 2 sum_i cos(Delta theta_i), Delta = 0 .. n-1 (Sec. 3.2)."""
    delta = np.arange(n, dtype=np.float64)
    return 2.0 * np.cos(np.outer(delta, theta)).sum(axis=1)


def argtopk(values: np.ndarray, K: int) -> np.ndarray:
    """Indices of the K largest values (lower index first among equals),
    ascending; 0..n-1 then -1 padding when n <= K."""
    v = np.asarray(values, dtype=np.float64)
    n = v.shape[0]
    out = np.full(K, -1, dtype=np.int32)
    if n <= K:
        out[:n] = np.arange(n, dtype=np.int32)
        return out
    # A stable sort on -v keeps equal values in index order.
    order = np.argsort(-v, kind="stable")
    out[:] = np.sort(order[:K]).astype(np.int32)
    return out


def static_prior(n: int, K: int, theta: np.ndarray) -> np.ndarray:
    """P_static = argtopk_{0 <= Delta < n} g(Delta) (Sec. 3.3)."""
    return argtopk(g_delta(n, theta), K)
