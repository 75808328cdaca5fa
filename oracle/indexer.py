"""CPU oracle for the FP8 indexer scores -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module; the GPU product path never does, and the
two share no code. Plain numpy in float64.

What it computes (Sec. 2.1, Eq. indexer): for query row b of a decode batch
and past token s,

    I[b][s] = sum_j w[b][j] * ReLU( q[b][j] . k'[g][s] ),  k'[g][s] = k_scale[g][s] * k[g][s],

with g = b // group (rows of one request share its key cache) and q, k given
as FP8 E4M3 bytes of the OCP format: 1 sign bit, 4 exponent bits with bias 7,
3 mantissa bits; exponent 0 holds the subnormals m / 8 * 2^-6; the pattern
with every exponent and mantissa bit set is NaN; there are no infinities.
The decoding is written from that definition, the products and sums are
exact float64 operations up to the final rounding of each dot product.

Parity status: pinned by ``tests/test_indexer_pins.py`` (every byte decoded
against torch's float8_e4m3fn, hand-decoded values, a pure-Python loop
version on small shapes, ReLU and scale-sign cases, linearity in w, cache
sharing by group; ``magnitude`` against a pure-Python loop, equal to the
score when no term can cancel and never below |score|; planted mistakes).
"""
from __future__ import annotations

import numpy as np


def decode_e4m3(b) -> np.ndarray:
    """float64 values of OCP FP8 E4M3 bytes."""
    u = np.asarray(b, dtype=np.uint8).astype(np.int64)
    sign = np.where(u >> 7, -1.0, 1.0)
    e = (u >> 3) & 15
    m = u & 7
    normal = (1.0 + m / 8.0) * np.exp2(e - 7.0)
    sub = (m / 8.0) * 2.0 ** -6
    v = sign * np.where(e == 0, sub, normal)
    return np.where((e == 15) & (m == 7), np.nan, v)


def indexer_scores(q, w, k, k_scale, group: int = 1, row_len=None) -> np.ndarray:
    """I [B][ld] float64 (Sec. 2.1, Eq. indexer); entries s >= n_b are NaN.

    q [B][H][D] uint8, w [B][H], k [B/group][ld][D] uint8, k_scale [B/group][ld].
    """
    q = np.asarray(q)
    k = np.asarray(k)
    w = np.asarray(w, dtype=np.float64)
    k_scale = np.asarray(k_scale, dtype=np.float64)
    B, H, D = q.shape
    ld = k.shape[1]
    out = np.full((B, ld), np.nan)
    for b in range(B):
        n = ld if row_len is None else int(min(max(int(row_len[b]), 0), ld))
        if n == 0:
            continue
        g = b // group
        Q = decode_e4m3(q[b])                                   # [H][D]
        Kd = decode_e4m3(k[g, :n]) * k_scale[g, :n, None]       # [n][D]: k'
        logits = Q @ Kd.T                                       # [H][n]
        out[b, :n] = w[b] @ np.maximum(logits, 0.0)
    return out


def magnitude(q, w, k, k_scale, group: int = 1, row_len=None) -> np.ndarray:
    """sum_j |w_j| sum_d |q_jd k'_d| per score: the scale of its rounding error."""
    q = np.asarray(q)
    k = np.asarray(k)
    B, H, D = q.shape
    ld = k.shape[1]
    out = np.full((B, ld), np.nan)
    for b in range(B):
        n = ld if row_len is None else int(min(max(int(row_len[b]), 0), ld))
        if n == 0:
            continue
        g = b // group
        Q = np.abs(decode_e4m3(q[b]))
        Kd = np.abs(decode_e4m3(k[g, :n]) * np.asarray(k_scale, dtype=np.float64)[g, :n, None])
        out[b, :n] = np.abs(np.asarray(w, dtype=np.float64)[b]) @ (Q @ Kd.T)
    return out
