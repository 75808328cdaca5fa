"""CPU replay of gvr_topk's default control flow (test infrastructure).

Predicts, for every row of a call, the path the kernel takes and its number
of full-row passes from the same fp32 rows, with integer arithmetic only, so
that the GPU's per-row stats (``gvr_row_stats``) can be compared with an
independent prediction (the paper replays its own kernel's control flow to
count Phase 2 iterations, Appendix "Per-Phase Timing Measurement
Methodology"). The steps follow the method:

* Phase 1 (Sec. 4.2.1) on a strided sample of prev_topk: every st-th entry,
  st = ceil(K / 256); keys of the valid gathered scores; a histogram of 1024
  bins over [pmin, pmax]; the speculative threshold T_spec is the lower edge
  of the bin holding the sampled key of rank ceil(65 m / 2048) from the
  bottom (m valid samples), and at least key 1.
* One pass counts f(T_spec) = #{key >= T_spec} (Sec. 4.1) per streaming wave
  (a wave's list holds 1024 entries); K <= f <= C accepts it (Lemma 1).
* Otherwise, if K <= f <= C (a list overflowed), one collect pass at T_spec
  (a part of one row) or again at exact per-wave offsets (one part). If
  f > C, the first refine level (2048 bins of 2^s keys from T_spec, s the
  smallest shift whose bins span [T_spec, max(pmax, T_spec)], higher keys in
  the top bin) counts every key >= T_spec: the bin holding the K-th key gives
  T' = its lower edge, and if f(T') <= C one collect pass lists the keys >= T'
  (each of the 16 waves its full-row share, up to 1024 entries; a share
  past that costs one more pass at exact offsets).
* Otherwise count passes narrow a window of 256 bins around the K-th key
  (each evaluates f at 257 thresholds) until a threshold with K <= f <= C is
  found (one collect pass) or the K-th key is isolated (one emit pass).
* Without a guess (the radix schedule) nothing bounds the K-th key: a digit
  pass counts the top 11 key bits of every element (2048 bins); the bin
  holding the K-th key is collected (as above) or narrowed.

The row split (parts, workgroup slabs) mirrors the launch the library plans
for the 16-wave shape: rows of a call up to the number of compute units.
"""
from __future__ import annotations

import numpy as np

K_MAX = 2048
CAP = 16384            # C of the 16-wave shape
WAVES = 16             # waves per workgroup; wave 0 computes the guess
WAVE_CAP = 1024        # list entries per wave
GUESS_SAMPLES = 256
GUESS_BINS_LG = 10     # 1024 bins
REF_BINS_LG = 11       # first refine level: 2048 bins
SPEC_QUANTILE = 65
WINDOW_BINS_LG = 8     # 256 bins per counting window
DIGIT_SHIFT = 21       # radix digit: key >> 21
MAX_PARTS = 16
MIN_PART_ELEMS = 16384
PATH = {"trivial": 0, "all": 1, "guess": 2, "narrowed": 3, "ties": 4, "no_guess": 5}


def keys(x: np.ndarray) -> np.ndarray:
    """Sortable keys of fp32 values: flip all bits of negatives, the sign bit of the rest."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    neg = (u >> 31) == 1
    return np.where(neg, (~u) & 0xFFFFFFFF, u | 0x80000000).astype(np.uint64)


def bin_shift(width: int, lg_bins: int) -> int:
    """Smallest s with (2^lg_bins << s) >= width."""
    bits = int(width - 1).bit_length() if width > 1 else 0
    return max(0, bits - lg_bins)


def choose_parts(rows: int, ld: int, cus: int = 256) -> int:
    """Workgroups per row of an automatic split (the library's rule)."""
    if rows <= 0 or rows >= cus:
        return 1
    if rows <= 2 and ld >= 32768 and cus >= 32 * rows:
        return 8 if ld < 196608 else MAX_PARTS
    if ld >= 49152 and cus // rows >= 4:
        return min(cus // rows, MAX_PARTS, 8 if ld < 196608 else MAX_PARTS)
    s = cus // rows
    s = min(s, max(1, ld // MIN_PART_ELEMS), MAX_PARTS)
    if s <= 1:
        return 1
    stream_us = ld * 4.0 / 33.0e3
    return s if stream_us * (1.0 - 1.0 / s) > 8.0 else 1


def spec_threshold(xk: np.ndarray, n: int, prev: np.ndarray | None, K: int, with_max: bool = False):
    """(T_spec, valid samples) of Phase 1 on the sampled guess; T_spec None
    without a valid sample. With `with_max`, also pmax (largest sampled key)."""
    st = -(-K // GUESS_SAMPLES)
    m = -(-K // st)
    if prev is None:
        return (None, 0, 0) if with_max else (None, 0)
    idx = np.asarray(prev[: m * st: st][:m], dtype=np.int64)
    ok = (idx >= 0) & (idx < n)
    if not ok.any():
        return (None, 0, 0) if with_max else (None, 0)
    gk = xk[idx[ok]]
    mn, mx = int(gk.min()), int(gk.max())
    sh = bin_shift(mx - mn + 1, GUESS_BINS_LG)
    h = np.bincount(((gk - mn) >> sh).astype(np.int64), minlength=1 << GUESS_BINS_LG)
    cnt = int(ok.sum())
    target = max(1, -(-SPEC_QUANTILE * cnt // K_MAX))
    b = int(np.argmax(np.cumsum(h) >= target))
    t = max(mn + (b << sh), 1)
    return (t, cnt, mx) if with_max else (t, cnt)


def wave_ranges(n: int, aoff: int, parts: int, part: int):
    """Element ranges [lo, hi) of the streaming waves 1..15 of one part."""
    nq = (n + aoff + 3) >> 2
    nslab = (nq + 63) >> 6
    ps = -(-nslab // parts)
    ps0 = min(part * ps, nslab)
    ps1 = min(ps0 + ps, nslab)
    ws = -(-(ps1 - ps0) // (WAVES - 1)) if ps1 > ps0 else 0
    out = []
    for sw in range(WAVES - 1):
        s0 = min(ps0 + sw * ws, ps1)
        s1 = min(ps0 + min((sw + 1) * ws, ps1 - ps0), ps1) if ws else s0
        out.append((max(0, 256 * s0 - aoff), max(0, min(n, 256 * s1 - aoff))))
    return out, ws


def count_ge(xk: np.ndarray, t: int) -> int:
    return int((xk >= t).sum())


def row_share_overflow(xk: np.ndarray, n: int, aoff: int, t: int) -> bool:
    """Some wave's full-row share (16 waves, whole slabs each) holds more
    than a list's 1024 keys >= t."""
    nq = (n + aoff + 3) >> 2
    nslab = (nq + 63) >> 6
    per = -(-nslab // WAVES) * 64
    for w in range(WAVES):
        qb = min(w * per, nq)
        qe = min(qb + per, nq)
        lo, hi = max(0, 4 * qb - aoff), max(0, min(n, 4 * qe - aoff))
        if hi > lo and count_ge(xk[lo:hi], t) > WAVE_CAP:
            return True
    return False


def kth_level_bin(xk: np.ndarray, K: int, t: int, gmax: int):
    """The first refine level over [t, max(gmax, t)]: (lower edge, upper edge
    (0xFFFFFFFF for the open top bin), keys in the bins above, the bin's count)
    of the bin holding the K-th key."""
    sh = bin_shift(max(gmax, t) - t + 1, REF_BINS_LG)
    kk = xk[xk >= t]
    b = np.minimum((kk - t) >> sh, (1 << REF_BINS_LG) - 1).astype(np.int64)
    h = np.bincount(b, minlength=1 << REF_BINS_LG)
    above = np.concatenate([np.cumsum(h[::-1])[::-1][1:], [0]])   # keys in the bins above each bin
    j = int(np.nonzero((above < K) & (above + h >= K))[0][0])
    lo = t + (j << sh)
    hi = 0xFFFFFFFF if j == (1 << REF_BINS_LG) - 1 else min(lo + (1 << sh) - 1, 0xFFFFFFFF)
    return lo, hi, int(above[j]), int(h[j])


def digit_then(xk: np.ndarray, n: int, aoff: int, K: int, cap: int, passes: int):
    """The digit pass and what follows it: (outcome, passes, threshold, candidates)."""
    h = np.bincount((xk >> DIGIT_SHIFT).astype(np.int64), minlength=1 << (32 - DIGIT_SHIFT))
    above = np.concatenate([np.cumsum(h[::-1])[::-1][1:], [0]])
    j = int(np.nonzero((above < K) & (above + h >= K))[0][0])
    lo = j << DIGIT_SHIFT
    hi = lo + (1 << DIGIT_SHIFT) - 1
    if above[j] + h[j] <= cap:
        extra = 1 if row_share_overflow(xk, n, aoff, lo) else 0
        return "collect", passes + 2 + extra, lo, int(above[j] + h[j])
    return narrow(xk, K, cap, lo, hi, passes + 1)


def narrow(xk: np.ndarray, K: int, cap: int, lo: int, hi: int, passes: int):
    """Count passes over 256-bin windows starting from [lo, hi] (from the
    row's [min, max] after one min/max pass when nothing bounds the K-th key,
    [lo, hi] = the whole key range); returns (outcome, passes, threshold,
    candidates)."""
    def window(a, b):
        return a, bin_shift(b - a + 1, WINDOW_BINS_LG)

    if lo == 0 and hi == 0xFFFFFFFF:
        passes += 1
        lo, hi = int(xk.min()), int(xk.max())
    wlo, ws = window(lo, hi)
    while True:
        passes += 1                                   # one count pass
        edges = [wlo + (j << ws) for j in range(1 << WINDOW_BINS_LG)] + [wlo + ((1 << WINDOW_BINS_LG) << ws)]
        F = [count_ge(xk, e) if e <= 0xFFFFFFFF else 0 for e in edges] + [0]
        F[0] = count_ge(xk, wlo)
        j = -1
        for c in range(len(F) - 1):
            if F[c] >= K and F[c + 1] < K:
                j = c
        if j < 0:
            wlo, ws = window(0, wlo - 1)
            continue
        if F[j] <= cap:
            return "collect", passes + 1, edges[j], F[j]
        if j == (1 << WINDOW_BINS_LG):
            wlo, ws = window(edges[j], 0xFFFFFFFF)
            continue
        if ws == 0:
            return "ties", passes + 1, edges[j], 0
        e = edges[j]
        wlo, ws = window(e, min(e + (1 << ws) - 1, 0xFFFFFFFF))


def replay_row(x: np.ndarray, n: int, prev: np.ndarray | None, K: int, parts: int, aoff: int, cap: int = CAP):
    """Predicted {path, passes, spec_threshold, spec_count, threshold, candidates} of one row."""
    n = max(0, min(int(n), x.shape[0]))
    if n <= K:
        return {"path": PATH["trivial"], "passes": 0}
    xk = keys(x[:n])
    res = {}
    # every element is a candidate: short rows (n <= 2K) whose waves hold them all
    nq = (n + aoff + 3) >> 2
    nslab = (nq + 63) >> 6
    ps = -(-nslab // parts)
    ws_all = -(-min(ps, nslab) // (WAVES - 1))
    all_mode = (prev is None or n <= 2 * K) and n <= cap and ws_all * 256 <= WAVE_CAP
    if all_mode:
        return {"path": PATH["all"], "passes": 1, "candidates": n}
    if prev is None:   # the guess-free kernel: a digit pass, then collect or narrow
        outcome, passes, thr, cands = digit_then(xk, n, aoff, K, cap, 0)
        return {"path": PATH["ties" if outcome == "ties" else "no_guess"], "passes": passes, "threshold": thr,
                "candidates": cands}
    tspec, gvalid, gmax = spec_threshold(xk, n, prev, K, with_max=True)
    have_prev = prev is not None and gvalid > 0
    t = tspec if tspec is not None else 0xFFFFFFFF
    res["spec_threshold"] = t
    # the speculative pass: per-part, per-wave counts at T_spec
    f = 0
    overflow = False
    for part in range(parts):
        ranges, _ = wave_ranges(n, aoff, parts, part)
        for lo, hi in ranges:
            c = count_ge(xk[lo:hi], t) if hi > lo else 0
            overflow |= c > WAVE_CAP
            f += c
    # every wave counts past its list's capacity: f(T_spec) is exact on every path
    res["spec_count"] = f
    path = "guess" if have_prev else "no_guess"
    if not overflow and K <= f <= cap:
        res.update(path=PATH[path], passes=1, threshold=t, candidates=f)
        return res
    if overflow and parts == 1 and K <= f <= cap:      # collected again at packed offsets
        res.update(path=PATH[path], passes=2, threshold=t, candidates=f)
        return res
    p = "narrowed" if path == "guess" else "no_guess"
    if K <= f <= cap:                                  # a part's list overflowed: collect at T_spec
        extra = 1 if row_share_overflow(xk, n, aoff, t) else 0
        res.update(path=PATH[p], passes=2 + extra, threshold=t, candidates=f)
        return res
    if f < K:
        lo, hi = 0, t - 1
    else:                                              # f > C: the K-th key's bin of the first refine level
        lo, hi, above, cnt = kth_level_bin(xk, K, t, gmax)
        if above + cnt <= cap:
            extra = 1 if row_share_overflow(xk, n, aoff, lo) else 0
            res.update(path=PATH[p], passes=2 + extra, threshold=lo, candidates=above + cnt)
            return res
    outcome, passes, thr, cands = narrow(xk, K, cap, lo, hi, 1)
    p = "ties" if outcome == "ties" else ("narrowed" if path == "guess" else "no_guess")
    res.update(path=PATH[p], passes=passes, threshold=thr, candidates=cands)
    return res
