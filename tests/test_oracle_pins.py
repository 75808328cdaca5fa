"""Pins for the CPU oracle (no GPU).

The oracle computes the plain definition of exact Top-K (Sec. 4.1, problem
statement; f(T) and Lemma 1 of the same section). These tests tie it to
things other than itself:

* brute force: a pure-Python full sort on tiny rows drawn from 2-5 levels, so
  ties dominate, with an order written from IEEE-754 semantics (not from the
  oracle's bit trick);
* the pairwise definition of "the K largest, lower index first";
* closed forms: rows with a known answer (n <= K, constant, increasing,
  decreasing), x_i = i for f(T), the hand-ordered list of special values;
* invariants at full size that characterise the answer uniquely: K distinct
  indices, #{key > T*} < K <= #{key >= T*}, every key > T* taken, ties
  resolved by index (Lemma 1 gives the containment these rest on);
* numpy: ``argpartition`` on distinct rows (set equality, the paper's own
  correctness check against a library Top-K, Sec. 6.2) and ``np.sort`` on any
  row (the value multiset of a Top-K is unique whatever the tie rule);
* planted mistakes: a mutated copy of the oracle source must fail the pins.
"""
import math
import os
import re
import shutil
import struct

import numpy as np
import pytest

import oracle

K_DEFAULT = 2048


def f32_from_bits(u: int) -> float:
    return struct.unpack("<f", struct.pack("<I", u & 0xFFFFFFFF))[0]


def bits_of(x: float) -> int:
    return struct.unpack("<I", struct.pack("<f", x))[0]


# Ascending total order, written out by hand from IEEE-754 (Sec. 2.2 names the
# "sortable FP32 score key"; the place of NaNs and of -0.0 is this build's
# reading): negative NaNs (larger payload = smaller), -inf, negative finite
# values, -0.0, +0.0, positive finite values, +inf, positive NaNs.
ORDERED_BITS = [
    0xFFFFFFFF, 0xFFC00000, 0xFF800001,              # -NaN, larger payload first
    0xFF800000,                                      # -inf
    bits_of(-3.4028234663852886e38),                 # -FLT_MAX
    bits_of(-1.0), bits_of(-1.1754943508222875e-38),  # -1, -FLT_MIN
    0x80000001,                                      # -denorm_min
    0x80000000, 0x00000000,                          # -0.0, +0.0
    0x00000001, bits_of(1.1754943508222875e-38),     # denorm_min, FLT_MIN
    bits_of(1.0), bits_of(1.0000001192092896),       # 1, nextafter(1)
    bits_of(3.4028234663852886e38), 0x7F800000,      # FLT_MAX, +inf
    0x7F800001, 0x7FC00000, 0x7FFFFFFF,              # +NaN, larger payload last
]


def total_order_rank(x: float):
    """Sort key of a non-NaN float in the total order (ascending)."""
    assert not math.isnan(x)
    return (x, 0 if math.copysign(1.0, x) < 0 else 1)


def brute_topk(row, K):
    """Full stable sort by (larger first, lower index first), first K, ascending."""
    n = len(row)
    if n <= K:
        return list(range(n)) + [-1] * (K - n)
    order = sorted(range(n), key=lambda i: (tuple(-v for v in total_order_rank(float(row[i]))), i))
    return sorted(order[:K])


def pairwise_ok(row, sel, K):
    """Every selected i beats every unselected j: larger, or equal and i < j."""
    n = len(row)
    s = set(int(i) for i in sel if i >= 0)
    if n <= K:
        return list(sel) == list(range(n)) + [-1] * (K - n)
    if len(s) != K or any(i < 0 or i >= n for i in s):
        return False
    r = [total_order_rank(float(v)) for v in row]
    for i in s:
        for j in range(n):
            if j in s:
                continue
            if not (r[i] > r[j] or (r[i] == r[j] and i < j)):
                return False
    return True


# ---------------------------------------------------------------- check sets
# Each returns a list of failure strings so that the planted-mistake test can
# run the same checks against a mutated oracle.

def check_key_order(o):
    fails = []
    # Built from raw bits so that NaN payloads survive.
    raw = np.array(ORDERED_BITS, dtype=np.uint32).view(np.float32)
    keys = o.key(raw)
    if not all(int(keys[i]) < int(keys[i + 1]) for i in range(len(keys) - 1)):
        fails.append("special values not strictly increasing: %s" % [hex(int(k)) for k in keys])
    if int(o.key(np.float32(0.0))) != 0x80000000:
        fails.append("key(+0.0) != 0x80000000")
    if int(o.key(np.float32(0.0))) - int(o.key(np.float32(-0.0))) != 1:
        fails.append("-0.0 and +0.0 are not adjacent keys")
    rng = np.random.default_rng(7)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-30, 30, 20000))).astype(np.float32)
    x = np.unique(x)
    k = o.key(x)
    if not np.array_equal(np.argsort(x, kind="stable"), np.argsort(k, kind="stable")):
        fails.append("key order differs from float order on finite values")
    return fails


def check_bruteforce(o, cases=300, seed=1):
    fails = []
    rng = np.random.default_rng(seed)
    pool = np.array([-np.inf, -2.5, -1.0, -0.0, 0.0, 0.5, 1.0, 3.0, np.inf], dtype=np.float32)
    for c in range(cases):
        n = int(rng.integers(0, 65))
        nlev = int(rng.integers(2, 6))
        levels = rng.choice(pool, size=nlev, replace=False)
        row = rng.choice(levels, size=n).astype(np.float32)
        K = int(rng.integers(1, 70))
        got = o.topk(row.reshape(1, n) if n else np.zeros((1, 0), np.float32), K, row_len=[n])[0][0]
        exp = brute_topk(row, K)
        if list(got) != exp:
            fails.append("case %d n=%d K=%d levels=%s: got %s expected %s" % (c, n, K, levels, list(got), exp))
        elif c % 3 == 0 and not pairwise_ok(row, got, K):
            fails.append("case %d pairwise check failed" % c)
        if len(fails) > 3:
            break
    return fails


def check_special_rows(o, K=K_DEFAULT):
    fails = []
    ld = 3 * K + 5
    rows = np.zeros((8, ld), dtype=np.float32)
    rows[0, :] = 1.25                                    # constant
    rows[1, :] = np.arange(ld, dtype=np.float32)         # increasing
    rows[2, :] = -np.arange(ld, dtype=np.float32)        # decreasing
    rows[3, :] = np.arange(ld, dtype=np.float32)         # n = K - 1
    rows[4, :] = np.arange(ld, dtype=np.float32)         # n = K
    rows[5, :] = 7.0                                     # n = 0
    rows[6, :] = np.arange(ld, dtype=np.float32)         # row_len > ld clamps
    rows[7, :] = np.arange(ld, dtype=np.float32)         # row_len < 0 -> 0
    rl = [ld, ld, ld, K - 1, K, 0, ld + 100, -5]
    idx, kth, ngt = o.topk(rows, K, row_len=rl)
    exp = [
        list(range(K)),
        list(range(ld - K, ld)),
        list(range(K)),
        list(range(K - 1)) + [-1],
        list(range(K)),
        [-1] * K,
        list(range(ld - K, ld)),
        [-1] * K,
    ]
    for r in range(8):
        if list(idx[r]) != exp[r]:
            fails.append("special row %d wrong (first entries %s)" % (r, list(idx[r][:6])))
    if int(kth[0]) != int(o.key(np.float32(1.25))) or int(ngt[0]) != 0:
        fails.append("constant row: kth/n_gt wrong")
    if int(kth[1]) != int(o.key(np.float32(ld - K))) or int(ngt[1]) != K - 1:
        fails.append("increasing row: kth/n_gt wrong")
    # Positive NaNs rank above +inf, negative NaNs below -inf.
    row = np.arange(100, dtype=np.float32)
    row_bits = row.view(np.uint32).copy()
    row_bits[[3, 50, 97]] = 0x7FC00000
    row_bits[[1, 2]] = 0xFFC00000
    row_bits[10] = 0x7F800000
    r2 = row_bits.view(np.float32)
    got = o.topk(r2, 5)[0][0]
    if list(got) != [3, 10, 50, 97, 99]:
        fails.append("NaN/inf row: got %s" % list(got))
    got = o.topk(-r2, 4)[0][0]          # negate: -NaN now lowest, +NaN (from the -NaN) highest
    if list(got) != [0, 1, 2, 4]:
        fails.append("negated NaN row: got %s" % list(got))
    return fails


def check_count_closed_forms(o):
    fails = []
    n = 1000
    x = np.arange(n, dtype=np.float32)
    for t in [0, 1, 17, 500, 999, 1000]:
        c = o.count_ge(x, int(o.key(np.float32(t))))
        if c != n - t:
            fails.append("f(%d) = %d, expected %d" % (t, c, n - t))
    if o.count_ge(x, int(o.key(np.float32(-np.inf)))) != n:
        fails.append("f(-inf) != n")
    if o.count_ge(x, int(o.key(np.float32(np.inf)))) != 0:
        fails.append("f(+inf) != 0")
    if o.count_ge(x, 0) != n:
        fails.append("f(smallest key) != n")
    if o.count_ge(x, int(o.key(np.float32(0.5))), n=10) != 9:
        fails.append("f with n prefix wrong")
    z = np.array([-0.0, 0.0, 0.0, -0.0], dtype=np.float32)
    if o.count_ge(z, int(o.key(np.float32(0.0)))) != 2:
        fails.append("f(+0.0) must not count -0.0")
    return fails


def check_invariants(o, seed=3, B=3, ld=60000, K=K_DEFAULT):
    """Lemma-1 style characterisation at full size on tie-heavy rows."""
    fails = []
    rng = np.random.default_rng(seed)
    rows = np.empty((B, ld), dtype=np.float32)
    rows[0] = rng.integers(0, 40, ld).astype(np.float32)            # 40 levels: heavy ties
    rows[1] = (rng.standard_normal(ld) * 3).astype(np.float16).astype(np.float32)
    rows[2] = rng.standard_normal(ld).astype(np.float32)
    rl = [ld, ld - 777, ld]
    idx, kth, ngt = o.topk(rows, K, row_len=rl)
    for b in range(B):
        n = rl[b]
        keys = o.key(rows[b, :n]).astype(np.int64)
        sel = idx[b]
        if len(set(sel.tolist())) != K or sel.min() < 0 or sel.max() >= n:
            fails.append("row %d: not K distinct indices in [0,n)" % b)
            continue
        if not np.all(np.diff(sel) > 0):
            fails.append("row %d: output not ascending" % b)
        t = keys[sel].min()
        if int(t) != int(kth[b]):
            fails.append("row %d: kth key mismatch" % b)
        gt = int((keys > t).sum())
        ge = int((keys >= t).sum())
        if not (gt < K <= ge) or gt != int(ngt[b]):
            fails.append("row %d: count invariant gt=%d ge=%d" % (b, gt, ge))
        mask = np.zeros(n, dtype=bool)
        mask[sel] = True
        if not np.all(mask[keys > t]):
            fails.append("row %d: a key above T* is missing" % b)
        eq = np.nonzero(keys == t)[0]
        eq_sel = eq[mask[eq]]
        eq_uns = eq[~mask[eq]]
        if len(eq_uns) and len(eq_sel) and eq_sel.max() > eq_uns.min():
            fails.append("row %d: tie not resolved by lower index" % b)
    return fails


def check_numpy(o, seed=5, K=K_DEFAULT):
    fails = []
    rng = np.random.default_rng(seed)
    n = 50000
    x = rng.permutation(n).astype(np.float32) * np.float32(0.5) - np.float32(100.0)   # distinct values
    got = o.topk(x, K)[0][0]
    exp = np.sort(np.argpartition(-x, K - 1)[:K])
    if not np.array_equal(got, exp):
        fails.append("distinct row: differs from numpy argpartition")
    y = rng.integers(-50, 50, n).astype(np.float32)                                   # ties
    got = o.topk(y, K)[0][0]
    if not np.array_equal(np.sort(y[got]), np.sort(y)[-K:]):
        fails.append("tied row: selected value multiset differs from numpy sort")
    return fails


# ---------------------------------------------------------------- the pins

def test_key_total_order(oracle_lib):
    assert check_key_order(oracle_lib) == []


def test_bruteforce_tiny_rows(oracle_lib):
    assert check_bruteforce(oracle_lib) == []


def test_special_rows(oracle_lib):
    assert check_special_rows(oracle_lib) == []
    assert check_special_rows(oracle_lib, K=7) == []


def test_count_closed_forms(oracle_lib):
    assert check_count_closed_forms(oracle_lib) == []


def test_invariants_full_size(oracle_lib):
    assert check_invariants(oracle_lib) == []


def test_numpy_cross_check(oracle_lib):
    assert check_numpy(oracle_lib) == []


def test_lemma1_containment(oracle_lib):
    """Lemma 1 (Sec. 4.1): if K <= f(T) then the exact answer lies in {x >= T}."""
    rng = np.random.default_rng(11)
    x = rng.gamma(2.0, 1.0, 40000).astype(np.float32)
    K = 2048
    sel = oracle_lib.topk(x, K)[0][0]
    keys = oracle_lib.key(x)
    for q in [0.5, 0.8, 0.9, 0.94, 0.948]:
        t = np.float32(np.quantile(x, q))
        f = oracle_lib.count_ge(x, int(oracle_lib.key(t)))
        assert f >= K
        assert np.all(keys[sel] >= oracle_lib.key(t))


MUTATIONS = [
    ("tie rule reversed", r"return a->idx < b->idx \? -1 : 1;", "return a->idx > b->idx ? -1 : 1;"),
    ("negative keys not flipped", r"return ~u;", "return u;"),
    ("off by one in the take", r"out\[i\] = p\[i\]\.idx;", "out[i] = p[i + 1].idx;"),
    ("padding value", r"\(i < n\) \? i : -1", "(i < n) ? i : 0"),
    ("strict count", r"if \(oracle_key\(row\[i\]\) >= tkey\)", "if (oracle_key(row[i]) > tkey)"),
    ("sign bit dropped for positives", r"return u \| 0x80000000u;", "return u;"),
]


@pytest.mark.parametrize("name,pattern,repl", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(tmp_path, name, pattern, repl):
    """A plausible mistake planted in a copy of the oracle must fail a pin."""
    src = open(oracle.SOURCE).read()
    mutated, nsub = re.subn(pattern, repl, src)
    assert nsub >= 1, "mutation pattern no longer matches the oracle source"
    path = tmp_path / "mutant.c"
    path.write_text(mutated)
    lib = oracle.compile_library(str(path), str(tmp_path / "libmutant.so"))
    m = oracle.Oracle(lib)
    fails = (check_key_order(m) + check_bruteforce(m, cases=120) + check_special_rows(m, K=7)
             + check_count_closed_forms(m) + check_invariants(m, B=3, ld=8000, K=300))
    assert fails, "mutation '%s' was not caught by any pin" % name
