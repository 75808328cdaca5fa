"""Pins for the FP8 indexer oracle (no GPU).

The oracle (``oracle/indexer.py``) computes the indexer scores of Sec. 2.1
(Eq. indexer) from FP8 E4M3 bytes in float64. These tests tie it to things
other than its own formulas:

* the decoder against torch's float8_e4m3fn for all 256 bytes, and against
  values decoded by hand (1.0, 448, -1, the smallest subnormal and normal,
  -0.0, NaN);
* a pure-Python loop version of the score on small shapes (math.fsum), with
  draft rows sharing a cache and ragged lengths;
* ReLU cases: a head whose logits are all negative adds nothing; a negative
  key scale flips a logit before the ReLU; one head with weight 1 and
  positive logits gives k_scale * numpy.dot;
* linearity in the head weights and invariance under a permutation of the
  heads; a row reads its own request's cache;
* the magnitude (the scale of the GPU tolerances) from both sides: a
  pure-Python loop on mixed signs, equality with the score when nothing can
  cancel, and |I| <= magnitude;
* planted mistakes in copies of the oracle (also in the magnitude).
"""
import importlib.util
import math
import re

import numpy as np
import pytest
import torch

from oracle import indexer as IX
from workloads import indexer as WI


def check_decoder_vs_torch(m):
    b = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(b).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = m.decode_e4m3(b)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])
    assert np.array_equal(np.signbit(got[ok]), np.signbit(ref[ok]))


def check_decoder_hand_values(m):
    cases = {0x38: 1.0, 0x7E: 448.0, 0xB8: -1.0, 0x01: 2.0 ** -9, 0x08: 2.0 ** -6, 0x07: 7 * 2.0 ** -9,
             0x40: 2.0, 0x3C: 1.5, 0x00: 0.0}
    for byte, v in cases.items():
        assert m.decode_e4m3(np.array([byte], np.uint8))[0] == v, hex(byte)
    z = m.decode_e4m3(np.array([0x80], np.uint8))[0]
    assert z == 0.0 and math.copysign(1.0, z) < 0
    assert np.isnan(m.decode_e4m3(np.array([0x7F, 0xFF], np.uint8))).all()


def _by_hand(q, w, k, ks, group, row_len):
    """Pure-Python score: every product and sum written out."""
    def dec(byte):
        s = -1.0 if byte & 0x80 else 1.0
        e, mm = (byte >> 3) & 15, byte & 7
        return s * (mm / 8.0 * 2.0 ** -6 if e == 0 else (1 + mm / 8.0) * 2.0 ** (e - 7))
    B, H, D = q.shape
    ld = k.shape[1]
    out = np.full((B, ld), np.nan)
    for b in range(B):
        g = b // group
        for s in range(min(int(row_len[b]), ld)):
            tot = []
            for j in range(H):
                logit = math.fsum(dec(int(q[b, j, d])) * (float(ks[g, s]) * dec(int(k[g, s, d]))) for d in range(D))
                tot.append(float(w[b, j]) * max(logit, 0.0))
            out[b, s] = math.fsum(tot)
    return out


def _small(seed, requests=2, group=2, ld=9, H=3, D=8):
    rng = np.random.default_rng(seed)
    B = requests * group
    q = WI.to_e4m3_bytes(torch.from_numpy(rng.standard_normal((B, H, D)))).numpy()
    k = WI.to_e4m3_bytes(torch.from_numpy(rng.standard_normal((requests, ld, D)))).numpy()
    ks = rng.uniform(-1.0, 1.5, (requests, ld))
    w = rng.standard_normal((B, H))
    rl = rng.integers(0, ld + 1, B)
    return q, w, k, ks, rl


def check_loops(m):
    for seed in range(6):
        q, w, k, ks, rl = _small(seed)
        got = m.indexer_scores(q, w, k, ks, group=2, row_len=rl)
        ref = _by_hand(q, w, k, ks, 2, rl)
        assert np.array_equal(np.isnan(got), np.isnan(ref))
        ok = ~np.isnan(ref)
        assert np.allclose(got[ok], ref[ok], rtol=1e-12, atol=1e-12), seed


def check_relu_and_scale_sign(m):
    q, w, k, ks, rl = _small(7, requests=1, group=1, ld=6, H=1, D=8)
    ks = np.abs(ks) + 0.1
    w = np.ones_like(w)
    # one head, weight 1, positive logits: k_scale * dot
    qv = IX.decode_e4m3(q[0, 0])
    kv = IX.decode_e4m3(k[0])
    pos = kv @ qv > 0
    got = m.indexer_scores(q, w, k, ks, group=1)[0]
    assert np.allclose(got[pos], (ks[0] * (kv @ qv))[pos], rtol=1e-13)
    assert np.all(got[~pos] == 0.0)
    # a negative scale flips the logit before the ReLU
    got_neg = m.indexer_scores(q, w, k, -ks, group=1)[0]
    assert np.all(got_neg[pos] == 0.0)
    assert np.allclose(got_neg[~pos], (-ks[0] * (kv @ qv))[~pos], rtol=1e-13)


def check_weights_and_heads(m):
    q, w, k, ks, rl = _small(11, requests=2, group=2, ld=7, H=5, D=16)
    a = m.indexer_scores(q, w, k, ks, group=2)
    assert np.allclose(m.indexer_scores(q, 2.0 * w, k, ks, group=2), 2.0 * a, rtol=1e-14)
    perm = np.random.default_rng(1).permutation(5)
    assert np.allclose(m.indexer_scores(q[:, perm], w[:, perm], k, ks, group=2), a, rtol=1e-12)
    # rows 2 and 3 read cache 1: swapping caches swaps row pairs
    b = m.indexer_scores(q[[2, 3, 0, 1]], w[[2, 3, 0, 1]], k[[1, 0]], ks[[1, 0]], group=2)
    assert np.allclose(b[[2, 3, 0, 1]], a, rtol=1e-14)


def _magnitude_by_hand(q, w, k, ks, group, row_len):
    """Pure-Python sum_j |w_j| sum_d |q_jd| |k_scale k_d|, every term written out."""
    def dec(byte):
        s = -1.0 if byte & 0x80 else 1.0
        e, mm = (byte >> 3) & 15, byte & 7
        return s * (mm / 8.0 * 2.0 ** -6 if e == 0 else (1 + mm / 8.0) * 2.0 ** (e - 7))
    B, H, D = q.shape
    ld = k.shape[1]
    out = np.full((B, ld), np.nan)
    for b in range(B):
        g = b // group
        for s in range(min(int(row_len[b]), ld)):
            out[b, s] = math.fsum(abs(float(w[b, j])) * math.fsum(abs(dec(int(q[b, j, d])))
                                                                 * abs(float(ks[g, s]) * dec(int(k[g, s, d])))
                                                                 for d in range(D))
                                  for j in range(H))
    return out


def check_magnitude_by_hand(m):
    """The error scale the GPU tolerances come from, against a pure-Python
    loop on mixed-sign inputs: a factor too many or too few (a dropped key
    scale, a missing absolute value) fails here."""
    for seed in range(4):
        q, w, k, ks, rl = _small(20 + seed, H=4, D=8)
        got = m.magnitude(q, w, k, ks, group=2, row_len=rl)
        ref = _magnitude_by_hand(q, w, k, ks, 2, rl)
        assert np.array_equal(np.isnan(got), np.isnan(ref))
        ok = ~np.isnan(ref)
        assert np.allclose(got[ok], ref[ok], rtol=1e-12, atol=0.0), seed


def check_magnitude_all_positive(m):
    """With every weight, query byte, key byte and key scale non-negative no
    term cancels and the ReLU passes everything: the magnitude equals the
    score itself (the upper side of |I| <= magnitude is reached)."""
    rng = np.random.default_rng(5)
    B, H, D, ld = 2, 4, 16, 11
    q = WI.to_e4m3_bytes(torch.from_numpy(np.abs(rng.standard_normal((B, H, D))))).numpy()
    k = WI.to_e4m3_bytes(torch.from_numpy(np.abs(rng.standard_normal((1, ld, D))))).numpy()
    assert not ((q & 0x80).any() or (k & 0x80).any())
    ks = rng.uniform(0.2, 1.5, (1, ld))
    w = rng.uniform(0.1, 2.0, (B, H))
    s = m.indexer_scores(q, w, k, ks, group=2)
    mag = m.magnitude(q, w, k, ks, group=2)
    assert np.all(s > 0)
    assert np.allclose(mag, s, rtol=1e-13, atol=0.0)


ALL_CHECKS = [check_decoder_vs_torch, check_decoder_hand_values, check_loops, check_relu_and_scale_sign,
              check_weights_and_heads, check_magnitude_by_hand, check_magnitude_all_positive]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=[c.__name__ for c in ALL_CHECKS])
def test_oracle_pin(check):
    check(IX)


def test_magnitude_bounds_scores():
    """Lower side of the two-sided pin: |I| <= magnitude on mixed signs
    (the upper side, equality, is check_magnitude_all_positive)."""
    q, w, k, ks, rl = _small(3, requests=2, group=2, ld=9, H=4, D=16)
    s = IX.indexer_scores(q, w, k, ks, group=2, row_len=rl)
    mag = IX.magnitude(q, w, k, ks, group=2, row_len=rl)
    ok = ~np.isnan(s)
    assert np.all(np.abs(s[ok]) <= mag[ok] * (1 + 1e-12))


def test_generator_shapes_and_seed():
    a = WI.generate(3, 2, 500, [400, 499, 100], steps=2, H=32, D=64, seed=5)
    b = WI.generate(3, 2, 500, [400, 499, 100], steps=2, H=32, D=64, seed=5)
    assert a.q.shape == (2, 6, 32, 64) and a.q.dtype == torch.uint8
    assert a.k.shape == (3, 500, 64) and a.k_scale.shape == (3, 500) and a.w.shape == (6, 32)
    assert torch.equal(a.q, b.q) and torch.equal(a.k, b.k)
    assert a.row_len.tolist() == [[400, 401, 499, 500, 100, 101], [401, 402, 500, 500, 101, 102]]
    # no NaN bytes (0x7F / 0xFF) from N(0, 1) values
    assert not bool(((a.k & 0x7F) == 0x7F).any()) and not bool(((a.q & 0x7F) == 0x7F).any())


MUTATIONS = [
    ("exponent bias 8", r"np\.exp2\(e - 7\.0\)", "np.exp2(e - 8.0)"),
    ("key scale dropped", r"decode_e4m3\(k\[g, :n\]\) \* k_scale\[g, :n, None\]", "decode_e4m3(k[g, :n])"),
    ("no ReLU", r"np\.maximum\(logits, 0\.0\)", "logits"),
    ("subnormal scale", r"\(m / 8\.0\) \* 2\.0 \*\* -6", "(m / 8.0) * 2.0 ** -7"),
    ("wrong cache", r"g = b // group", "g = b % max(k.shape[0], 1)"),
    ("sign ignored", r"sign = np\.where\(u >> 7, -1\.0, 1\.0\)", "sign = 1.0"),
    ("magnitude: key scale dropped",
     r"np\.abs\(decode_e4m3\(k\[g, :n\]\) \* np\.asarray\(k_scale, dtype=np\.float64\)\[g, :n, None\]\)",
     "np.abs(decode_e4m3(k[g, :n]))"),
    ("magnitude: |w| dropped", r"np\.abs\(np\.asarray\(w, dtype=np\.float64\)\[b\]\) @",
     "np.asarray(w, dtype=np.float64)[b] @"),
    ("magnitude: |q| dropped", r"Q = np\.abs\(decode_e4m3\(q\[b\]\)\)", "Q = decode_e4m3(q[b])"),
    ("magnitude: extra factor", r"@ \(Q @ Kd\.T\)", "@ (Q @ Kd.T) * 2.0"),
]


@pytest.mark.parametrize("name,pattern,repl", MUTATIONS, ids=[x[0] for x in MUTATIONS])
def test_planted_mistake_is_caught(tmp_path, name, pattern, repl):
    src = open(IX.__file__).read()
    mutated, nsub = re.subn(pattern, repl, src)
    assert nsub >= 1, "mutation pattern no longer matches the oracle source"
    path = tmp_path / "mutant_indexer.py"
    path.write_text(mutated)
    spec = importlib.util.spec_from_file_location("mutant_indexer", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    caught = 0
    for check in ALL_CHECKS:
        try:
            check(mod)
        except AssertionError:
            caught += 1
    assert caught, "mutation '%s' was not caught by any pin" % name
