"""GPU parity: gvr_topk / radix_topk through the C ABI vs the CPU oracle.

Bar: bit-exact (same indices, same order -- ascending) on every row of every
step. Inputs are the seeded decode workloads; the previous-step guess handed
to the GPU is the oracle's answer of the previous step.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_cases import K_TOPK, assert_rows_equal, note, run_decode, workload

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2604_22312_amd as g
    g.lib()
    oracle.build(force=False)


def gvr(scores, row_len, prev, K, stats=None):
    import paper_2604_22312_amd as g
    if stats is None:
        return g.gvr_topk(scores, row_len, prev, K)
    return g.gvr_topk_ex(scores, row_len, prev, K, stats=stats)


def radix(scores, row_len, prev, K, stats=None):
    import paper_2604_22312_amd as g
    if stats is None:
        return g.radix_topk(scores, row_len, prev, K)
    return g.radix_topk_ex(scores, row_len, K, stats=stats)


FNS = [gvr, radix]

# (config, steps, queries, sub) -- parity sizes that still span several
# workgroups per row and ragged tails; full-size launches are further below.
CASES = [
    (0, 16, 1, None),
    (1, 6, 4, None),
    (2, 4, 4, None),
    (3, 3, 8, "a"),
    (3, 3, 8, "b"),
    (3, 3, 8, "c"),
    (3, 3, 8, "d"),
    (4, 3, 2, None),
]


@pytest.mark.parametrize("fn", FNS, ids=lambda f: f.__name__)
@pytest.mark.parametrize("case", CASES, ids=lambda c: "c%d%s" % (c[0], c[3] or ""))
def test_decode_parity(fn, case):
    cfg, nsteps, q, sub = case
    run_decode(fn, cfg, nsteps, q, sub=sub, dev=DEV)


@pytest.mark.parametrize("fn", FNS, ids=lambda f: f.__name__)
def test_full_size_config2(fn):
    """The benchmark's launch: 64 queries x 2 draft rows at ~102K (128 rows)."""
    run_decode(fn, 2, 3, 64, dev=DEV)


@pytest.mark.parametrize("fn", FNS, ids=lambda f: f.__name__)
def test_full_size_config1(fn):
    """32 queries at ~32.8K (the whole 32-row launch), four decode steps."""
    run_decode(fn, 1, 4, 32, dev=DEV)


@pytest.mark.parametrize("fn", FNS, ids=lambda f: f.__name__)
def test_full_size_config4(fn):
    """16 queries x 3 draft rows, rows of 65K..262K keys (48 rows)."""
    run_decode(fn, 4, 2, 16, dev=DEV)


def test_stats_invariants_config2():
    """Lemma 1 on the GPU's own threshold: K <= f(T) <= C and the candidate
    count equals the oracle's f(T); the K-th key and #{key > T*} match."""
    w, res = run_decode(gvr, 2, 3, 8, dev=DEV, stats_check=True)
    for i, st, kth, ngt in res:
        s_host = w.scores[i].numpy()
        rl = w.row_len[i].numpy()
        for r in range(w.rows):
            path = int(st["path"][r])
            assert path in (1, 2, 3, 5), path
            if i > 0:
                assert path in (2, 3), "step %d row %d: guess not used (path %d)" % (i, r, path)
            T = int(st["threshold"][r])
            f = oracle.count_ge(s_host[r], T, n=int(rl[r]))
            assert int(st["candidates"][r]) == f
            assert K_TOPK <= f <= 16384
            if i > 0 and path == 2:
                # one pass: the lists at T = T_spec (the guessed threshold)
                # held the answer
                assert int(st["passes"][r]) == 1
                assert T >= int(st["spec_threshold"][r])
                assert int(st["spec_count"][r]) == f
            assert int(st["kth_key"][r]) == int(kth[r])
            assert int(st["n_gt"][r]) == int(ngt[r])
            assert int(st["n"][r]) == int(rl[r])
            stamps = [int(st[k][r]) for k in ("t_start", "t_guess", "t_search", "t_collect", "t_refine")]
            assert stamps == sorted(stamps) and stamps[0] > 0, stamps


def test_guess_does_not_change_the_answer():
    """Metamorphic: exact, random, reversed, -1, duplicated, out-of-range and
    absent guesses all give the same output."""
    import paper_2604_22312_amd as g
    w = workload(2, 2, 4, None)
    K = w.K
    S = w.scores[1].to(DEV)
    RL = w.row_len[1].to(DEV)
    exp, _, _ = oracle.topk(w.scores[1].numpy(), K, row_len=w.row_len[1].numpy())
    prev_exact, _, _ = oracle.topk(w.scores[0].numpy(), K, row_len=w.row_len[0].numpy())
    n = int(w.row_len[1].min())
    rng = np.random.default_rng(3)
    variants = {
        "exact": prev_exact,
        "current": exp,
        "random": rng.integers(0, n, size=exp.shape).astype(np.int32),
        "reversed": prev_exact[:, ::-1].copy(),
        "minus1": np.full(exp.shape, -1, np.int32),
        "dup": np.repeat(prev_exact[:, :1], K, axis=1),
        "oob": np.full(exp.shape, 1 << 30, np.int32),
        "mixed_oob": np.where(rng.random(exp.shape) < 0.5, prev_exact, -7).astype(np.int32),
    }
    for name, pv in variants.items():
        note("metamorphic prev=%s" % name)
        out = g.gvr_topk(S, RL, torch.from_numpy(np.ascontiguousarray(pv)).to(DEV), K)
        assert_rows_equal(out.cpu().numpy(), exp, "prev=%s" % name)
    out = g.gvr_topk(S, RL, None, K)
    assert_rows_equal(out.cpu().numpy(), exp, "prev=None")


def test_options_force_other_paths():
    """capacity = K and 'ignore guess' force narrowing / tie paths; same answer."""
    import paper_2604_22312_amd as g
    w = workload(2, 2, 4, None)
    K = w.K
    S = w.scores[1].to(DEV)
    RL = w.row_len[1].to(DEV)
    exp, _, _ = oracle.topk(w.scores[1].numpy(), K, row_len=w.row_len[1].numpy())
    prev, _, _ = oracle.topk(w.scores[0].numpy(), K, row_len=w.row_len[0].numpy())
    pd = torch.from_numpy(prev).to(DEV)
    for opts in ({"capacity": K}, {"flags": 1}, {"capacity": K + 1}, {"capacity": 2500},
                  {"capacity": 16384}):
        note("options %s" % opts)
        st = g.new_stats(w.rows, DEV)
        out = g.gvr_topk_ex(S, RL, pd, K, options=opts, stats=st)
        assert_rows_equal(out.cpu().numpy(), exp, "options %s" % opts)
        paths = set(g.decode_stats(st)["path"].tolist())
        assert -1 not in paths
        if opts.get("flags") == 1:
            assert paths <= {5}
        out = g.radix_topk_ex(S, RL, K, options=opts)
        assert_rows_equal(out.cpu().numpy(), exp, "radix options %s" % opts)


def _special_rows(ld, K, rng):
    rows = []
    lens = []
    base = rng.standard_normal(ld).astype(np.float32)
    rows.append(np.full(ld, 1.5, np.float32)); lens.append(ld)                  # all equal
    x = base.copy(); x[::7] = np.inf; rows.append(x); lens.append(ld)           # many +inf
    x = base.copy(); x[::5] = -np.inf; rows.append(x); lens.append(ld)          # many -inf
    x = base.copy(); xb = x.view(np.uint32); xb[::11] = 0x7FC00000; rows.append(x); lens.append(ld)  # +NaN
    x = base.copy(); xb = x.view(np.uint32); xb[::3] = 0xFFC00000; rows.append(x); lens.append(ld)   # -NaN
    x = np.where(rng.random(ld) < 0.5, np.float32(0.0), np.float32(-0.0)).astype(np.float32)
    rows.append(x); lens.append(ld)                                              # +0 / -0 only
    x = rng.integers(0, 3, ld).astype(np.float32); rows.append(x); lens.append(ld)  # 3 levels
    x = np.arange(ld, dtype=np.float32); rows.append(x); lens.append(ld)        # increasing
    x = -np.arange(ld, dtype=np.float32); rows.append(x); lens.append(ld)       # decreasing
    for n in (0, 1, K - 1, K, K + 1, 6144, 6145, ld - 1):
        rows.append(base.copy()); lens.append(n)
    x = np.full(ld, 2.0, np.float32); x[: ld // 2] = 3.0; rows.append(x); lens.append(ld)  # 2 levels
    x = rng.standard_normal(ld).astype(np.float16).astype(np.float32); rows.append(x); lens.append(ld)
    return np.stack(rows), np.array(lens, np.int32)


@pytest.mark.parametrize("fn", FNS, ids=lambda f: f.__name__)
@pytest.mark.parametrize("ld,K", [(20001, 2048), (9999, 7), (70003, 1), (4097, 2048), (131071, 2000)])
def test_special_rows(fn, ld, K):
    rng = np.random.default_rng(ld + K)
    rows, lens = _special_rows(ld, K, rng)
    exp, _, _ = oracle.topk(rows, K, row_len=lens)
    S = torch.from_numpy(rows).to(DEV)
    RL = torch.from_numpy(lens).to(DEV)
    prev = torch.from_numpy(np.ascontiguousarray(exp)).to(DEV)   # also try a guess
    note("special rows %s ld=%d K=%d" % (fn.__name__, ld, K))
    out = fn(S, RL, None, K)
    assert_rows_equal(out.cpu().numpy(), exp, "special rows ld=%d K=%d" % (ld, K))
    out = fn(S, RL, prev, K)
    assert_rows_equal(out.cpu().numpy(), exp, "special rows with guess ld=%d K=%d" % (ld, K))


@pytest.mark.parametrize("fn", FNS, ids=lambda f: f.__name__)
def test_misaligned_row_starts(fn):
    """Rows whose first element is not 16-byte aligned (ld % 4 != 0) and a
    scores view offset by one float."""
    rng = np.random.default_rng(9)
    K = 2048
    for ld in (30001, 30002, 30003):
        big = rng.gamma(2.0, 1.0, size=(6 * ld + 1)).astype(np.float32)
        rows = big[1:].reshape(6, ld)
        lens = np.array([ld, ld - 1, ld - 2, ld - 3, 12345, 2049], np.int32)
        exp, _, _ = oracle.topk(rows, K, row_len=lens)
        t = torch.from_numpy(big).to(DEV)
        S = t[1:].view(6, ld)
        assert S.is_contiguous()
        note("misaligned %s ld=%d" % (fn.__name__, ld))
        out = fn(S, torch.from_numpy(lens).to(DEV), None, K)
        assert_rows_equal(out.cpu().numpy(), exp, "misaligned ld=%d" % ld)


@pytest.mark.parametrize("fn", FNS, ids=lambda f: f.__name__)
def test_poison_beyond_row_len(fn):
    """Values past row_len are NaN / +inf: they must never be used."""
    w = workload(3, 1, 8, "c")
    K = w.K
    s = w.scores[0].numpy().copy()
    rl = w.row_len[0].numpy()
    exp, _, _ = oracle.topk(s, K, row_len=rl)
    for poison in (np.float32(np.nan), np.float32(np.inf), np.float32(1e30)):
        p = s.copy()
        for r in range(p.shape[0]):
            p[r, rl[r]:] = poison
        note("poison %s %r" % (fn.__name__, float(poison)))
        out = fn(torch.from_numpy(p).to(DEV), torch.from_numpy(rl).to(DEV), None, K)
        assert_rows_equal(out.cpu().numpy(), exp, "poison %r" % float(poison))


def test_determinism():
    import paper_2604_22312_amd as g
    w = workload(2, 2, 4, None)
    K = w.K
    S = w.scores[1].to(DEV)
    RL = w.row_len[1].to(DEV)
    prev, _, _ = oracle.topk(w.scores[0].numpy(), K, row_len=w.row_len[0].numpy())
    pd = torch.from_numpy(prev).to(DEV)
    note("determinism x30")
    ref = g.gvr_topk(S, RL, pd, K).clone()
    st0 = g.new_stats(w.rows, DEV)
    g.gvr_topk_ex(S, RL, pd, K, stats=st0)
    for _ in range(30):
        assert torch.equal(g.gvr_topk(S, RL, pd, K), ref)
        assert torch.equal(g.radix_topk(S, RL, pd, K), ref)
    st1 = torch.zeros_like(st0)
    g.gvr_topk_ex(S, RL, pd, K, stats=st1)
    a, b = g.decode_stats(st0), g.decode_stats(st1)
    for key in ("path", "passes", "candidates", "threshold", "kth_key", "n_gt"):
        assert torch.equal(a[key], b[key]), key


def test_many_rows_several_launches():
    """More rows than one co-resident launch holds: the host splits the batch."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(21)
    B, ld, K = 700, 60000, 2048
    x = rng.standard_normal((B, ld)).astype(np.float32)
    lens = rng.integers(K + 1, ld + 1, size=B).astype(np.int32)
    exp, _, _ = oracle.topk(x, K, row_len=lens, threads=8)
    note("many rows B=%d ld=%d" % (B, ld))
    S = torch.from_numpy(x).to(DEV)
    RL = torch.from_numpy(lens).to(DEV)
    out = g.gvr_topk(S, RL, torch.from_numpy(exp).to(DEV), K)
    assert_rows_equal(out.cpu().numpy(), exp, "many rows gvr")
    out = g.radix_topk(S, RL, None, K)
    assert_rows_equal(out.cpu().numpy(), exp, "many rows radix")


@pytest.mark.parametrize("dist", ["gamma", "lognormal", "beta", "logistic", "weibull", "uniform_ties"])
def test_distribution_families(dist):
    """Score families named in the paper's distribution analysis (Sec. 6.4)."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(abs(hash(dist)) % 1000)
    B, ld, K = 16, 70690, 2048
    gen = {
        "gamma": lambda: rng.gamma(2.0, 1.0, (B, ld)),
        "lognormal": lambda: rng.lognormal(-1.0, 1.0, (B, ld)),
        "beta": lambda: rng.beta(2.0, 5.0, (B, ld)) - 3.0,
        "logistic": lambda: rng.logistic(-0.5, 1.0, (B, ld)),
        "weibull": lambda: rng.weibull(1.5, (B, ld)) - 2.2,
        "uniform_ties": lambda: rng.integers(0, 200, (B, ld)) * 0.25,
    }[dist]
    x = gen().astype(np.float32)
    exp, _, _ = oracle.topk(x, K)
    # guess: exact answer of a perturbed copy (temporal correlation)
    y = (x + 0.05 * rng.standard_normal(x.shape)).astype(np.float32)
    pv, _, _ = oracle.topk(y, K)
    note("distribution %s" % dist)
    S = torch.from_numpy(x).to(DEV)
    out = g.gvr_topk(S, None, torch.from_numpy(pv).to(DEV), K)
    assert_rows_equal(out.cpu().numpy(), exp, "gvr %s" % dist)
    out = g.radix_topk(S, None, None, K)
    assert_rows_equal(out.cpu().numpy(), exp, "radix %s" % dist)


def test_alternating_shapes():
    """Calls of different shapes back to back (the library keeps no state)."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(5)
    K = 2048
    shapes = [(128, 102463), (4, 102463), (700, 60000), (32, 32831), (9, 262144), (128, 102463)]
    for B, ld in shapes:
        x = rng.gamma(2.0, 1.0, size=(B, ld)).astype(np.float32)
        lens = rng.integers(K + 1, ld + 1, size=B).astype(np.int32)
        exp, _, _ = oracle.topk(x, K, row_len=lens, threads=8)
        note("shape B=%d ld=%d" % (B, ld))
        S = torch.from_numpy(x).to(DEV)
        RL = torch.from_numpy(lens).to(DEV)
        out = g.gvr_topk(S, RL, torch.from_numpy(exp).to(DEV), K)
        assert_rows_equal(out.cpu().numpy(), exp, "gvr B=%d ld=%d" % (B, ld))
        out = g.radix_topk(S, RL, None, K)
        assert_rows_equal(out.cpu().numpy(), exp, "radix B=%d ld=%d" % (B, ld))


def _gvr_parts(S, RL, prev, K, parts):
    import paper_2604_22312_amd as g
    return g.gvr_topk_ex(S, RL, prev, K, options={"parts": parts})


def test_parts_do_not_change_the_answer():
    """The row split (1..16 workgroups per row, merged by the last part to
    arrive) gives the oracle's answer for every split, with stats of one pass."""
    import paper_2604_22312_amd as g
    w = workload(2, 2, 4, None)
    K = w.K
    S = w.scores[1].to(DEV)
    RL = w.row_len[1].to(DEV)
    exp, _, _ = oracle.topk(w.scores[1].numpy(), K, row_len=w.row_len[1].numpy())
    prev, _, _ = oracle.topk(w.scores[0].numpy(), K, row_len=w.row_len[0].numpy())
    pd = torch.from_numpy(prev).to(DEV)
    for parts in (1, 2, 3, 5, 7, 16):
        note("parts=%d" % parts)
        st = g.new_stats(w.rows, DEV)
        out = g.gvr_topk_ex(S, RL, pd, K, options={"parts": parts}, stats=st)
        assert_rows_equal(out.cpu().numpy(), exp, "parts=%d" % parts)
        d = g.decode_stats(st)
        assert set(d["path"].tolist()) <= {2, 3}, d["path"].tolist()
        for r in range(w.rows):
            if int(d["path"][r]) == 2:
                assert int(d["passes"][r]) == 1
                cnt = oracle.count_ge(w.scores[1].numpy()[r], int(d["threshold"][r]), n=int(w.row_len[1][r]))
                assert int(d["candidates"][r]) == cnt


@pytest.mark.parametrize("case", [(2, 2, 4, None, 3), (3, 2, 8, "a", 8), (3, 2, 8, "b", 8), (4, 2, 2, None, 5)],
                         ids=["c2_p3", "c3a_p8", "c3b_p8", "c4_p5"])
def test_ordered_merge(case):
    """Option flag 128 (agent-scope release / acquire at the split-row
    handoff): the oracle's answer on split rows, including rows whose guess
    fails (random previous Top-K), and the same row stats as the default
    handoff."""
    import paper_2604_22312_amd as g
    cfg, steps, queries, sub, parts = case
    w = workload(cfg, steps, queries, sub)
    K = w.K
    S = w.scores[1].to(DEV)
    RL = w.row_len[1].to(DEV)
    exp, _, _ = oracle.topk(w.scores[1].numpy(), K, row_len=w.row_len[1].numpy())
    if w.random_prev is not None:
        pd = w.random_prev[1].to(DEV)
    else:
        prev, _, _ = oracle.topk(w.scores[0].numpy(), K, row_len=w.row_len[0].numpy())
        pd = torch.from_numpy(prev).to(DEV)
    note("ordered merge c%d%s parts=%d" % (cfg, sub or "", parts))
    st1, st2 = g.new_stats(w.rows, DEV), g.new_stats(w.rows, DEV)
    out = g.gvr_topk_ex(S, RL, pd, K, options={"parts": parts, "flags": 128}, stats=st1)
    assert_rows_equal(out.cpu().numpy(), exp, "ordered merge c%d%s parts=%d" % (cfg, sub or "", parts))
    g.gvr_topk_ex(S, RL, pd, K, options={"parts": parts}, stats=st2)
    torch.cuda.synchronize()
    a, b = g.decode_stats(st1), g.decode_stats(st2)
    for f in ("path", "passes", "threshold", "candidates", "spec_count"):
        assert torch.equal(a[f], b[f]), f


def test_parts_on_different_xcds():
    """Parts of a row placed on different XCDs (flag bit 1): the last part
    cannot use the lists through a shared L2 and reads the row itself; the
    answer is the same."""
    import paper_2604_22312_amd as g
    w = workload(2, 2, 4, None)
    K = w.K
    S = w.scores[1].to(DEV)
    RL = w.row_len[1].to(DEV)
    exp, _, _ = oracle.topk(w.scores[1].numpy(), K, row_len=w.row_len[1].numpy())
    prev, _, _ = oracle.topk(w.scores[0].numpy(), K, row_len=w.row_len[0].numpy())
    pd = torch.from_numpy(prev).to(DEV)
    for parts in (2, 3, 5):
        note("scatter parts=%d" % parts)
        st = g.new_stats(w.rows, DEV)
        out = g.gvr_topk_ex(S, RL, pd, K, options={"parts": parts, "flags": 2}, stats=st)
        assert_rows_equal(out.cpu().numpy(), exp, "scatter parts=%d" % parts)
        assert -1 not in set(g.decode_stats(st)["path"].tolist())


@pytest.mark.parametrize("parts", [1, 4])
@pytest.mark.parametrize("ld,K", [(20001, 2048), (131071, 2000), (9999, 7)])
def test_special_rows_with_guess_and_parts(ld, K, parts):
    rng = np.random.default_rng(ld + 7 * K)
    rows, lens = _special_rows(ld, K, rng)
    exp, _, _ = oracle.topk(rows, K, row_len=lens)
    S = torch.from_numpy(rows).to(DEV)
    RL = torch.from_numpy(lens).to(DEV)
    guesses = {"exact": exp,
               "random": rng.integers(0, ld, size=exp.shape).astype(np.int32)}
    for name, pv in guesses.items():
        note("special rows guess=%s ld=%d K=%d parts=%d" % (name, ld, K, parts))
        out = _gvr_parts(S, RL, torch.from_numpy(np.ascontiguousarray(pv)).to(DEV), K, parts)
        assert_rows_equal(out.cpu().numpy(), exp, "special rows guess=%s ld=%d K=%d parts=%d"
                          % (name, ld, K, parts))


def _crowded_rows(ld, K, rng):
    """Rows whose K-th key sits in a crowd of ~1.5 K candidates packed into a
    few ulps (far narrower than a first-level refine bin): all one value, two
    alternating values, consecutive floats, and consecutive floats with ties."""
    rows = []
    n_top = K - K // 4                          # the crowd holds the K-th largest
    crowd = K + K // 2
    one = np.float32(1.0).view(np.uint32)
    kinds = [np.full(crowd, one, np.uint32),
             one + (np.arange(crowd) % 2).astype(np.uint32),
             one + np.arange(crowd, dtype=np.uint32),
             one + (np.arange(crowd) // 3).astype(np.uint32)]
    for bits in kinds:
        x = rng.uniform(0.0, 0.5, ld).astype(np.float32)
        pos = rng.permutation(ld)
        x[pos[:n_top]] = rng.uniform(10.0, 20.0, n_top).astype(np.float32)
        x[pos[n_top:n_top + crowd]] = rng.permutation(bits).view(np.float32)
        rows.append(x)
    rows = np.stack(rows)
    return rows, np.full(rows.shape[0], ld, np.int32)


@pytest.mark.parametrize("parts", [1, 4])
@pytest.mark.parametrize("ld,K", [(100003, 2048), (60001, 300)])
def test_crowded_kth_bin(ld, K, parts):
    """The refine's K-th bin holds more candidates than one wave ranks:
    resolved from the bin's min / max (one key) or by narrowing between
    them; with the oracle's previous answer and a random guess, split or not,
    and the radix path on the same rows."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(ld + K + parts)
    rows, lens = _crowded_rows(ld, K, rng)
    exp, _, _ = oracle.topk(rows, K, row_len=lens)
    S = torch.from_numpy(rows).to(DEV)
    RL = torch.from_numpy(lens).to(DEV)
    guesses = {"exact": exp, "random": rng.integers(0, ld, size=exp.shape).astype(np.int32)}
    for name, pv in guesses.items():
        note("crowded rows guess=%s ld=%d K=%d parts=%d" % (name, ld, K, parts))
        out = _gvr_parts(S, RL, torch.from_numpy(np.ascontiguousarray(pv)).to(DEV), K, parts)
        assert_rows_equal(out.cpu().numpy(), exp, "crowded rows guess=%s ld=%d K=%d parts=%d"
                          % (name, ld, K, parts))
    out = g.radix_topk(S, RL, None, K)
    assert_rows_equal(out.cpu().numpy(), exp, "crowded rows radix ld=%d K=%d" % (ld, K))


@pytest.mark.parametrize("parts", [1, 3])
def test_misaligned_rows_with_guess(parts):
    rng = np.random.default_rng(19)
    K = 2048
    for ld in (30001, 30002, 30003):
        big = rng.gamma(2.0, 1.0, size=(6 * ld + 1)).astype(np.float32)
        rows = big[1:].reshape(6, ld)
        lens = np.array([ld, ld - 1, ld - 2, ld - 3, 12345, 2049], np.int32)
        exp, _, _ = oracle.topk(rows, K, row_len=lens)
        t = torch.from_numpy(big).to(DEV)
        S = t[1:].view(6, ld)
        pv = torch.from_numpy(np.ascontiguousarray(exp)).to(DEV)
        note("misaligned with guess ld=%d parts=%d" % (ld, parts))
        out = _gvr_parts(S, torch.from_numpy(lens).to(DEV), pv, K, parts)
        assert_rows_equal(out.cpu().numpy(), exp, "misaligned with guess ld=%d parts=%d" % (ld, parts))


def test_streamed_call_edges():
    """A call of at least 16 MiB of rows in one round of 16-wave workgroups
    (the speculative pass loads with the non-temporal hint): misaligned rows,
    ragged lengths, NaN beyond each row's length, and guesses that hold the
    answer, miss it (shifted indices) or are absent (-1)."""
    rng = np.random.default_rng(23)
    K, B, ld = 2048, 128, 40001
    big = rng.gamma(2.0, 1.0, size=(B * ld + 1)).astype(np.float32)
    rows = big[1:].reshape(B, ld)
    lens = rng.integers(2049, ld + 1, size=B).astype(np.int32)
    lens[:4] = (ld, ld - 1, 2049, 12345)
    exp, _, _ = oracle.topk(rows, K, row_len=lens)
    poisoned = big.copy()
    pr = poisoned[1:].reshape(B, ld)
    for r in range(B):
        pr[r, lens[r]:] = np.nan
    guess = exp.copy()
    guess[1::3] = (exp[1::3] + 7) % 2049   # a poor guess
    guess[2::3] = -1                      # no usable guess
    t = torch.from_numpy(poisoned).to(DEV)
    S = t[1:].view(B, ld)
    import paper_2604_22312_amd as g
    RL = torch.from_numpy(lens).to(DEV)
    GU = torch.from_numpy(np.ascontiguousarray(guess)).to(DEV)
    note("streamed call edges B=%d ld=%d" % (B, ld))
    out = g.gvr_topk(S, RL, GU, K)
    assert_rows_equal(out.cpu().numpy(), exp, "streamed call edges")
    # the same call split in two parts per row (the hinted kernel's merge)
    note("streamed call edges B=%d ld=%d parts=2" % (B, ld))
    out = g.gvr_topk_ex(S, RL, GU, K, options={"parts": 2})
    assert_rows_equal(out.cpu().numpy(), exp, "streamed call edges, two parts")


@pytest.mark.parametrize("parts", [1, 2])
def test_poison_beyond_row_len_with_guess(parts):
    w = workload(3, 1, 8, "c")
    K = w.K
    s = w.scores[0].numpy().copy()
    rl = w.row_len[0].numpy()
    exp, _, _ = oracle.topk(s, K, row_len=rl)
    pv = torch.from_numpy(np.ascontiguousarray(exp)).to(DEV)
    for poison in (np.float32(np.nan), np.float32(np.inf), np.float32(1e30)):
        p = s.copy()
        for r in range(p.shape[0]):
            p[r, rl[r]:] = poison
        note("poison with guess %r parts=%d" % (float(poison), parts))
        out = _gvr_parts(torch.from_numpy(p).to(DEV), torch.from_numpy(rl).to(DEV), pv, K, parts)
        assert_rows_equal(out.cpu().numpy(), exp, "poison with guess %r parts=%d" % (float(poison), parts))


@pytest.mark.parametrize("case", [(1, 4, 4, None), (2, 3, 4, None), (3, 2, 8, "a"), (3, 2, 8, "b"),
                                  (3, 2, 8, "c"), (4, 2, 2, None)], ids=lambda c: "c%d%s" % (c[0], c[3] or ""))
def test_secant_schedule_parity(case):
    """The paper's own schedule (flag bit 2: T0 = pmean, secant counting
    passes, a collect pass) gives the oracle's answer; when it accepts, the
    threshold satisfies Lemma 1."""
    import paper_2604_22312_amd as g

    def secant(scores, row_len, prev, K, stats=None):
        return g.gvr_topk_ex(scores, row_len, prev, K, options={"flags": 4}, stats=stats)
    secant.__name__ = "gvr_secant"
    cfg, steps, queries, sub = case
    w, res = run_decode(secant, cfg, steps, queries, sub, dev=DEV, stats_check=True)
    for i, st, kth, ngt in res:
        s_host = w.scores[i].numpy()
        rl = w.row_len[i].numpy()
        for r in range(w.rows):
            path = int(st["path"][r])
            assert path != -1
            if path == 6:
                T = int(st["threshold"][r])
                f = oracle.count_ge(s_host[r], T, n=int(rl[r]))
                assert int(st["candidates"][r]) == f
                assert K_TOPK <= f <= 16384
            if int(rl[r]) > K_TOPK:
                assert int(st["kth_key"][r]) == int(kth[r])


@pytest.mark.parametrize("flags", [8, 12], ids=["paper_refine", "paper_schedule_and_refine"])
@pytest.mark.parametrize("case", [(0, 4, 1, None), (1, 3, 4, None), (2, 3, 4, None), (3, 2, 8, "a"),
                                  (3, 2, 8, "b"), (3, 2, 8, "c"), (3, 2, 8, "d"), (4, 2, 2, None)],
                         ids=lambda c: "c%d%s" % (c[0], c[3] or ""))
def test_paper_refine_parity(case, flags):
    """The paper's own exact selection (flag bit 3: min / max, 2048-bin
    histogram with the wave-parallel bin search, snap iterations, partition),
    alone and after the paper's threshold search, gives the oracle's answer;
    the K-th key it reports is the oracle's."""
    import paper_2604_22312_amd as g

    def paper(scores, row_len, prev, K, stats=None):
        return g.gvr_topk_ex(scores, row_len, prev, K, options={"flags": flags}, stats=stats)
    paper.__name__ = "gvr_flags%d" % flags
    cfg, steps, queries, sub = case
    w, res = run_decode(paper, cfg, steps, queries, sub, dev=DEV, stats_check=True)
    for i, st, kth, ngt in res:
        rl = w.row_len[i].numpy()
        for r in range(w.rows):
            assert int(st["path"][r]) != -1
            if int(rl[r]) > K_TOPK and int(st["path"][r]) != 4:   # the ties path emits without a refine
                assert int(st["kth_key"][r]) == int(kth[r])
                assert int(st["n_gt"][r]) == int(ngt[r])
                assert 1 <= int(st["refine_iters"][r]) <= 64


@pytest.mark.parametrize("ld,K", [(20001, 2048), (9999, 7), (70003, 1), (131071, 2000)])
def test_paper_refine_special_rows(ld, K):
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(ld + 3 * K)
    rows, lens = _special_rows(ld, K, rng)
    exp, _, _ = oracle.topk(rows, K, row_len=lens)
    S = torch.from_numpy(rows).to(DEV)
    RL = torch.from_numpy(lens).to(DEV)
    prev = torch.from_numpy(np.ascontiguousarray(exp)).to(DEV)
    for flags in (8, 12):
        note("paper refine special rows ld=%d K=%d flags=%d" % (ld, K, flags))
        out = g.gvr_topk_ex(S, RL, None, K, options={"flags": flags})
        assert_rows_equal(out.cpu().numpy(), exp, "paper refine, no guess, ld=%d K=%d" % (ld, K))
        out = g.gvr_topk_ex(S, RL, prev, K, options={"flags": flags})
        assert_rows_equal(out.cpu().numpy(), exp, "paper refine with guess ld=%d K=%d" % (ld, K))
        out = g.radix_topk_ex(S, RL, K, options={"flags": flags})
        assert_rows_equal(out.cpu().numpy(), exp, "radix with the paper refine ld=%d K=%d" % (ld, K))


SHAPES = [("short", 16), ("long", 32), ("mid", 64)]


@pytest.mark.parametrize("shape", SHAPES, ids=[x[0] for x in SHAPES])
@pytest.mark.parametrize("case", [(0, 4, 1, None), (1, 3, 8, None), (2, 2, 4, None), (3, 2, 8, "a"),
                                  (3, 2, 8, "b"), (3, 2, 8, "c"), (3, 2, 8, "d")],
                         ids=lambda c: "c%d%s" % (c[0], c[3] or ""))
def test_forced_workgroup_shape_parity(case, shape):
    """Every workgroup shape (flag bit 4: 4 waves, 4096-entry lists; bit 5:
    16 waves; bit 6: 8 waves, 6144-entry lists) gives the oracle's answer on
    every decode workload, whatever the automatic choice would be."""
    import paper_2604_22312_amd as g
    flags = shape[1]

    def shaped(scores, row_len, prev, K, stats=None):
        return g.gvr_topk_ex(scores, row_len, prev, K, options={"flags": flags}, stats=stats)
    shaped.__name__ = "gvr_%s_shape" % shape[0]
    cfg, steps, queries, sub = case
    w, res = run_decode(shaped, cfg, steps, queries, sub, dev=DEV, stats_check=True)
    for i, st, kth, ngt in res:
        rl = w.row_len[i].numpy()
        for r in range(w.rows):
            assert int(st["path"][r]) != -1
            if int(rl[r]) > K_TOPK and int(st["path"][r]) != 4:
                assert int(st["kth_key"][r]) == int(kth[r])


@pytest.mark.parametrize("shape", [16, 64], ids=["short", "mid"])
@pytest.mark.parametrize("ld,K", [(20001, 2048), (9999, 7), (4097, 2048), (70003, 1)])
def test_short_shape_special_rows(ld, K, shape):
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(ld + 5 * K)
    rows, lens = _special_rows(ld, K, rng)
    exp, _, _ = oracle.topk(rows, K, row_len=lens)
    S = torch.from_numpy(rows).to(DEV)
    RL = torch.from_numpy(lens).to(DEV)
    prev = torch.from_numpy(np.ascontiguousarray(exp)).to(DEV)
    for flags in (shape, shape | 8, shape | 4):
        note("short shape special rows ld=%d K=%d flags=%d" % (ld, K, flags))
        out = g.gvr_topk_ex(S, RL, None, K, options={"flags": flags})
        assert_rows_equal(out.cpu().numpy(), exp, "short shape, no guess, ld=%d K=%d flags=%d" % (ld, K, flags))
        out = g.gvr_topk_ex(S, RL, prev, K, options={"flags": flags})
        assert_rows_equal(out.cpu().numpy(), exp, "short shape with guess ld=%d K=%d flags=%d" % (ld, K, flags))
        out = g.radix_topk_ex(S, RL, K, options={"flags": flags})
        assert_rows_equal(out.cpu().numpy(), exp, "radix, short shape ld=%d K=%d flags=%d" % (ld, K, flags))


@pytest.mark.parametrize("B,ld,guess", [(600, 12000, True), (600, 12000, False), (700, 3000, False),
                                         (500, 45000, True), (600, 45000, True)],
                         ids=["8w_guess", "8w_radix", "4w_radix", "16w_long", "8w_long_many"])
def test_many_rows_automatic_shape(B, ld, guess):
    """More rows than compute units: the automatic choice runs 8-wave
    workgroups (rows <= 40K with a guess, rows > 4K without), 4-wave ones
    (rows <= 4K without a guess) or 16-wave ones (rows > 40K, at most two
    per compute unit); ragged lengths; the answer is the oracle's."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(123 + ld)
    K = 2048
    x = rng.standard_normal((B, ld)).astype(np.float32)
    lens = rng.integers(0, ld + 1, B).astype(np.int32)
    lens[:4] = [ld, K, K + 1, 2 * K + 1]
    exp, _, _ = oracle.topk(x, K, row_len=lens)
    prev = None
    if guess:
        prev_rows = x + 0.1 * rng.standard_normal((B, ld)).astype(np.float32)
        pexp, _, _ = oracle.topk(prev_rows, K, row_len=lens)
        prev = torch.from_numpy(pexp).to(DEV)
    S = torch.from_numpy(x).to(DEV)
    RL = torch.from_numpy(lens).to(DEV)
    note("many rows B=%d ld=%d guess=%s" % (B, ld, guess))
    st = g.new_stats(B, DEV)
    out = g.gvr_topk_ex(S, RL, prev, K, stats=st)
    assert_rows_equal(out.cpu().numpy(), exp, "many rows B=%d ld=%d guess=%s" % (B, ld, guess))
    assert -1 not in set(g.decode_stats(st)["path"].tolist())
    out = g.radix_topk(S, RL, None, K)
    assert_rows_equal(out.cpu().numpy(), exp, "many rows, radix B=%d ld=%d" % (B, ld))


def test_graph_replays_match_the_oracle():
    """Calls captured into a HIP graph (split rows through the workspace, the
    8-wave shape, the guess-free kernel in the 4-wave shape) give the
    oracle's answer on every replay, with eager calls and synchronisations
    between replays."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(31)
    K = 2048
    cases = []
    # two long rows: split into parts (workspace); 800 short rows: 8-wave
    # shape; 3 rows <= 2K; 600 rows <= 2K: guess-free, 4-wave shape
    for B, ld in ((2, 131072), (800, 9000), (3, 4000), (600, 4000)):
        x = rng.standard_normal((B, ld)).astype(np.float32)
        prevx = x + 0.05 * rng.standard_normal((B, ld)).astype(np.float32)
        exp, _, _ = oracle.topk(x, K)
        pexp, _, _ = oracle.topk(prevx, K)
        cases.append((torch.from_numpy(x).to(DEV), torch.from_numpy(pexp).to(DEV), exp))
    outs = [torch.empty((c[0].shape[0], K), dtype=torch.int32, device=DEV) for c in cases]
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):   # eager calls first: the workspace exists before capture
        for (S, P, _), o in zip(cases, outs):
            g.gvr_topk(S, None, P, K, out_idx=o, stream=stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    note("graph capture of gvr_topk calls")
    with torch.cuda.graph(graph, stream=stream):
        for (S, P, _), o in zip(cases, outs):
            g.gvr_topk(S, None, P, K, out_idx=o, stream=stream)
    for rep in range(4):
        for o in outs:
            o.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for (_, _, exp), o in zip(cases, outs):
            assert_rows_equal(o.cpu().numpy(), exp, "graph replay %d" % rep)
        # eager work between replays on the same buffers
        S, P, exp = cases[0]
        o = g.gvr_topk(S, None, P, K)
        torch.cuda.synchronize()
        assert_rows_equal(o.cpu().numpy(), exp, "eager call between replays")


def test_graph_survives_workspace_growth():
    """A graph captured with a split call keeps its workspace after a later,
    larger eager call on the same stream has made the stream's workspace
    grow: every replay still equals the oracle (the outgrown workspace is
    kept, not freed)."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(37)
    K, ld = 2048, 70000
    x = rng.standard_normal((8, ld)).astype(np.float32)
    prevx = x + 0.05 * rng.standard_normal((8, ld)).astype(np.float32)
    exp, _, _ = oracle.topk(x, K)
    pexp, _, _ = oracle.topk(prevx, K)
    S, P = torch.from_numpy(x).to(DEV), torch.from_numpy(pexp).to(DEV)
    small = {"parts": 4}
    out2 = torch.empty((2, K), dtype=torch.int32, device=DEV)
    stream = torch.cuda.Stream()
    note("workspace growth after capture: eager 2 x 4 parts, capture, eager 8 x 4 parts, replays")
    with torch.cuda.stream(stream):   # 8 (row, part) slots: the stream's first workspace
        g.gvr_topk_ex(S[:2], None, P[:2], K, out_idx=out2, stream=stream, options=small)
    torch.cuda.synchronize()
    assert_rows_equal(out2.cpu().numpy(), exp[:2], "eager 2-row split call")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        g.gvr_topk_ex(S[:2], None, P[:2], K, out_idx=out2, stream=stream, options=small)
    for rep in range(3):
        with torch.cuda.stream(stream):   # 32 slots: the workspace grows (new buffer)
            o8 = g.gvr_topk_ex(S, None, P, K, stream=stream, options=small)
        torch.cuda.synchronize()
        assert_rows_equal(o8.cpu().numpy(), exp, "eager 8-row split call %d" % rep)
        out2.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert_rows_equal(out2.cpu().numpy(), exp[:2], "replay %d after the workspace grew" % rep)


def test_prepared_calls():
    """The binding's prepared calls (arguments checked and marshalled once)
    enqueue the same work as the plain calls: equal to the oracle on every
    call, also after the input buffers were rewritten in place; an option the
    library refuses raises on the call."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(43)
    K, B, ld = 2048, 4, 70001
    x = rng.standard_normal((B, ld)).astype(np.float32)
    lens = np.array([ld, ld - 5, 50000, 4096], np.int32)
    S = torch.from_numpy(x).to(DEV)
    RL = torch.from_numpy(lens).to(DEV)
    exp, _, _ = oracle.topk(x, K, row_len=lens)
    P = torch.from_numpy(np.ascontiguousarray(exp)).to(DEV)
    stream = torch.cuda.Stream()
    preps = {"gvr": g.prepare_gvr_topk(S, RL, P, K, stream=stream),
             "gvr_ex": g.prepare_gvr_topk(S, RL, P, K, stream=stream, options={"parts": 3}),
             "radix": g.prepare_radix_topk(S, RL, K, stream=stream),
             "radix_ex": g.prepare_radix_topk(S, RL, K, stream=stream, options={"parts": 2})}
    note("prepared calls")
    for rep in range(2):
        for name, pc in preps.items():
            pc.out_idx.fill_(-7)
            out = pc()
            torch.cuda.synchronize()
            assert out is pc.out_idx
            assert_rows_equal(out.cpu().numpy(), exp, "prepared %s call %d" % (name, rep))
        # new contents in the same buffers (the guess stays the old answer)
        x = rng.standard_normal((B, ld)).astype(np.float32)
        S.copy_(torch.from_numpy(x))
        exp, _, _ = oracle.topk(x, K, row_len=lens)
    bad = g.prepare_gvr_topk(S, RL, P, K, stream=stream, options={"flags": 256})
    with pytest.raises(g.GvrError):
        bad()


def test_concurrent_streams_and_threads():
    """Split-row calls from two host threads, each on its own stream and with
    no synchronisation between the streams: every (device, stream) pair has
    its own workspace, so the calls overlap on the device without sharing
    arrival words or part lists, and every result equals the oracle."""
    import threading
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(41)
    K, ld, B = 2048, 131072, 3
    cases = []
    for _ in range(2):
        x = rng.standard_normal((B, ld)).astype(np.float32)
        prevx = x + 0.05 * rng.standard_normal((B, ld)).astype(np.float32)
        exp, _, _ = oracle.topk(x, K)
        pexp, _, _ = oracle.topk(prevx, K)
        cases.append((torch.from_numpy(x).to(DEV), torch.from_numpy(pexp).to(DEV), exp))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    reps = 12
    outs = [[torch.empty((B, K), dtype=torch.int32, device=DEV) for _ in range(reps)] for _ in range(2)]
    errors = []

    def worker(i):
        try:
            S, P, _ = cases[i]
            with torch.cuda.stream(streams[i]):
                for r in range(reps):
                    opts = {"parts": 4 if r % 2 == 0 else 8}
                    if r % 3 == 2:   # the guess-free schedule splits too
                        g.radix_topk_ex(S, None, K, out_idx=outs[i][r], stream=streams[i], options=opts)
                    else:
                        g.gvr_topk_ex(S, None, P, K, out_idx=outs[i][r], stream=streams[i], options=opts)
        except Exception as e:   # reported by the main thread
            errors.append(e)

    note("two host threads, two streams, split calls")
    torch.cuda.synchronize()
    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for i in range(2):
        for r in range(reps):
            assert_rows_equal(outs[i][r].cpu().numpy(), cases[i][2], "thread %d call %d" % (i, r))


@pytest.mark.parametrize("opts", [{"flags": 16, "capacity": 2048}, {"flags": 16, "capacity": 2500},
                                  {"flags": 16 | 1}, {"flags": 16 | 8, "capacity": 3000},
                                  {"flags": 64, "capacity": 2048}, {"flags": 64, "capacity": 2500},
                                  {"flags": 64, "capacity": 6144}, {"flags": 64 | 1},
                                  {"flags": 64 | 8, "capacity": 3000}, {"flags": 64 | 4}],
                         ids=["short_cap_K", "short_cap_2500", "short_no_guess", "short_paper_refine_cap",
                              "mid_cap_K", "mid_cap_2500", "mid_cap_max", "mid_no_guess", "mid_paper_refine_cap",
                              "mid_secant"])
def test_short_shape_forced_paths(opts):
    """The 4-wave and 8-wave shapes through their narrowing, ties and
    guess-free paths (small capacities force them); same answer as the
    oracle."""
    import paper_2604_22312_amd as g
    w = workload(1, 3, 8, None)
    K = w.K
    S = w.scores[2].to(DEV)
    RL = w.row_len[2].to(DEV)
    exp, _, _ = oracle.topk(w.scores[2].numpy(), K, row_len=w.row_len[2].numpy())
    prev, _, _ = oracle.topk(w.scores[1].numpy(), K, row_len=w.row_len[1].numpy())
    note("short shape forced paths %s" % opts)
    st = g.new_stats(w.rows, DEV)
    out = g.gvr_topk_ex(S, RL, torch.from_numpy(prev).to(DEV), K, options=opts, stats=st)
    assert_rows_equal(out.cpu().numpy(), exp, "short shape %s" % opts)
    assert -1 not in set(g.decode_stats(st)["path"].tolist())
    out = g.radix_topk_ex(S, RL, K, options=opts)
    assert_rows_equal(out.cpu().numpy(), exp, "radix short shape %s" % opts)


@pytest.mark.parametrize("ld", [(1 << 29) - 4096, (1 << 29) - 4095, (1 << 30) + 4099],
                         ids=["guess_path_limit", "past_the_limit", "past_4GB"])
def test_rows_at_the_offset_limit(ld):
    """The longest stride the guess path takes (its byte offsets are 32-bit),
    one past it, and a row of more than 4 GB (past 32-bit byte offsets of
    any kind), which run the guess-free schedule: 4096 planted values
    (1, 2, ..., 4096 at random indices, the rest 0) in a 2 GB row, the guess
    the planted values of ranks 1025..3072. The answer is known by
    construction: the indices of the 2048 largest planted values."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(ld & 0xFFFF)
    K = 2048
    idx = rng.choice(ld, size=4096, replace=False)
    idx[-1] = ld - 1   # the largest value in the row's last element
    vals = np.arange(1, 4097, dtype=np.float32)
    exp = np.sort(idx[2048:]).astype(np.int32)[None, :]
    guess = np.sort(idx[1024:3072]).astype(np.int32)[None, :]
    note("row at the offset limit ld=%d" % ld)
    S = torch.zeros((1, ld), dtype=torch.float32, device=DEV)
    S[0, torch.from_numpy(idx).to(DEV)] = torch.from_numpy(vals).to(DEV)
    prev = torch.from_numpy(guess).to(DEV)
    st = g.new_stats(1, DEV)
    out = g.gvr_topk_ex(S, None, prev, K, stats=st)
    torch.cuda.synchronize()
    assert_rows_equal(out.cpu().numpy(), exp, "gvr_topk ld=%d" % ld)
    path = g.PATH_NAMES[int(g.decode_stats(st)["path"][0])]
    if ld <= (1 << 29) - 4096:
        assert path not in ("error", "no_guess"), path
    else:
        assert path == "no_guess", path
    del S
    torch.cuda.empty_cache()


CAPTURE_FIRST_TOPK = r"""
import sys, numpy as np, torch
sys.path.insert(0, sys.argv[1])
import oracle
import paper_2604_22312_amd as g
rng = np.random.default_rng(43)
B, ld, K = 600, 9000, 2048
x = rng.standard_normal((B, ld)).astype(np.float32)
exp, _, _ = oracle.topk(x, K)
pexp, _, _ = oracle.topk(x + 0.05 * rng.standard_normal((B, ld)).astype(np.float32), K)
dev = torch.device("cuda:0")
S, P = torch.from_numpy(x).to(dev), torch.from_numpy(pexp).to(dev)
out = torch.full((B, K), -7, dtype=torch.int32, device=dev)
stream = torch.cuda.Stream()
graph = torch.cuda.CUDAGraph()
with torch.cuda.graph(graph, stream=stream):   # the process's first Top-K call (no split: no workspace)
    g.gvr_topk(S, None, P, K, out_idx=out, stream=stream)
for rep in range(3):
    out.fill_(-7)
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), exp), rep
    o2 = g.gvr_topk(S, None, P, K)   # eager work between replays
    torch.cuda.synchronize()
    assert np.array_equal(o2.cpu().numpy(), exp)
print("ok")
"""


def test_topk_captured_as_first_call(tmp_path):
    """A fresh process whose first gvr_topk call (600 rows of 9000: the
    8-wave shape, no row split, so no workspace) is captured into a HIP
    graph: every replay and the eager calls between them equal the oracle."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    script = tmp_path / "capture_first_topk.py"
    script.write_text(CAPTURE_FIRST_TOPK)
    note("gvr_topk captured as the first call (subprocess)")
    r = subprocess.run([sys.executable, str(script), root], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr


def test_read_floor_reads_every_element_once():
    """gvr_read_floor (the plain read-rate helper the bench reports beside the
    Top-K): the xor of a row's 16 words equals the xor of the bit patterns of
    its elements [0, n_b), for misaligned row starts, ragged lengths, empty
    rows and batches that give a row 1 to 16 parts."""
    import paper_2604_22312_amd as g
    rng = np.random.default_rng(43)
    for B, ld in ((1, 131071), (3, 70003), (128, 102463), (600, 5001)):
        x = rng.standard_normal((B, ld)).astype(np.float32)
        lens = rng.integers(0, ld + 1, B).astype(np.int32)
        lens[0] = ld
        if B > 2:
            lens[1] = 0
            lens[2] = 1
        note("read floor B=%d ld=%d" % (B, ld))
        words = g.gvr_read_floor(torch.from_numpy(x).to(DEV), torch.from_numpy(lens).to(DEV)).cpu().numpy()
        got = np.bitwise_xor.reduce(words.view(np.uint32), axis=1)
        bits = x.view(np.uint32)
        exp = np.array([np.bitwise_xor.reduce(bits[b, :lens[b]]) if lens[b] > 0 else 0 for b in range(B)],
                       dtype=np.uint32)
        assert np.array_equal(got, exp), (B, ld)
