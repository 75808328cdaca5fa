"""GPU parity of the static RoPE/YaRN prior and of GVR guided by it.

* gvr_rope_g vs the oracle's angles and g(Delta): float64 on both sides, so
  they agree to rounding. Tolerance: each side rounds theta'_i (pow) within
  about one ulp, which moves Delta * theta'_i by up to Delta * 2^-52 * theta'_i
  <= n * 2^-52, and each cosine and the running sum add a few ulps of 64;
  |g_gpu - g_oracle| <= d * (n + 64) * 2^-50 bounds all of it.
* gvr_rope_prior vs the oracle's P_static: an index set, so bit-exact;
  entries whose oracle g lies within that tolerance of the K-th value (none
  at the lengths tested, but possible in principle) may be exchanged for
  other equally valid ones, and are checked for validity instead.
* gvr_topk on the synthetic rows of the paper's single-operator benchmark
  (Sec. 6.3.1) with P_static as the guess vs the oracle's exact Top-K of the
  scores: bit-exact, like every other gvr_topk result.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import rope_prior as RP
from tests.gpu_cases import K_TOPK, assert_rows_equal, note
from workloads import rope as WR

pytestmark = pytest.mark.gpu

DEV = "cuda"
PARAMS = [
    ("deepseek", dict()),
    ("d128_other", dict(d_rope=128, orig_ctx=8192, base=500000.0, scale=8.0)),
    ("plain_d2", dict(d_rope=2, scale=1.0)),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2604_22312_amd as g
    g.lib()
    oracle.build(force=False)


def oracle_theta(kw):
    p = dict(RP.DEFAULTS)
    p.update({("d" if k == "d_rope" else k): v for k, v in kw.items()})
    return RP.yarn_theta(**p), p["d"]


def g_tol(n, d):
    return d * (n + 64) * 2.0 ** -50


@pytest.mark.parametrize("n", [1, 1000, 131072, 262144])
@pytest.mark.parametrize("name,kw", PARAMS, ids=[p[0] for p in PARAMS])
def test_rope_g_matches_oracle(name, kw, n):
    import paper_2604_22312_amd as g
    th_o, d = oracle_theta(kw)
    note("gvr_rope_g %s n=%d" % (name, n))
    theta = torch.empty(d // 2, dtype=torch.float64, device=DEV)
    got = g.gvr_rope_g(n, kw, device=DEV, theta=theta)
    torch.cuda.synchronize()
    th = theta.cpu().numpy()
    assert np.allclose(th, th_o, rtol=1e-15, atol=0), np.max(np.abs(th / th_o - 1))
    ref = RP.g_delta(n, th_o)
    err = np.max(np.abs(got.cpu().numpy() - ref))
    assert err <= g_tol(n, d), (err, g_tol(n, d))


def check_prior(got, n, K, th_o, d):
    exp = RP.static_prior(n, K, th_o)
    if np.array_equal(got, exp):
        return
    # Only near-ties at the K-th value may differ; verify that case.
    g = RP.g_delta(n, th_o)
    tol = g_tol(n, d)
    kth = np.sort(g)[-K]
    sel = got[got >= 0]
    assert len(sel) == min(n, K) and np.all(np.diff(sel) > 0) and sel.min() >= 0 and sel.max() < n
    mask = np.zeros(n, bool)
    mask[sel] = True
    assert np.all(mask[g > kth + tol]), "a clearly larger g was left out"
    assert not np.any(mask[g < kth - tol]), "a clearly smaller g was taken"


@pytest.mark.parametrize("n,K", [(0, 2048), (1, 2048), (2047, 2048), (2048, 2048), (2049, 2048),
                                 (8192, 2048), (70690, 2048), (131072, 2048), (262144, 2048),
                                 (131072, 1), (100003, 777)])
def test_rope_prior_matches_oracle(n, K):
    import paper_2604_22312_amd as g
    th_o, d = oracle_theta({})
    note("gvr_rope_prior n=%d K=%d" % (n, K))
    got = g.gvr_rope_prior(n, K, device=DEV)
    torch.cuda.synchronize()
    check_prior(got.cpu().numpy(), n, K, th_o, d)


@pytest.mark.parametrize("name,kw", PARAMS[1:], ids=[p[0] for p in PARAMS[1:]])
def test_rope_prior_other_params(name, kw):
    import paper_2604_22312_amd as g
    th_o, d = oracle_theta(kw)
    n, K = 50000, 2048
    note("gvr_rope_prior %s n=%d" % (name, n))
    gbuf = torch.empty(n, dtype=torch.float64, device=DEV)
    got = g.gvr_rope_prior(n, K, kw, device=DEV, g=gbuf)
    torch.cuda.synchronize()
    check_prior(got.cpu().numpy(), n, K, th_o, d)
    # the g handed back is the one gvr_rope_g computes
    assert np.max(np.abs(gbuf.cpu().numpy() - RP.g_delta(n, th_o))) <= g_tol(n, d)


@pytest.mark.parametrize("n", list(WR.N_LIST) + [2049, 5000])
def test_gvr_with_static_prior_on_synthetic_rows(n):
    """Table 3's workload: one row per length, guess = P_static."""
    import paper_2604_22312_amd as g
    rows = 4
    s = WR.batch_scores(n, rows)
    exp, _, _ = oracle.topk(s, K_TOPK)
    note("gvr_topk synthetic rope rows n=%d" % n)
    prior = g.gvr_rope_prior(n, K_TOPK, device=DEV)
    prev = prior.view(1, K_TOPK).expand(rows, K_TOPK).contiguous()
    scores = torch.from_numpy(s).to(DEV)
    row_len = torch.full((rows,), n, dtype=torch.int32, device=DEV)
    stats = g.new_stats(rows, DEV)
    got = g.gvr_topk_ex(scores, row_len, prev, K_TOPK, stats=stats)
    got_r = g.radix_topk(scores, row_len, None, K_TOPK)
    torch.cuda.synchronize()
    assert_rows_equal(got.cpu().numpy(), exp, "gvr_topk with the static prior, n=%d" % n)
    assert_rows_equal(got_r.cpu().numpy(), exp, "radix_topk, n=%d" % n)
    st = g.decode_stats(stats)
    if n > 2 * K_TOPK:
        assert bool((st["guess_valid"] > 0).all()), "the static prior was not taken as the guess"
    else:   # rows of at most 2K elements list every element (the guess would cut few)
        assert st["path"].tolist() == [1] * rows
    note("  paths %s passes %s" % (st["path"].tolist(), st["passes"].tolist()))


def test_gvr_with_static_prior_ragged_rows():
    """A prior computed for the longest row guides shorter rows too (its
    entries beyond a row's length are ignored)."""
    import paper_2604_22312_amd as g
    nmax = 70690
    lens = [nmax, 65536, 40001, 2049, 2048, 100, 0, 9000]
    s = np.stack([WR.row_scores(nmax, r) for r in range(len(lens))])
    exp, _, _ = oracle.topk(s, K_TOPK, row_len=np.array(lens, np.int32))
    note("gvr_topk synthetic rope ragged rows")
    prior = g.gvr_rope_prior(nmax, K_TOPK, device=DEV)
    prev = prior.view(1, K_TOPK).expand(len(lens), K_TOPK).contiguous()
    got = g.gvr_topk(torch.from_numpy(s).to(DEV), torch.tensor(lens, dtype=torch.int32, device=DEV), prev,
                     K_TOPK)
    torch.cuda.synchronize()
    assert_rows_equal(got.cpu().numpy(), exp, "gvr_topk ragged rows with the static prior")


def test_gvr_repacks_bunched_candidates():
    """Candidates bunched in a few waves' ranges overflow a wave's list when a
    row runs in one workgroup: the synthetic RoPE row 0 at N = 131072 keeps
    most of its Top-K in the first tenth of the row, and a decode row with a
    recency bump keeps it in the last few thousand keys. f(T_spec) is still
    exact, so when it lies in [K, C] the kernel collects the lists again at
    packed offsets (two passes in all) instead of narrowing. (The recency rows
    take the narrowing path: their guess puts f(T_spec) just below K.) Every
    answer stays exact."""
    import paper_2604_22312_amd as g
    n = 131072
    rows_rope = WR.batch_scores(n, 2)
    rng = np.random.default_rng(77)
    base = rng.standard_normal((2, n)).astype(np.float32)
    base[:, -3500:] += 3.0                       # recent keys score higher
    prev_rows = base + 0.05 * rng.standard_normal((2, n)).astype(np.float32)
    s = np.concatenate([rows_rope, base]).astype(np.float32)
    exp, _, _ = oracle.topk(s, K_TOPK)
    prev_exp, _, _ = oracle.topk(prev_rows, K_TOPK)
    note("gvr_topk bunched candidates, one workgroup per row")
    prior = g.gvr_rope_prior(n, K_TOPK, device=DEV).cpu().numpy()
    prev = torch.from_numpy(np.concatenate([np.stack([prior, prior]), prev_exp]).astype(np.int32)).to(DEV)
    stats = g.new_stats(4, DEV)
    got = g.gvr_topk_ex(torch.from_numpy(s).to(DEV), torch.full((4,), n, dtype=torch.int32, device=DEV), prev,
                        K_TOPK, options={"parts": 1}, stats=stats)
    torch.cuda.synchronize()
    assert_rows_equal(got.cpu().numpy(), exp, "gvr_topk bunched candidates")
    st = g.decode_stats(stats)
    note("  paths %s passes %s" % (st["path"].tolist(), st["passes"].tolist()))
    assert int(st["path"][0]) == 2 and int(st["passes"][0]) == 2, "the RoPE row was not repacked"
    assert int(st["passes"].max()) <= 3


@pytest.mark.parametrize("rows,n", [(r, n) for r in (1, 2) for n in (32768, 65537, 131072, 262144)]
                         + [(16, 49153), (48, 65536), (64, 60001)])
def test_gvr_small_batch_split_rows(rows, n):
    """Calls of a few long rows split each row over several workgroups (one
    or two rows: 8 or 16 parts; up to a quarter as many rows as compute
    units from 48K elements: 4 to 8 parts); the answer is exact whatever the
    split."""
    import paper_2604_22312_amd as g
    s = WR.batch_scores(n, rows)
    exp, _, _ = oracle.topk(s, K_TOPK)
    note("gvr_topk small batch rows=%d n=%d" % (rows, n))
    prior = g.gvr_rope_prior(n, K_TOPK, device=DEV)
    prev = prior.view(1, K_TOPK).expand(rows, K_TOPK).contiguous()
    got = g.gvr_topk(torch.from_numpy(s).to(DEV), torch.full((rows,), n, dtype=torch.int32, device=DEV), prev,
                     K_TOPK)
    torch.cuda.synchronize()
    assert_rows_equal(got.cpu().numpy(), exp, "gvr_topk small batch rows=%d n=%d" % (rows, n))
