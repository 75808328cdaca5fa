"""GPU parity of the FP8 indexer (Sec. 2.1, Eq. indexer) and of the indexer
followed by gvr_topk, against the float64 oracle on the same FP8 bytes.

Scores: the GPU accumulates each dot product of D FP8 products (exact in
float32) in float32 on the matrix cores, scales, applies ReLU and sums the H
weighted heads in float32. Recursive summation bounds the error of a sum of
m terms by (m - 1) u times the sum of their magnitudes (u = 2^-24), so
|I_gpu - I| <= (D + H + 4) u * mag, mag = sum_j |w_j| sum_d |q_jd k'_d|
(the oracle's ``magnitude``), whatever order the hardware adds in.

Top-K, two checks. (1) Bit-exact: gvr_indexer_topk returns the float32
scores it selected from, and its out_idx must equal the oracle's Top-K over
exactly those scores (the Top-K parity bar). (2) Against the float64 scores:
the answer on the GPU's float32 scores and the oracle's on its exact scores
may differ only among keys within that tolerance of the K-th score: every
key clearly above it is selected, none clearly below it is, and the output
is K distinct indices in ascending order.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import indexer as IX
from tests.gpu_cases import K_TOPK, assert_rows_equal, note
from workloads import indexer as WI

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2604_22312_amd as g
    g.lib()


def tol_of(mag, H, D):
    return (D + H + 4) * 2.0 ** -24 * mag


def inputs(requests, group, ld, lengths, H, D, seed, steps=1):
    x = WI.generate(requests, group, ld, lengths, steps=steps, H=H, D=D, seed=seed, device="cpu")
    return x


def gpu_scores(x, t=0, sentinel=-7.0):
    import paper_2604_22312_amd as g
    B, ld = x.rows, x.ld
    sc = torch.full((B, ld), sentinel, dtype=torch.float32, device=DEV)
    g.gvr_indexer_scores(x.q[t].to(DEV), x.w.to(DEV), x.k.to(DEV), x.k_scale.to(DEV), x.row_len[t].to(DEV),
                         scores=sc)
    torch.cuda.synchronize()
    return sc.cpu().numpy().astype(np.float64)


def oracle_scores(x, t=0):
    args = (x.q[t].numpy(), x.w.numpy(), x.k.numpy(), x.k_scale.numpy())
    rl = x.row_len[t].numpy()
    return (IX.indexer_scores(*args, group=x.group, row_len=rl),
            IX.magnitude(*args, group=x.group, row_len=rl))


SHAPES = [(64, 128, 2), (64, 128, 1), (32, 64, 3), (128, 128, 4), (64, 64, 1), (32, 128, 2), (64, 128, 4),
          (32, 64, 4), (128, 64, 2)]


@pytest.mark.parametrize("H,D,group", SHAPES, ids=["h%d_d%d_g%d" % s for s in SHAPES])
def test_indexer_scores_parity(H, D, group):
    ld = 5000
    lengths = [ld, 1, 0, 31, 33, 1024, 1025, 2047][:3]
    x = inputs(3, group, ld, lengths[:3], H, D, seed=H + D + group)
    # ragged lengths inside each request's group too
    x.row_len[0, :] = torch.tensor(([ld, 4999, 1, 0, 33, 1025, 32, 2049, 1024, 4097, 3, 64] * 2)[:x.rows],
                                   dtype=torch.int32)
    note("indexer scores H=%d D=%d group=%d" % (H, D, group))
    got = gpu_scores(x)
    exp, mag = oracle_scores(x)
    rl = x.row_len[0].numpy()
    for b in range(x.rows):
        n = int(rl[b])
        err = np.abs(got[b, :n] - exp[b, :n])
        assert np.all(err <= tol_of(mag[b, :n], H, D)), (b, float(err.max()))
        assert np.all(got[b, n:] == -7.0), "row %d: scores past its length were written" % b


@pytest.mark.parametrize("requests,group,ld,H,D", [(1, 2, 40000, 64, 128), (3, 1, 70001, 32, 64),
                                                    (500, 1, 4200, 32, 64), (200, 3, 4500, 64, 64)],
                         ids=["one_request_long", "three_rows_long", "many_caches", "many_caches_g3"])
def test_indexer_grid_sizing(requests, group, ld, H, D):
    """The launch resizes the key chunks to the device (a few caches: fine
    chunks over many compute units; many caches: whole rounds of resident
    workgroups, the last chunk of a cache partial); every score matches the
    oracle and nothing past a row's length is written."""
    rng = np.random.default_rng(ld + requests)
    lengths = [int(v) for v in rng.integers(1, ld + 1, requests)]
    lengths[0] = ld - group + 1
    x = inputs(requests, group, ld, lengths, H, D, seed=requests + ld)
    note("indexer grid sizing requests=%d group=%d ld=%d H=%d D=%d" % (requests, group, ld, H, D))
    got = gpu_scores(x)
    exp, mag = oracle_scores(x)
    rl = x.row_len[0].numpy()
    for b in range(x.rows):
        n = int(rl[b])
        err = np.abs(got[b, :n] - exp[b, :n])
        assert np.all(err <= tol_of(mag[b, :n], H, D)), (b, float(err.max()))
        assert np.all(got[b, n:] == -7.0), "row %d: scores past its length were written" % b


def check_topk_exact(got, gpu_scores, rl, K, what):
    """The Top-K the call returned equals the oracle's Top-K over the very
    float32 scores the call wrote, on every row (bit-exact)."""
    exp, _, _ = oracle.topk(np.ascontiguousarray(gpu_scores, dtype=np.float32), K, row_len=np.asarray(rl))
    assert_rows_equal(got, exp, what)


def check_topk(got, exp_scores, mag, rl, K, H, D):
    for b in range(got.shape[0]):
        n = int(rl[b])
        sel = got[b]
        if n <= K:
            assert sel.tolist() == list(range(n)) + [-1] * (K - n)
            continue
        assert np.all(np.diff(sel) > 0) and sel[0] >= 0 and sel[-1] < n
        s = exp_scores[b, :n]
        tol = tol_of(mag[b, :n], H, D)
        kth = np.sort(s)[-K]
        mask = np.zeros(n, bool)
        mask[sel] = True
        assert np.all(mask[s - tol > kth + tol.max()]), "row %d: a clearly larger score was left out" % b
        assert not np.any(mask[s + tol < kth - tol.max()]), "row %d: a clearly smaller score was taken" % b


def check_fused_guess(st, sc, rl, prev, K, what):
    """gvr_indexer_topk's Top-K took each row's guess statistics from the
    indexer (which scored the sampled keys itself): the same T_spec, valid
    sample count, pmean, path and passes as gvr_topk_ex gathering the
    sample from the same scores."""
    import paper_2604_22312_amd as g
    st2 = g.new_stats(sc.shape[0], DEV)
    out2 = g.gvr_topk_ex(sc, rl, prev, K, stats=st2)
    torch.cuda.synchronize()
    a, b = g.decode_stats(st), g.decode_stats(st2)
    for f in ("path", "passes", "spec_threshold", "spec_count", "guess_valid", "threshold", "candidates"):
        assert torch.equal(a[f], b[f]), "%s: %s differs (fused guess)" % (what, f)
    assert torch.equal(a["pmean"].view(torch.int32), b["pmean"].view(torch.int32)), "%s: pmean differs" % what
    return out2


@pytest.mark.parametrize("group", [1, 2])
def test_indexer_topk_parity(group):
    """Two decode steps: the second is guided by the first step's Top-K."""
    import paper_2604_22312_amd as g
    H, D, ld = 64, 128, 40000
    x = inputs(4, group, ld, [39000, 2100, 20000, 2048], H, D, seed=17 + group, steps=2)
    ex0, _ = oracle_scores(x, 0)
    prev = np.full((x.rows, K_TOPK), -1, np.int32)
    for b in range(x.rows):
        n = int(x.row_len[0, b])
        prev[b, :min(n, K_TOPK)] = IX_argtopk(ex0[b, :n], K_TOPK)
    ex1, mag1 = oracle_scores(x, 1)
    note("indexer + topk group=%d" % group)
    st = g.new_stats(x.rows, DEV)
    out, sc = g.gvr_indexer_topk(x.q[1].to(DEV), x.w.to(DEV), x.k.to(DEV), x.k_scale.to(DEV), x.row_len[1].to(DEV),
                                 torch.from_numpy(prev).to(DEV), K_TOPK, stats=st)
    torch.cuda.synchronize()
    check_topk_exact(out.cpu().numpy(), sc.cpu().numpy(), x.row_len[1].numpy(), K_TOPK,
                     "indexer + topk group=%d" % group)
    check_topk(out.cpu().numpy(), ex1, mag1, x.row_len[1].numpy(), K_TOPK, H, D)
    out_u = check_fused_guess(st, sc, x.row_len[1].to(DEV), torch.from_numpy(prev).to(DEV), K_TOPK,
                              "indexer + topk group=%d" % group)
    assert torch.equal(out_u, out)
    # and without a guess (radix schedule inside gvr_topk)
    out2, _ = g.gvr_indexer_topk(x.q[1].to(DEV), x.w.to(DEV), x.k.to(DEV), x.k_scale.to(DEV), x.row_len[1].to(DEV),
                                 None, K_TOPK)
    torch.cuda.synchronize()
    assert np.array_equal(out2.cpu().numpy(), out.cpu().numpy())
    d = g.decode_stats(st)
    note("  paths %s passes %s" % (d["path"].tolist(), d["passes"].tolist()))


def test_indexer_topk_many_rows():
    """More rows than compute units (160 requests x 2 draft rows): the
    Top-K inside gvr_indexer_topk runs the 8-wave workgroup shape, guided by
    the first step's Top-K; same checks, and the same answer without the
    guess."""
    import paper_2604_22312_amd as g
    H, D, ld, requests = 32, 64, 6000, 160
    rng = np.random.default_rng(29)
    lengths = [int(v) for v in rng.integers(2100, ld - 1, requests)]
    x = inputs(requests, 2, ld, lengths, H, D, seed=29, steps=2)
    ex0, _ = oracle_scores(x, 0)
    prev = np.full((x.rows, K_TOPK), -1, np.int32)
    for b in range(x.rows):
        n = int(x.row_len[0, b])
        prev[b, :min(n, K_TOPK)] = IX_argtopk(ex0[b, :n], K_TOPK)
    ex1, mag1 = oracle_scores(x, 1)
    note("indexer + topk, %d rows" % x.rows)
    st = g.new_stats(x.rows, DEV)
    out, sc = g.gvr_indexer_topk(x.q[1].to(DEV), x.w.to(DEV), x.k.to(DEV), x.k_scale.to(DEV), x.row_len[1].to(DEV),
                                 torch.from_numpy(prev).to(DEV), K_TOPK, stats=st)
    torch.cuda.synchronize()
    check_topk_exact(out.cpu().numpy(), sc.cpu().numpy(), x.row_len[1].numpy(), K_TOPK,
                     "indexer + topk, %d rows" % x.rows)
    check_topk(out.cpu().numpy(), ex1, mag1, x.row_len[1].numpy(), K_TOPK, H, D)
    assert "error" not in {g.PATH_NAMES[int(v)] for v in g.decode_stats(st)["path"].tolist()}
    check_fused_guess(st, sc, x.row_len[1].to(DEV), torch.from_numpy(prev).to(DEV), K_TOPK,
                      "indexer + topk, %d rows" % x.rows)
    out2, _ = g.gvr_indexer_topk(x.q[1].to(DEV), x.w.to(DEV), x.k.to(DEV), x.k_scale.to(DEV), x.row_len[1].to(DEV),
                                 None, K_TOPK)
    torch.cuda.synchronize()
    assert np.array_equal(out2.cpu().numpy(), out.cpu().numpy())


@pytest.mark.parametrize("K,flags", [(2048, 4), (5, 0), (300, 0)], ids=["paper_schedule", "K5", "K300"])
def test_indexer_topk_guess_variants(K, flags):
    """gvr_indexer_topk with the paper's Phase 2 schedule (not fused: it
    reads every guessed score), with a K below the fused guess's words (not
    fused) and with K = 300 (fused, st = 2): exact Top-K of the call's own
    scores, and the fused rows' statistics equal gvr_topk_ex's."""
    import paper_2604_22312_amd as g
    H, D, ld = 64, 128, 30000
    x = inputs(3, 2, ld, [29000, 12000, 30000], H, D, seed=41 + K, steps=2)
    ex0, _ = oracle_scores(x, 0)
    prev = np.full((x.rows, K), -1, np.int32)
    for b in range(x.rows):
        n = int(x.row_len[0, b])
        prev[b, :min(n, K)] = IX_argtopk(ex0[b, :n], K)
    note("indexer + topk K=%d flags=%d" % (K, flags))
    st = g.new_stats(x.rows, DEV)
    pv = torch.from_numpy(prev).to(DEV)
    out, sc = g.gvr_indexer_topk(x.q[1].to(DEV), x.w.to(DEV), x.k.to(DEV), x.k_scale.to(DEV), x.row_len[1].to(DEV),
                                 pv, K, options={"flags": flags} if flags else None, stats=st)
    torch.cuda.synchronize()
    check_topk_exact(out.cpu().numpy(), sc.cpu().numpy(), x.row_len[1].numpy(), K, "indexer + topk K=%d" % K)
    if flags == 0:
        check_fused_guess(st, sc, x.row_len[1].to(DEV), pv, K, "indexer + topk K=%d" % K)
        # the guess and the output in one buffer (the decode loop's in-place form)
        inplace = pv.clone()
        g.gvr_indexer_topk(x.q[1].to(DEV), x.w.to(DEV), x.k.to(DEV), x.k_scale.to(DEV), x.row_len[1].to(DEV),
                           inplace, K, out_idx=inplace)
        torch.cuda.synchronize()
        assert torch.equal(inplace, out), "indexer + topk K=%d: prev_topk aliasing out_idx" % K


def IX_argtopk(s, K):
    """K largest (lower index first among equals), ascending: from the oracle's scores."""
    order = np.argsort(-s, kind="stable")[:K]
    return np.sort(order).astype(np.int32)


def test_indexer_full_size_sampled_rows():
    """The benchmark's shape (64 requests x 2 draft rows, ~100K keys, H = 64,
    D = 128) on the GPU, checked on four sampled rows."""
    import paper_2604_22312_amd as g
    H, D, ld = 64, 128, 102463
    x = WI.generate(64, 2, ld, [102400] * 64, steps=1, H=H, D=D, seed=3, device=DEV)
    note("indexer full size B=%d ld=%d" % (x.rows, ld))
    sc = g.gvr_indexer_scores(x.q[0], x.w, x.k, x.k_scale, x.row_len[0])
    torch.cuda.synchronize()
    for b in (0, 1, 77, 127):
        g_idx = b // 2
        args = (x.q[0][b:b + 1].cpu().numpy(), x.w[b:b + 1].cpu().numpy(), x.k[g_idx:g_idx + 1].cpu().numpy(),
                x.k_scale[g_idx:g_idx + 1].cpu().numpy())
        rl = x.row_len[0][b:b + 1].cpu().numpy()
        exp = IX.indexer_scores(*args, group=1, row_len=rl)[0]
        mag = IX.magnitude(*args, group=1, row_len=rl)[0]
        n = int(rl[0])
        got = sc[b, :n].cpu().numpy().astype(np.float64)
        assert np.all(np.abs(got - exp[:n]) <= tol_of(mag[:n], H, D)), b


CAPTURE_FIRST = r"""
import sys, numpy as np, torch
sys.path.insert(0, sys.argv[1])
import paper_2604_22312_amd as g
from oracle import indexer as IX
from workloads import indexer as WI
x = WI.generate(2, 2, 7000, [6900, 5000], steps=1, H=64, D=128, seed=41, device="cpu")
dev = torch.device("cuda:0")
q, w, k, ks, rl = (t.to(dev) for t in (x.q[0], x.w, x.k, x.k_scale, x.row_len[0]))
sc = torch.full((x.rows, x.ld), -7.0, dtype=torch.float32, device=dev)
stream = torch.cuda.Stream()
graph = torch.cuda.CUDAGraph()
with torch.cuda.graph(graph, stream=stream):   # the process's first indexer call
    g.gvr_indexer_scores(q, w, k, ks, rl, scores=sc, stream=stream)
args = (x.q[0].numpy(), x.w.numpy(), x.k.numpy(), x.k_scale.numpy())
exp = IX.indexer_scores(*args, group=2, row_len=x.row_len[0].numpy())
mag = IX.magnitude(*args, group=2, row_len=x.row_len[0].numpy())
for rep in range(3):
    sc.fill_(-7.0)
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    got = sc.cpu().numpy().astype(np.float64)
    for b in range(x.rows):
        n = int(x.row_len[0, b])
        assert np.all(np.abs(got[b, :n] - exp[b, :n]) <= (128 + 64 + 4) * 2.0 ** -24 * mag[b, :n]), (rep, b)
        assert np.all(got[b, n:] == -7.0)
    g.gvr_indexer_scores(q, w, k, ks, rl, scores=sc)   # eager work between replays
    torch.cuda.synchronize()
print("ok")
"""


def test_indexer_captured_as_first_call(tmp_path):
    """A fresh process whose first indexer call is captured into a HIP graph
    (the launch then sizes its grid without querying the device): every
    replay matches the oracle, with eager calls between replays."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    script = tmp_path / "capture_first.py"
    script.write_text(CAPTURE_FIRST)
    note("indexer captured as the first call (subprocess)")
    r = subprocess.run([sys.executable, str(script), root], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
