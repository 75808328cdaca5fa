"""GPU parity of the caller-workspace entry points (gvr_topk_ex_ws,
radix_topk_ex_ws, sized by gvr_workspace_size): the split schedule of Sec. 4
with the parts' counts, thresholds, histograms and lists in a buffer the
caller owns. Every result is compared with the oracle's exact Top-K (bit-exact
indices) and with the library-owned-workspace call of the same shape.
"""
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import oracle
from tests.gpu_cases import K_TOPK, assert_rows_equal, note

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2604_22312_amd as g
    g.lib()
    oracle.build(force=False)


def _rows(seed, B, ld, row_len=None):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, ld)).astype(np.float32)
    prevx = x + 0.05 * rng.standard_normal((B, ld)).astype(np.float32)
    exp, _, _ = oracle.topk(x, K_TOPK, row_len=row_len)
    pexp, _, _ = oracle.topk(prevx, K_TOPK, row_len=row_len)
    return x, exp, pexp


# (rows, ld, radix): shapes that split their rows into 8, 16, 8 and 4..8 parts
SPLIT_SHAPES = [(1, 262144, False), (2, 70690, False), (8, 131079, False), (16, 65536, False),
                (8, 131079, True), (1, 262144, True)]


@pytest.mark.parametrize("B,ld,radix", SPLIT_SHAPES)
def test_caller_workspace_matches_oracle(B, ld, radix):
    """A workspace of gvr_workspace_size bytes, zero-filled once: two calls in
    a row on it (the second on fewer, ragged rows, so the buffer is reused
    without clearing) equal the oracle and the library-workspace call."""
    import paper_2604_22312_amd as g
    x, exp, pexp = _rows(100 + B, B, ld)
    S, P = torch.from_numpy(x).to(DEV), torch.from_numpy(pexp).to(DEV)
    nbytes = g.gvr_workspace_size(B, ld, K_TOPK, use_guess=not radix)
    assert nbytes > 0, "the shape was expected to split its rows"
    ws = g.new_workspace(B, ld, K_TOPK, use_guess=not radix)
    assert ws.numel() == nbytes
    note("caller workspace B=%d ld=%d radix=%d bytes=%d" % (B, ld, radix, nbytes))
    st_ws, st_ref = g.new_stats(B, DEV), g.new_stats(B, DEV)
    if radix:
        got = g.radix_topk_ex_ws(S, None, K_TOPK, ws, stats=st_ws)
        ref = g.radix_topk_ex(S, None, K_TOPK, stats=st_ref)
    else:
        got = g.gvr_topk_ex_ws(S, None, P, K_TOPK, ws, stats=st_ws)
        ref = g.gvr_topk_ex(S, None, P, K_TOPK, stats=st_ref)
    torch.cuda.synchronize()
    assert_rows_equal(got.cpu().numpy(), exp, "caller workspace, first call")
    assert np.array_equal(got.cpu().numpy(), ref.cpu().numpy())
    # the same schedule as the library-workspace call: every per-row statistic
    # but the clock stamps agrees
    a_st, r_st = g.decode_stats(st_ws), g.decode_stats(st_ref)
    for key in ("n", "path", "passes", "candidates", "threshold", "kth_key", "n_gt", "guess_valid",
                "spec_threshold", "spec_count"):
        assert torch.equal(a_st[key], r_st[key]), key
    # second call on the same buffer: fewer rows, ragged lengths
    B2 = max(1, B // 2)
    lens = np.array([ld - 1 - 977 * i for i in range(B2)], np.int32)
    exp2, _, _ = oracle.topk(x[:B2], K_TOPK, row_len=lens)
    RL = torch.from_numpy(lens).to(DEV)
    note("caller workspace second call B=%d ragged" % B2)
    if radix:
        got2 = g.radix_topk_ex_ws(S[:B2], RL, K_TOPK, ws)
    else:
        got2 = g.gvr_topk_ex_ws(S[:B2], RL, P[:B2], K_TOPK, ws)
    torch.cuda.synchronize()
    assert_rows_equal(got2.cpu().numpy(), exp2, "caller workspace, second call on fewer ragged rows")


def test_caller_workspace_smaller_than_needed():
    """A workspace smaller than asked for lowers an automatic split (down to
    one workgroup per row with no workspace at all), never the result; a
    forced split that does not fit is refused before anything is enqueued."""
    import paper_2604_22312_amd as g
    B, ld = 8, 131079
    x, exp, pexp = _rows(7, B, ld)
    S, P = torch.from_numpy(x).to(DEV), torch.from_numpy(pexp).to(DEV)
    full = g.gvr_workspace_size(B, ld, K_TOPK)
    for nbytes in (full // 2, full // 8, 1, 0):
        ws = torch.zeros(nbytes, dtype=torch.uint8, device=DEV) if nbytes else None
        note("caller workspace of %d of %d bytes" % (nbytes, full))
        got = g.gvr_topk_ex_ws(S, None, P, K_TOPK, ws)
        got_r = g.radix_topk_ex_ws(S, None, K_TOPK, ws)
        torch.cuda.synchronize()
        assert_rows_equal(got.cpu().numpy(), exp, "gvr, workspace %d bytes" % nbytes)
        assert_rows_equal(got_r.cpu().numpy(), exp, "radix, workspace %d bytes" % nbytes)
    # a forced split of 8 x 4 slots in a buffer sized for 8 x 2 is refused
    opt = {"parts": 4}
    small = torch.zeros(g.gvr_workspace_size(B, ld, K_TOPK, options={"parts": 2}), dtype=torch.uint8, device=DEV)
    out = torch.full((B, K_TOPK), -7, dtype=torch.int32, device=DEV)
    with pytest.raises(g.GvrError) as e:
        g.gvr_topk_ex_ws(S, None, P, K_TOPK, small, out_idx=out, options=opt)
    assert e.value.status == -3
    torch.cuda.synchronize()
    assert bool((out == -7).all()), "a refused call wrote its output"
    # the same forced split with room for it
    ws4 = g.new_workspace(B, ld, K_TOPK, options=opt)
    got = g.gvr_topk_ex_ws(S, None, P, K_TOPK, ws4, out_idx=out, options=opt)
    torch.cuda.synchronize()
    assert_rows_equal(got.cpu().numpy(), exp, "forced 4-part split in a caller workspace")


def test_caller_workspace_unsplit_shapes_need_none():
    """Shapes that run one workgroup per row report a size of 0 and run with
    no workspace."""
    import paper_2604_22312_amd as g
    for B, ld in ((600, 9000), (128, 102463), (3, 4000)):
        assert g.gvr_workspace_size(B, ld, K_TOPK) == 0, (B, ld)
    x, exp, pexp = _rows(11, 128, 20000)
    note("caller workspace: unsplit 128 x 20000, no workspace")
    got = g.gvr_topk_ex_ws(torch.from_numpy(x).to(DEV), None, torch.from_numpy(pexp).to(DEV), K_TOPK, None)
    torch.cuda.synchronize()
    assert_rows_equal(got.cpu().numpy(), exp, "unsplit call without a workspace")


def test_prepared_calls_with_a_caller_workspace():
    """Prepared calls (checked and marshalled once) on a caller workspace,
    repeated with the rows rewritten in place, and captured into a HIP graph
    replayed several times: every result equals the oracle."""
    import paper_2604_22312_amd as g
    B, ld = 2, 131072
    rng = np.random.default_rng(61)
    S = torch.empty((B, ld), dtype=torch.float32, device=DEV)
    P = torch.empty((B, K_TOPK), dtype=torch.int32, device=DEV)
    ws = g.new_workspace(B, ld, K_TOPK)
    wsr = g.new_workspace(B, ld, K_TOPK, use_guess=False)
    assert ws.numel() > 1 and wsr.numel() > 1
    stream = torch.cuda.Stream()
    pg = g.prepare_gvr_topk(S, None, P, K_TOPK, stream=stream, workspace=ws)
    pr = g.prepare_radix_topk(S, None, K_TOPK, stream=stream, workspace=wsr)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        pg()
        pr()
    for rep in range(3):
        x = rng.standard_normal((B, ld)).astype(np.float32)
        exp, _, _ = oracle.topk(x, K_TOPK)
        pexp, _, _ = oracle.topk(x + 0.05 * rng.standard_normal((B, ld)).astype(np.float32), K_TOPK)
        S.copy_(torch.from_numpy(x))
        P.copy_(torch.from_numpy(pexp))
        note("prepared caller-workspace calls, round %d" % rep)
        for pc in (pg, pr):
            pc.out_idx.fill_(-7)
            torch.cuda.synchronize()
            out = pc()
            torch.cuda.synchronize()
            assert_rows_equal(out.cpu().numpy(), exp, "prepared %s, round %d" % (pc._name, rep))
        pg.out_idx.fill_(-7)
        pr.out_idx.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert_rows_equal(pg.out_idx.cpu().numpy(), exp, "graph replay (gvr), round %d" % rep)
        assert_rows_equal(pr.out_idx.cpu().numpy(), exp, "graph replay (radix), round %d" % rep)


CAPTURE_FIRST_SPLIT = r"""
import sys, numpy as np, torch
sys.path.insert(0, sys.argv[1])
import oracle
import paper_2604_22312_amd as g
rng = np.random.default_rng(53)
B, ld, K = 4, 131079, 2048
dev = torch.device("cuda:0")
ws = g.new_workspace(B, ld, K)          # zero-filled before capture
assert ws.numel() > 1
S = torch.empty((B, ld), dtype=torch.float32, device=dev)
P = torch.empty((B, K), dtype=torch.int32, device=dev)
out = torch.full((B, K), -7, dtype=torch.int32, device=dev)
stream = torch.cuda.Stream()
graph = torch.cuda.CUDAGraph()
with torch.cuda.graph(graph, stream=stream):   # the process's first Top-K call: a split one
    g.gvr_topk_ex_ws(S, None, P, K, ws, out_idx=out, stream=stream)
for rep in range(4):
    x = rng.standard_normal((B, ld)).astype(np.float32)
    exp, _, _ = oracle.topk(x, K)
    pexp, _, _ = oracle.topk(x + 0.05 * rng.standard_normal((B, ld)).astype(np.float32), K)
    S.copy_(torch.from_numpy(x))
    P.copy_(torch.from_numpy(pexp))
    out.fill_(-7)
    torch.cuda.synchronize()
    print("[gpu-case] replay %d" % rep, flush=True)
    graph.replay()
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), exp), rep
    o2 = g.gvr_topk_ex_ws(S, None, P, K, ws)   # eager call on the same workspace between replays
    torch.cuda.synchronize()
    assert np.array_equal(o2.cpu().numpy(), exp), rep
print("ok")
"""


def test_caller_workspace_split_call_captured_first(tmp_path):
    """A fresh process whose first Top-K call is a split one (4 rows of 131079
    in 8 parts each), captured into a HIP graph through a caller workspace:
    no eager call has to come first. Every replay, on rows rewritten in place
    between replays, and the eager calls between them equal the oracle."""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    script = tmp_path / "capture_first_split.py"
    script.write_text(CAPTURE_FIRST_SPLIT)
    note("split gvr_topk_ex_ws captured as the first call (subprocess)")
    r = subprocess.run([sys.executable, str(script), root], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
