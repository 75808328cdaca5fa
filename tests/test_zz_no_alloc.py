"""The allocation-free entry point gvr_topk_ex_noalloc, through the C ABI.

Its split-row workspace is a static device array of the library (no
allocation inside the call). Two calls in a row on split rows, the second
with a smaller input, must equal gvr_topk_ex (the entry point it varies) and
the oracle bit-exactly; a forced split beyond the array's slots is refused
before anything is enqueued; an unsplit call and a call at the slot limit
work too.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_cases import assert_rows_equal, note

pytestmark = pytest.mark.gpu

DEV = "cuda"
K = 2048


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2604_22312_amd as g
    g.lib()
    oracle.build(force=False)


def _rows(seed, B, ld, lens=None):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, ld)).astype(np.float32)
    prevx = x + 0.05 * rng.standard_normal((B, ld)).astype(np.float32)
    rl = np.full(B, ld, np.int32) if lens is None else np.asarray(lens, np.int32)
    exp, _, _ = oracle.topk(x, K, row_len=rl)
    pexp, _, _ = oracle.topk(prevx, K, row_len=rl)
    return (torch.from_numpy(x).to(DEV), torch.from_numpy(rl).to(DEV), torch.from_numpy(pexp).to(DEV), exp)


def _both(S, RL, P, opts, what):
    import paper_2604_22312_amd as g
    note("noalloc %s: B=%d ld=%d options=%s" % (what, S.shape[0], S.shape[1], opts))
    ref = g.gvr_topk_ex(S, RL, P, K, options=opts)
    st = g.new_stats(S.shape[0], DEV)
    got = g.gvr_topk_ex_noalloc(S, RL, P, K, options=opts, stats=st)
    torch.cuda.synchronize()
    return got.cpu().numpy(), ref.cpu().numpy(), g.decode_stats(st)


def test_noalloc_two_calls_second_smaller():
    """8 rows of 131K (automatic split into parts), then 2 rows of ~70K with
    ragged lengths: both equal gvr_topk_ex and the oracle."""
    big = _rows(71, 8, 131072)
    small = _rows(72, 2, 70001, lens=[70001, 52345])
    for (S, RL, P, exp), what in ((big, "first call"), (small, "second, smaller call")):
        got, ref, st = _both(S, RL, P, None, what)
        assert_rows_equal(ref, exp, "gvr_topk_ex %s" % what)
        assert_rows_equal(got, ref, "gvr_topk_ex_noalloc vs gvr_topk_ex, %s" % what)
        assert -1 not in set(st["path"].tolist())


def test_noalloc_forced_split_limits():
    """A forced split at the slot limit (16 rows x 16 parts = 256 slots)
    works; one slot more than the array holds is refused with
    GVR_ERR_WORKSPACE; an unsplit call needs no scratch."""
    import paper_2604_22312_amd as g
    S, RL, P, exp = _rows(73, 16, 40000)
    got, ref, _ = _both(S, RL, P, {"parts": 16}, "16 x 16 parts")
    assert_rows_equal(got, ref, "noalloc at the slot limit")
    assert_rows_equal(got, exp, "noalloc at the slot limit vs oracle")
    S2, RL2, P2, exp2 = _rows(74, 17, 40000)
    note("noalloc: 17 rows x 16 parts is refused")
    with pytest.raises(g.GvrError) as ei:
        g.gvr_topk_ex_noalloc(S2, RL2, P2, K, options={"parts": 16})
    assert ei.value.status == -3
    got, ref, _ = _both(S2, RL2, P2, {"parts": 1}, "17 rows unsplit")
    assert_rows_equal(got, exp2, "noalloc unsplit vs oracle")
    assert_rows_equal(got, ref, "noalloc unsplit vs gvr_topk_ex")
