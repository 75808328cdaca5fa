"""Values the paper prints, kept as cited text fixtures under tests/golden/,
checked against every place that uses them (no GPU).

* rope_yarn_params.txt: the RoPE / YaRN parameters of Sec. 3.2-3.3 and the
  appendix's synthetic-data description, against the oracle's defaults, the
  C ABI's gvr_rope_params_default and the synthetic-row generator.
* rope_periods.txt: the shortest RoPE period the paper prints (Sec. 3.2),
  against the oracle's plain and YaRN angles (YaRN keeps the highest
  frequency and divides the lowest by the scaling factor, Sec. 3.2).
* table3_synthetic_latency_ns.txt: Table 3 (Sec. 6.3.1), against the copy
  bench.py reports as context.
"""
import inspect
import math
import os

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")


def read_table(name):
    rows = []
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#", 1)[0].strip()
        if line:
            rows.append(line.split())
    return rows


def rope_params():
    return {k: float(v) for k, v in read_table("rope_yarn_params.txt")}


def test_rope_parameters_everywhere_equal_the_paper():
    from oracle import rope_prior as RP
    from workloads import rope as WR
    import paper_2604_22312_amd as g
    p = rope_params()
    assert p == {"d_rope": 64, "base": 10000, "scale": 40, "orig_ctx": 4096, "beta_fast": 32, "beta_slow": 1}
    d = RP.DEFAULTS
    assert (d["d"], d["base"], d["scale"], d["orig_ctx"], d["beta_fast"], d["beta_slow"]) == \
        (p["d_rope"], p["base"], p["scale"], p["orig_ctx"], p["beta_fast"], p["beta_slow"])
    sig = inspect.signature(WR.angles).parameters
    assert (sig["d"].default, sig["base"].default, sig["scale"].default, sig["orig_ctx"].default,
            sig["beta_fast"].default, sig["beta_slow"].default) == \
        (p["d_rope"], p["base"], p["scale"], p["orig_ctx"], p["beta_fast"], p["beta_slow"])
    if not os.path.exists(g.library_path()):
        from paper_2604_22312_amd import build
        build.build()
    c = g.gvr_rope_params()
    assert (c.d_rope, c.base, c.scale, c.orig_ctx, c.beta_fast, c.beta_slow) == \
        (p["d_rope"], p["base"], p["scale"], p["orig_ctx"], p["beta_fast"], p["beta_slow"])


def test_shortest_period_is_the_printed_one():
    from oracle import rope_prior as RP
    p = rope_params()
    (name, value, decimals), = read_table("rope_periods.txt")
    assert name == "period_theta0"
    th = RP.rope_theta(int(p["d_rope"]), p["base"])
    assert round(2 * math.pi / th[0], int(decimals)) == float(value)
    ty = RP.yarn_theta(int(p["d_rope"]), p["base"], p["scale"], int(p["orig_ctx"]), p["beta_fast"], p["beta_slow"])
    # YaRN keeps the highest frequency and interpolates the lowest by the scaling factor
    assert round(2 * math.pi / ty[0], int(decimals)) == float(value)
    assert np.isclose(ty[-1], th[-1] / p["scale"], rtol=1e-12)


def test_table3_transcription():
    import bench
    rows = read_table("table3_synthetic_latency_ns.txt")
    table = {int(n): (int(a), int(b)) for n, a, b in rows}
    assert table == bench.PAPER_TABLE3_NS
