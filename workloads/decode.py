"""Synthetic sparse-attention indexer score rows at decode time.

The paper's rows are DeepSeek-V3.2 indexer logits (Sec. 6.3.2), which are not
available here. These seeded rows stand in for them. They use the indexer's
functional form (Sec. 2.1, Eq. indexer): a weighted sum over heads of ReLU'd
query-key dot products,

    s_t[j] = sum_h w_h * ReLU(q_{t,h} . k_j / sqrt(d)),

with keys k_j ~ N(0, I_d), head weights w_h ~ U(0.5, 1.5), and per-head
queries following an AR(1) process q_t = rho q_{t-1} + sqrt(1 - rho^2) eps_t
(the temporal correlation of consecutive decode steps, Sec. 3.1). The score
is computed in float64 and rounded once to float32.

Decode structure: step t of query b has base length L_t = L0_b + t * next_n
(drafted tokens assumed accepted); draft row r < next_n has length L_t + r and
its own query noise; the AR state advances from the last draft row.

Every row buffer is filled to the full stride ``ld`` with scores of the keys
that lie beyond the row's length (values of the same distribution), so a
kernel that reads past ``row_len`` gets a wrong answer rather than a lucky
one. Sub-case (c) of config 3 writes -inf there instead.

Random numbers come from ``numpy.random.default_rng`` seeded per query
(``1000 * (config + 1) + 10000 * sub + b``), drawn in a fixed order: row
length, keys, head weights, initial query, then per step and draft row the
query noise. The matrix products run in torch float64 on the requested device;
both the GPU path and the oracle consume the same float32 buffer, so a
rounding difference between devices never matters for parity.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

K_TOPK = 2048

# Configs (decode workloads). rows per call = B * next_n.
CONFIGS = {
    0: dict(name="c0_n8k_b1", B=1, next_n=1, L0=8192, steps=16, H=4, d=64, rho=0.98),
    1: dict(name="c1_n32k_b32", B=32, next_n=1, L0=32768, steps=64, H=4, d=64, rho=0.98),
    2: dict(name="c2_n100k_b64_mtp2", B=64, next_n=2, L0=102400, steps=32, H=4, d=64, rho=0.98),
    3: dict(name="c3_n128k_b8_adversarial", B=8, next_n=1, L0=131072, steps=8, H=4, d=64, rho=0.98),
    4: dict(name="c4_n64k_256k_b16_mtp3", B=16, next_n=3, L0=(65536, 262144 - 384), steps=128,
            H=8, d=128, rho=0.95, ld=262144),
}
SUBCASES_3 = ("a", "b", "c", "d")


@dataclass
class Workload:
    config: int
    sub: str | None
    name: str
    B: int
    next_n: int
    ld: int
    K: int
    steps: list
    scores: torch.Tensor            # [T][rows][ld] float32
    row_len: torch.Tensor           # [T][rows] int32
    random_prev: torch.Tensor | None = None   # [T][rows][K] int32 (sub-case a only)
    meta: dict = field(default_factory=dict)

    @property
    def rows(self) -> int:
        return self.B * self.next_n


def spec(config: int) -> dict:
    c = dict(CONFIGS[config])
    L0 = c["L0"]
    if "ld" not in c:
        c["ld"] = L0 + (c["steps"] - 1) * c["next_n"] + c["next_n"] - 1
    return c


def _rng(config: int, sub: str | None, b: int) -> np.random.Generator:
    s = 0 if sub is None else 1 + SUBCASES_3.index(sub)
    return np.random.default_rng(1000 * (config + 1) + 10000 * s + b)


def generate(config: int, steps=None, queries=None, sub: str | None = None,
             device="cpu", K: int = K_TOPK, L0: int | None = None) -> Workload:
    """Build the score rows of ``config`` for the decode ``steps`` requested.

    ``steps``   -- iterable of step numbers (default: all of the config's steps);
                   the random state is advanced through the skipped steps so a
                   step's rows do not depend on which other steps were asked for.
    ``queries`` -- number of queries B to build (default: the config's B).
    ``sub``     -- config 3 sub-case: 'a' random guess, 'b' bf16-quantised,
                   'c' ragged lengths with -inf padding, 'd' lengths <= K.
    ``L0``      -- another first-step length for the config's rows (configs
                   with one L0 only; the stride follows as in ``spec``).
    """
    c = spec(config)
    if L0 is not None:
        if isinstance(c["L0"], tuple) or sub is not None:
            raise ValueError("L0 override needs a config with one L0 and no sub-case")
        c["L0"] = int(L0)
        c["ld"] = c["L0"] + (c["steps"] - 1) * c["next_n"] + c["next_n"] - 1
        c["name"] = "%s_L%d" % (c["name"].split("_")[0], c["L0"])
    if config == 3 and sub not in SUBCASES_3:
        raise ValueError("config 3 needs sub in %s" % (SUBCASES_3,))
    if config != 3 and sub is not None:
        raise ValueError("sub-cases exist for config 3 only")
    nsteps = c["steps"]
    steps = list(range(nsteps)) if steps is None else sorted(int(t) for t in steps)
    if any(t < 0 or t >= nsteps for t in steps):
        raise ValueError("step out of range")
    B = c["B"] if queries is None else int(queries)
    nn, H, d, rho, ld = c["next_n"], c["H"], c["d"], c["rho"], c["ld"]
    T = len(steps)
    rows = B * nn
    dev = torch.device(device)
    scores = torch.empty((T, rows, ld), dtype=torch.float32, device=dev)
    row_len = torch.empty((T, rows), dtype=torch.int32)
    rprev = torch.empty((T, rows, K), dtype=torch.int32) if sub == "a" else None
    tmax = steps[-1] if steps else -1
    want = {t: i for i, t in enumerate(steps)}
    noise_scale = math.sqrt(1.0 - rho * rho)
    inv_sqrt_d = 1.0 / math.sqrt(d)

    for b in range(B):
        rng = _rng(config, sub, b)
        if isinstance(c["L0"], tuple):
            L0 = int(rng.integers(c["L0"][0], c["L0"][1] + 1))
        elif sub == "c":
            L0 = int(rng.integers(4096, 131072 + 1))
        else:
            L0 = c["L0"]
        if sub == "d":
            pool = [0, 1, K - 1, K] + [int(v) for v in rng.integers(1, K + 1, size=4)]
            fixed_len = pool[b % len(pool)]
        keys = rng.standard_normal((ld, d))
        w = rng.uniform(0.5, 1.5, size=H)
        q = rng.standard_normal((H, d))
        # Queries of every (step, draft row) up to the last requested step.
        qs = np.empty((tmax + 1, nn, H, d))
        for t in range(tmax + 1):
            for r in range(nn):
                qs[t, r] = rho * q + noise_scale * rng.standard_normal((H, d))
            q = qs[t, nn - 1]
        keys_t = torch.from_numpy(keys).to(dev)
        w_t = torch.from_numpy(w).to(dev)
        # Scores for the requested steps, in blocks that keep the float64
        # intermediate [ld][block*nn*H] under ~512 MB.
        per = max(1, (512 << 20) // (ld * nn * H * 8))
        for i0 in range(0, T, per):
            blk = steps[i0:i0 + per]
            qb = torch.from_numpy(qs[blk].reshape(-1, d)).to(dev)           # [(t,r,h)][d]
            z = torch.relu((keys_t @ qb.T) * inv_sqrt_d)                     # [ld][(t,r,h)]
            s = (z.view(ld, len(blk) * nn, H) * w_t).sum(-1)               # [ld][(t,r)]
            s32 = s.T.contiguous().to(torch.float32).view(len(blk), nn, ld)
            if sub == "b":
                s32 = s32.to(torch.bfloat16).to(torch.float32)
            for j, t in enumerate(blk):
                i = want[t]
                scores[i, b * nn:(b + 1) * nn] = s32[j]
        for t in steps:
            i = want[t]
            for r in range(nn):
                n = fixed_len if sub == "d" else L0 + t * nn + r
                row_len[i, b * nn + r] = n
                if sub == "c" and n < ld:
                    scores[i, b * nn + r, n:] = float("-inf")
        if sub == "a":
            prng = np.random.default_rng(rng.integers(1 << 62))
            for t in range(tmax + 1):
                for r in range(nn):
                    n = L0 + t * nn + r
                    p = prng.choice(n, size=K, replace=False).astype(np.int32)
                    if t in want:
                        rprev[want[t], b * nn + r] = torch.from_numpy(p)
    name = c["name"] + ("" if sub is None else "_" + sub)
    return Workload(config=config, sub=sub, name=name, B=B, next_n=nn, ld=ld, K=K,
                    steps=steps, scores=scores, row_len=row_len.to(dev),
                    random_prev=None if rprev is None else rprev.to(dev),
                    meta=dict(H=H, d=d, rho=rho))
