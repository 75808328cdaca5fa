"""Seeded synthetic inputs of the FP8 indexer (Sec. 2.1, Eq. indexer).

DeepSeek-V3.2's indexer shape: H = 64 heads of D = 128 dimensions, one key
vector per past token shared by the heads, FP8 E4M3 queries and keys, one
float32 dequantisation scale per key, float32 head weights. The model's
tensors are not available here, so these are drawn at random with that
shape: keys and queries N(0, 1) per dimension rounded to FP8 E4M3 (OCP),
key scales U(0.5, 1.5) / sqrt(D), head weights N(0, 1) / sqrt(H) (both
signs, as a learned projection gives). A request's draft rows (``group`` of
them, the speculative rows of one decode step) share its key cache and have
lengths L, L + 1, ...; their queries follow an AR(1) process over decode
steps (q_t = rho q_{t-1} + sqrt(1 - rho^2) eps_t, rho = 0.98), the temporal
correlation a previous step's Top-K exploits (Sec. 3.1).

Random numbers come from a ``torch.Generator`` seeded with ``seed`` on the
device the tensors are made on (``cpu`` in tests, the GPU for the benchmark's
large caches): keys first, then key scales, head weights, initial queries and
per step the query noise. Rounding to FP8 is torch's float8_e4m3fn
conversion. This module holds none of the indexer's arithmetic.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import torch

H_DEFAULT = 64
D_DEFAULT = 128


@dataclass
class IndexerInputs:
    q: torch.Tensor        # [steps][B][H][D] uint8 (FP8 E4M3 bytes)
    w: torch.Tensor        # [B][H] float32
    k: torch.Tensor        # [B / group][ld][D] uint8
    k_scale: torch.Tensor  # [B / group][ld] float32
    row_len: torch.Tensor  # [steps][B] int32
    group: int

    @property
    def rows(self) -> int:
        return self.w.shape[0]

    @property
    def ld(self) -> int:
        return self.k.shape[1]


def to_e4m3_bytes(x: torch.Tensor) -> torch.Tensor:
    return x.to(torch.float8_e4m3fn).view(torch.uint8)


def generate(requests: int, group: int, ld: int, lengths, steps: int = 1, H: int = H_DEFAULT,
             D: int = D_DEFAULT, seed: int = 0, rho: float = 0.98, device="cpu") -> IndexerInputs:
    """``lengths[r]``: length L_r of request r's first draft row at step 0
    (row j of the request has L_r + j keys at step 0, one more per step;
    the cache holds ld keys)."""
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(int(seed))
    B = requests * group
    k = to_e4m3_bytes(torch.randn((requests, ld, D), generator=gen, device=dev, dtype=torch.float16))
    k_scale = (0.5 + torch.rand((requests, ld), generator=gen, device=dev)) / math.sqrt(D)
    w = torch.randn((B, H), generator=gen, device=dev) / math.sqrt(H)
    qf = torch.randn((B, H, D), generator=gen, device=dev)
    qs = []
    noise = math.sqrt(1.0 - rho * rho)
    for _ in range(steps):
        qf = rho * qf + noise * torch.randn((B, H, D), generator=gen, device=dev)
        qs.append(to_e4m3_bytes(qf))
    q = torch.stack(qs)
    L = torch.as_tensor(list(lengths), dtype=torch.int64)
    assert L.numel() == requests
    rl = torch.empty((steps, B), dtype=torch.int32)
    for t in range(steps):
        for j in range(group):
            rl[t, j::group] = torch.clamp(L + j + t, max=ld).to(torch.int32)
    return IndexerInputs(q=q, w=w.float().contiguous(), k=k.contiguous(), k_scale=k_scale.float().contiguous(),
                         row_len=rl.to(dev), group=group)
