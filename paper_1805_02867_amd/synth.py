"""Seeded synthetic logits shaped like the paper's workloads.

The paper benchmarks batches of independent logit vectors (Section 5: 4,000
or 10 vectors, vector sizes from tens to millions).  This module only draws
inputs; it holds none of the softmax or top-k arithmetic, so both the HIP path
and the CPU oracle can consume what it produces.

Recipe (every draw is seeded; the same arguments give the same tensor on the
same device type):

* ``x = randn(N, V) * sigma`` in float32 with ``torch.Generator(device)``,
  drawn in row blocks of ``ROW_BLOCK`` rows so that huge batches need no
  full-size float32 temporary.  ``sigma`` is a standard deviation.
* ``shift_frac``: ``round(shift_frac * N)`` distinct rows, picked by a CPU
  generator seeded with ``seed + 1``, get ``+shift`` added in float32.
* ``tie_frac``: ``round(tie_frac * N)`` distinct rows, picked by a CPU
  generator seeded with ``seed + 2``; in each, ``tie_copies`` distinct
  positions other than the first arg-max receive the row maximum, so the
  maximum occurs ``tie_copies + 1`` times.
* ``dtype="bf16"``: the float32 draw rounded to bfloat16 (round to nearest
  even, torch's conversion).
"""
from __future__ import annotations

import torch

ROW_BLOCK = 4096


def logits(N: int, V: int, *, sigma: float = 1.0, seed: int = 0,
           dtype: str = "f32", device: str | torch.device = "cpu",
           shift_frac: float = 0.0, shift: float = 1000.0,
           tie_frac: float = 0.0, tie_copies: int = 3) -> torch.Tensor:
    device = torch.device(device)
    out_dtype = {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]
    x = torch.empty((N, V), dtype=out_dtype, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    # rows that get special treatment are drawn up front on the CPU
    n_shift = int(round(shift_frac * N))
    shift_rows = torch.randperm(N, generator=torch.Generator().manual_seed(seed + 1))[:n_shift]
    n_tie = int(round(tie_frac * N))
    tie_gen = torch.Generator().manual_seed(seed + 2)
    tie_rows = torch.randperm(N, generator=tie_gen)[:n_tie]
    tie_pos = [torch.randperm(max(V - 1, 0), generator=tie_gen)[:tie_copies]
               for _ in range(n_tie)]
    shift_set = set(shift_rows.tolist())
    tie_map = {int(r): p for r, p in zip(tie_rows.tolist(), tie_pos)}
    for r0 in range(0, N, ROW_BLOCK):
        r1 = min(N, r0 + ROW_BLOCK)
        blk = torch.randn((r1 - r0, V), generator=gen, device=device,
                          dtype=torch.float32)
        blk.mul_(sigma)
        for r in range(r0, r1):
            if r in shift_set:
                blk[r - r0].add_(shift)
            if r in tie_map and V > 1:
                row = blk[r - r0]
                amax = int(torch.argmax(row).item())
                pos = tie_map[r].clone()
                pos[pos >= amax] += 1  # skip the arg-max itself
                row.index_fill_(0, pos.to(device), row[amax].item())  # exact: f32 -> f64 -> f32
        x[r0:r1].copy_(blk)
    return x


def special_rows(N: int, *, seed: int = 0, shift_frac: float = 0.0,
                 tie_frac: float = 0.0) -> tuple[list[int], list[int]]:
    """The shifted and tied row indices that :func:`logits` uses."""
    n_shift = int(round(shift_frac * N))
    shift_rows = torch.randperm(N, generator=torch.Generator().manual_seed(seed + 1))[:n_shift]
    n_tie = int(round(tie_frac * N))
    tie_rows = torch.randperm(N, generator=torch.Generator().manual_seed(seed + 2))[:n_tie]
    return sorted(shift_rows.tolist()), sorted(tie_rows.tolist())


# The workloads of the benchmark and the parity tests, by what they are.
WORKLOADS = {
    "softmax_topk_16x1000_f32": dict(N=16, V=1000, sigma=1.0, dtype="f32", K=5),
    "softmax_4000x32000_f32_shift": dict(N=4000, V=32000, sigma=2.0, dtype="f32",
                                         shift_frac=0.01, K=5),
    "softmax_10x1e6_f32": dict(N=10, V=1_000_000, sigma=3.0, dtype="f32"),
    "topk_4000x50000_f32_ties": dict(N=4000, V=50000, sigma=2.0, dtype="f32",
                                     tie_frac=0.01, K=(5, 10)),
    "softmax_topk_32768x128256_bf16": dict(N=32768, V=128256, sigma=4.0,
                                           dtype="bf16", K=50),
}
