"""Comparison rules between the HIP path and the binary64 oracle.

binary32 outputs: |y - y64| <= 1e-5 * y64 elementwise; where y64 is below the
smallest normal binary32 (2^-126), |y - y64| <= 2^-126 instead (a subnormal
binary32 holds fewer than 24 significant bits, so a relative bound cannot
hold there; tests of the subnormal range check these outputs more tightly
themselves).  NaN where the oracle gives NaN.

bfloat16 outputs: the bit pattern is within 1 unit in the last place of the
oracle's value rounded to bfloat16 (to nearest even, from binary64),
subnormal values included.

top-k: indices bit-exact; values by the binary32 rule against y64 at the
oracle's indices.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle

FLT_MIN = 2.0 ** -126
RTOL = 1e-5


def to_host(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def host_dtype(t: torch.Tensor) -> str:
    return "bf16" if t.dtype == torch.bfloat16 else "f32"


def rel_err_f32(y: np.ndarray, y64: np.ndarray) -> np.ndarray:
    """Elementwise error in units of the tolerance: <= 1 passes."""
    y = y.astype(np.float64)
    err = np.abs(y - y64)
    small = y64 < FLT_MIN
    with np.errstate(divide="ignore", invalid="ignore"):
        scaled = np.where(small, err / FLT_MIN, err / (RTOL * y64))
    nan64 = np.isnan(y64)
    scaled = np.where(nan64, np.where(np.isnan(y), 0.0, np.inf), scaled)
    scaled = np.where(~nan64 & np.isnan(y), np.inf, scaled)
    return scaled


def assert_softmax_close(y: np.ndarray, y64: np.ndarray, what: str = ""):
    """y: GPU output (float32 array or uint16 bfloat16 patterns)."""
    if y.dtype == np.uint16:
        want = oracle.bf16_round(y64)
        nan64 = np.isnan(y64)
        gy = y.astype(np.int32)
        gw = want.astype(np.int32)
        is_nan_gpu = ((gy & 0x7F80) == 0x7F80) & ((gy & 0x007F) != 0)
        ulp = np.abs(gy - gw)
        bad = np.where(nan64, ~is_nan_gpu, ulp > 1)
        if bad.any():
            r, c = np.argwhere(bad)[0]
            raise AssertionError(
                f"{what}: {bad.sum()} bf16 outputs off by > 1 ulp; first at row {r} col {c}: "
                f"gpu 0x{y[r, c]:04x} want 0x{want[r, c]:04x} (y64={y64[r, c]!r})")
        return
    s = rel_err_f32(y, y64)
    worst = np.nanmax(s) if s.size else 0.0
    if not worst <= 1.0:
        r, c = np.unravel_index(np.nanargmax(s), s.shape)
        raise AssertionError(
            f"{what}: error {worst:.3g} x tolerance at row {r} col {c}: gpu {y[r, c]!r} "
            f"oracle {y64[r, c]!r}")


def assert_topk_equal(vals: np.ndarray, idx: np.ndarray, v64: np.ndarray, z64: np.ndarray,
                      what: str = ""):
    if not np.array_equal(idx, z64):
        bad = np.argwhere(idx != z64)
        r = bad[0][0]
        raise AssertionError(f"{what}: top-k indices differ in {len({b[0] for b in bad})} rows; "
                             f"row {r}: gpu {idx[r].tolist()} oracle {z64[r].tolist()}")
    s = rel_err_f32(vals, v64)
    if s.size and not np.nanmax(s) <= 1.0:
        r, c = np.unravel_index(np.nanargmax(s), s.shape)
        raise AssertionError(f"{what}: top-k value error {np.nanmax(s):.3g} x tolerance at "
                             f"row {r} slot {c}: gpu {vals[r, c]!r} oracle {v64[r, c]!r}")
