"""Small test helpers: BF16 bit views, plane allocation and tolerance checks.

Nothing here computes any part of the Lynx method; it only moves bytes.
"""
from __future__ import annotations

import numpy as np
import torch

HEAD_DIM = 128

# Attention tolerance for BF16 outputs against the fp64 oracle: elementwise
# |gpu - ref| <= ATOL + RTOL * |ref| (max abs 2e-2, relative 1e-2).
ATOL = 2e-2
RTOL = 1e-2

# Log-sum-exp (natural log) tolerance, an auxiliary output.  A caller uses the
# lse to merge this attention with another partial one; an error e in it
# scales that partial's weight by exp(e), so the outputs' relative tolerance
# of 1e-2 corresponds to |d lse| <= ln(1.01), about 1e-2.  The matrix-core
# decode carries the folded query 16 c q s as bf16 hi + lo (relative error at
# most 2^-18) against operands 128 + a <= 143, so a score term is off by at
# most 16 c |q s| 143 2^-18 (log2 units, c = log2(e) / sqrt(128)): 5.6e-4 at
# |q s| = 0.5, about 4.4e-3 in natural-log units over 128 dims of random sign.
# The inputs here have |q s| near 0.03 (0.3 on outlier channels), and the
# check below, tighter than the contract's 1e-2, holds with room.
LSE_ATOL = 2e-3
LSE_RTOL = 1e-4


def bf16_bits(x) -> np.ndarray:
    """uint16 bit patterns of a BF16 tensor (or of floats rounded to BF16)."""
    if not isinstance(x, torch.Tensor):
        x = torch.tensor(np.asarray(x, dtype=np.float32))
    if x.dtype != torch.bfloat16:
        x = x.to(torch.float32).to(torch.bfloat16)
    return x.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def assert_close(got, ref, atol=ATOL, rtol=RTOL, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - ref)
    bound = atol + rtol * np.abs(ref)
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(
            f"{what}: {bad.sum()} of {bad.size} elements out of tolerance; worst at {i}: "
            f"got {got[i]!r} ref {ref[i]!r} (max abs err {err.max():.3e})")
