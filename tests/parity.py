"""Shared tolerances for GPU-versus-oracle comparisons.

Float results: |gpu - oracle| <= RTOL * max|oracle row| per row (bf16 weights
and activations with float32 accumulation against a float64 oracle).
Integer decisions taken from floats (argmax, top-k) must agree wherever the
oracle's margin between the competing values exceeds the same tolerance.
"""
import numpy as np

RTOL = 2e-2


def row_close(gpu, ref, rtol=RTOL):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.abs(ref).max(axis=-1, keepdims=True)
    err = np.abs(gpu - ref)
    ok = err <= rtol * scale
    return bool(ok.all()), float((err / np.maximum(scale, 1e-30)).max())


def decided(row, rtol=RTOL):
    """True when the top-2 margin of an oracle logits row exceeds the tolerance."""
    s = np.sort(np.asarray(row, dtype=np.float64))[::-1]
    return (s[0] - s[1]) > rtol * np.abs(row).max()


def rank_decided(row, r, rtol=RTOL):
    """True when the r-th and (r+1)-th best values are separated (top-k boundary)."""
    s = np.sort(np.asarray(row, dtype=np.float64))[::-1]
    tol = rtol * np.abs(row).max()
    lo = (s[r - 1] - s[r]) > tol if r > 0 else True
    hi = (s[r] - s[r + 1]) > tol if r + 1 < len(s) else True
    return lo and hi
