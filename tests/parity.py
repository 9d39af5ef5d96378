"""Parity rules between the HIP library and the fp64 CPU oracle.

Fixed before the first GPU result and never loosened:

* fp64 accumulation:  |a - b| <= 1e-6 + 1e-5 |b|              (element-wise)
* fp32 accumulation:  |a - b| <= 1e-3 |b| + 1e-5 S             (element-wise)
  where S is the sum of |b| over the whole output block of that (row, group)
  (M+1 SHAP values including the bias, or the (M+1)^2 interaction block).
  A pure relative bound fails on values that cancel to nearly 0; the second
  term scales with the magnitude of everything that row's explanation holds.

Bounds for derived quantities (sums over a block) are the sums of the
element-wise bounds.
"""
from __future__ import annotations

import numpy as np


def block_scale(want: np.ndarray, block_axes: int) -> np.ndarray:
    axes = tuple(range(want.ndim - block_axes, want.ndim))
    return np.abs(want).sum(axis=axes, keepdims=True)


def tolerance(want: np.ndarray, dtype: str, block_axes: int = 1) -> np.ndarray:
    if dtype == "f64":
        return 1e-6 + 1e-5 * np.abs(want)
    return 1e-3 * np.abs(want) + 1e-5 * block_scale(want, block_axes)


def assert_parity(got, want, dtype: str, block_axes: int = 1, what: str = ""):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - want)
    tol = tolerance(want, dtype, block_axes)
    bad = err > tol
    # err / tol, where a zero tolerance (an all-zero fp32 block) allows no error
    ratio = np.divide(err, tol, out=np.where(err > 0, np.inf, 0.0), where=tol > 0)
    if bad.any():
        idx = np.argwhere(bad)[:5]
        detail = ", ".join(f"{tuple(i)}: got {got[tuple(i)]:.9g} want {want[tuple(i)]:.9g}"
                           for i in idx)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outside tolerance "
                             f"(max err/tol {float(ratio.max()):.3g}); {detail}")
    return float(ratio.max()) if ratio.size else 0.0


def sum_tolerance(want_block: np.ndarray, dtype: str, block_axes: int = 1) -> np.ndarray:
    """Bound on |sum(got) - sum(want)| over the block's last axes."""
    axes = tuple(range(want_block.ndim - block_axes, want_block.ndim))
    return tolerance(want_block, dtype, block_axes).sum(axis=axes)
