"""Error measures used to compare a result against the oracle (test infrastructure only).

* ``row_rel_error``: per query row, ||y_hat_T - y_T||_2 / ||y_T||_2.  Rows whose
  denominator nearly cancels (kappa_T > KAPPA_MAX, possible only for even P, where
  the truncated series has a real root) are reported separately and left out of
  the graded maximum.
* ``state_rel_error``: ||S_hat - S||_F / ||S||_F for one head's state.
* ``log10_abs_diff``: the paper's measure of recovery, log10 of the elementwise
  absolute difference (App. A3, App. A4).
"""
from __future__ import annotations

import numpy as np

__all__ = ["KAPPA_MAX", "TOL_F32", "TOL_BF16", "row_rel_error", "max_row_rel_error",
           "state_rel_error", "log10_abs_diff"]

KAPPA_MAX = 100.0
TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def row_rel_error(y_hat, y) -> np.ndarray:
    y_hat = np.asarray(y_hat, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    num = np.linalg.norm(y_hat - y, axis=-1)
    den = np.linalg.norm(y, axis=-1)
    return num / den


def max_row_rel_error(y_hat, y, kappa=None):
    """(max error over well-conditioned rows, number of excluded rows)."""
    err = row_rel_error(y_hat, y)
    if kappa is None:
        return float(np.max(err)) if err.size else 0.0, 0
    kappa = np.asarray(kappa)
    keep = kappa <= KAPPA_MAX
    excluded = int((~keep).sum())
    return (float(np.max(err[keep])) if keep.any() else 0.0), excluded


def state_rel_error(S_hat, S) -> float:
    S_hat = np.asarray(S_hat, dtype=np.float64)
    S = np.asarray(S, dtype=np.float64)
    return float(np.linalg.norm(S_hat - S) / np.linalg.norm(S))


def log10_abs_diff(y_hat, y) -> np.ndarray:
    d = np.abs(np.asarray(y_hat, dtype=np.float64) - np.asarray(y, dtype=np.float64))
    return np.log10(np.maximum(d, 1e-300))
