"""Error measures used to compare a result against the oracle (test infrastructure only).

* ``row_rel_error``: per query row, ||y_hat_T - y_T||_2 / ||y_T||_2, where, when
  the caller passes the rows' term scales rho_T (``taylor.term_scale``),
  ||y_T|| is floored at rho_T / CANCEL_FLOOR: a row whose numerator cancels by
  accident to below a tenth of the size that independent roundings of its
  terms add up to is judged against that size, as any finite-precision sum of
  those terms can be off by it.  Rows whose
  denominator nearly cancels (kappa_T > KAPPA_MAX, possible only for even P, where
  the truncated series has a real root) are reported separately and left out of
  the graded maximum; a comparison in which every row would be left out is an
  error, not a pass.
* ``state_rel_error``: ||S_hat - S||_F / ||S||_F for one head's state.
* ``state_elem_error``: max over entries of |S_hat - S| / S_abs, with S_abs the
  sum of the magnitudes of the terms of each entry (``state_abs_ref``).  Unlike
  the Frobenius measure, which the large degree-0 row dominates, it sees a
  single wrong entry of any row.
* ``state_tol``: the bound that ``state_elem_error`` must meet, derived from
  the arithmetic of the path that produced the state (see its docstring).
* ``log10_abs_diff``: the paper's measure of recovery, log10 of the elementwise
  absolute difference (App. A3, App. A4).
"""
from __future__ import annotations

import math

import numpy as np

__all__ = ["KAPPA_MAX", "CANCEL_FLOOR", "TOL_F32", "TOL_BF16", "TOL_F32_ARITH_BF16_OUT", "row_rel_error", "max_row_rel_error",
           "state_rel_error", "state_elem_error", "state_tol", "y_tol", "log10_abs_diff"]

KAPPA_MAX = 100.0
CANCEL_FLOOR = 10.0
TOL_F32 = 1e-4
TOL_BF16 = 2e-2
# float32 arithmetic whose output is stored in bfloat16: the storage rounding
# alone moves each element by up to 2^-9 of its size
TOL_F32_ARITH_BF16_OUT = 2.0 ** -8

_U32 = 2.0 ** -24  # unit roundoff of float32
_UBF16 = 2.0 ** -8  # unit roundoff of bfloat16 (8 significant bits)


def row_rel_error(y_hat, y, scale=None) -> np.ndarray:
    """||y_hat_T - y_T|| / max(||y_T||, scale_T / CANCEL_FLOOR) per row (plain
    ||y_T|| when scale is None)."""
    y_hat = np.asarray(y_hat, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    num = np.linalg.norm(y_hat - y, axis=-1)
    den = np.linalg.norm(y, axis=-1)
    if scale is not None:
        den = np.maximum(den, np.asarray(scale, dtype=np.float64) / CANCEL_FLOOR)
    return num / den


def max_row_rel_error(y_hat, y, kappa=None, scale=None):
    """(max error over well-conditioned rows, number of excluded rows).

    Raises ValueError when there is no row to grade (no rows at all, or every
    row excluded by kappa), so that such a comparison cannot pass vacuously."""
    err = row_rel_error(y_hat, y, scale)
    if err.size == 0:
        raise ValueError("no rows to compare")
    if kappa is None:
        return float(np.max(err)), 0
    kappa = np.asarray(kappa)
    keep = kappa <= KAPPA_MAX
    excluded = int((~keep).sum())
    if not keep.any():
        raise ValueError(f"all {err.size} rows excluded by kappa > {KAPPA_MAX}")
    return float(np.max(err[keep])), excluded


def state_rel_error(S_hat, S) -> float:
    S_hat = np.asarray(S_hat, dtype=np.float64)
    S = np.asarray(S, dtype=np.float64)
    return float(np.linalg.norm(S_hat - S) / np.linalg.norm(S))


def state_elem_error(S_hat, S, S_abs) -> float:
    """max_{f,j} |S_hat - S| / S_abs.  An entry with S_abs = 0 is a sum of zero
    terms: it must be exactly zero (error inf otherwise, 0 if it is)."""
    S_hat = np.asarray(S_hat, dtype=np.float64)
    S = np.asarray(S, dtype=np.float64)
    S_abs = np.asarray(S_abs, dtype=np.float64)
    diff = np.abs(S_hat - S)
    if not np.all(np.isfinite(S_hat)):
        return math.inf
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(S_abs > 0, diff / np.where(S_abs > 0, S_abs, 1.0), np.where(diff > 0, np.inf, 0.0))
    return float(r.max()) if r.size else 0.0


def state_tol(operands: str, n: int, chunk: int, P: int, steps: int = 0) -> float:
    """Bound on ``state_elem_error`` for a state summed over n tokens in chunks,
    then `steps` decode steps of one token each.

    Each term phi_f(k_t) [v_t, 1]_j enters as a product of operands rounded to
    the path's operand precision: bfloat16 operands (8 significant bits, unit
    roundoff u = 2^-8) carry two roundings, so a term is off by at most 2u
    (+ a second-order part) of its size; float32 operands carry at most ~P
    float32 roundings.  A chunk's sum of `chunk` terms and the n/chunk additions
    of chunk sums into the running state each add at most one float32 rounding
    of a partial sum, which is itself at most S_abs; so does each decode step.
    Split operands carry each float32 operand a as hi = bf16(a) and
    lo = bf16(a - hi), so |a - hi - lo| <= u^2 |a|, and form a product as
    hi*hi + hi*lo + lo*hi, leaving out |lo_a lo_b| <= u^2 |a b|: a term is off
    by at most 3u^2 of its size.  The bound allows twice the first-order term."""
    if n + steps <= 0:
        return 0.0
    accum = (chunk + math.ceil(n / chunk) + steps + 4 * P) * _U32
    if operands == "bf16":
        return 4.0 * _UBF16 + 2.0 * accum
    if operands == "split":
        return 6.0 * _UBF16 ** 2 + 2.0 * accum
    if operands == "f32":
        return 2.0 * accum
    raise ValueError(f"unknown operand precision {operands!r}")


def y_tol(operands: str, out_dtype: str) -> float:
    """Row tolerance for y: 2e-2 when the contractions take bfloat16 operands;
    with float32 (or split: float32 carried as bfloat16 pairs) arithmetic, 1e-4
    for a float32 output and 2^-8 for a bfloat16 one (whose storage rounding is
    up to 2^-9 per element)."""
    if operands == "bf16":
        return TOL_BF16
    if operands not in ("f32", "split"):
        raise ValueError(f"unknown operand precision {operands!r}")
    return TOL_F32 if out_dtype == "f32" else TOL_F32_ARITH_BF16_OUT


def log10_abs_diff(y_hat, y) -> np.ndarray:
    d = np.abs(np.asarray(y_hat, dtype=np.float64) - np.asarray(y, dtype=np.float64))
    return np.log10(np.maximum(d, 1e-300))
