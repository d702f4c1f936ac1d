"""Helpers shared by the GPU parity tests (host-side marshalling and the
comparisons against the oracle).

Tolerances follow the arithmetic of the path that produced a result, which
the library reports (``prefill_operands``): rows of y within 2e-2 when the
state contractions take bfloat16 operands, 1e-4 with float32 or split
(bfloat16 hi + lo pairs) arithmetic and a float32 output, 2^-8 with float32
arithmetic and a bfloat16 output; states element by element within the bound
of ``oracle.metrics.state_tol``.
"""
import numpy as np

import oracle
from oracle.metrics import (KAPPA_MAX, max_row_rel_error, state_elem_error, state_tol, y_tol)

__all__ = ["torch_dtype", "to_dev", "to_host", "operands", "check_rows", "check_state", "check_state_against",
           "check_prefill_head", "y_tol", "state_tol"]


def torch_dtype(dtype):
    import torch
    return torch.float32 if dtype == "f32" else torch.bfloat16


def to_dev(arr, dtype):
    """float32 array whose values are exact in `dtype` -> device tensor of that dtype."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda().to(torch_dtype(dtype))


def to_host(t):
    return t.float().cpu().numpy().astype(np.float64)


def operands(sata, dtype, B, H, n, dk, dv, P, chunk):
    """Operand precision ('bf16', 'split' or 'f32') of the prefill the library runs for these arguments."""
    return sata.prefill_operands(torch_dtype(dtype), B, H, n, dk, dv, P, chunk)


def check_rows(y_gpu, y_ref, kappa, tol, P, label="", scale=None):
    """Rows of one head against the oracle.  Rows whose denominator cancels
    (kappa > KAPPA_MAX, possible for even P only) are reported and left out;
    every other row must be finite and within `tol`.  For odd P no row may be
    left out, and at least one row is always graded.  With the rows' term
    scales (oracle.term_scale), a row whose numerator has cancelled by accident
    is judged against a tenth of that scale.  Returns (error, excluded)."""
    y_gpu = np.asarray(y_gpu)
    kappa = np.asarray(kappa)
    assert np.all(np.isfinite(y_gpu[kappa <= KAPPA_MAX])), f"{label}: non-finite well-conditioned row"
    err, excluded = max_row_rel_error(y_gpu, y_ref, kappa, scale)
    if P % 2 == 1:
        assert excluded == 0, f"{label}: {excluded} rows excluded at odd P={P}"
    assert err <= tol, f"{label}: max row rel error {err:.3e} > {tol:.1e} (excluded {excluded})"
    return err, excluded


def check_state_against(S_gpu, S_ref, S_abs, tol, label=""):
    """Element-wise |S_gpu - S_ref| <= tol * S_abs.  Returns the error."""
    e = state_elem_error(S_gpu, S_ref, S_abs)
    assert e <= tol, f"{label}: state element error {e:.3e} > {tol:.2e}"
    return e


def check_state(S_gpu, k, v, P, ops, n, chunk, label="", steps=0):
    """A state summed from tokens k, v (n prefill tokens in chunks, then
    `steps` decode steps) against the oracle, element by element."""
    return check_state_against(S_gpu, oracle.state_ref(k, v, P), oracle.state_abs_ref(k, v, P),
                               state_tol(ops, n, chunk, P, steps), label)


def check_prefill_head(y_gpu, S_gpu, q, k, v, P, ops, out_dtype, chunk, label=""):
    """Compare one head's GPU prefill output (and state) with the oracle.

    Returns (max row error, excluded rows, state error or None)."""
    y_ref, _, kappa = oracle.taylor_attention(q, k, v, P)
    err, excluded = check_rows(y_gpu, y_ref, kappa, y_tol(ops, out_dtype), P, label, oracle.term_scale(q, k, v, P))
    s_err = None
    if S_gpu is not None:
        s_err = check_state(S_gpu, k, v, P, ops, q.shape[0], chunk, label)
    return err, excluded, s_err
