"""Helpers shared by the GPU parity tests (host-side marshalling only)."""
import numpy as np

import oracle
from oracle.metrics import KAPPA_MAX, max_row_rel_error, state_rel_error

TOL = {"f32": oracle.TOL_F32, "bf16": oracle.TOL_BF16}


def torch_dtype(dtype):
    import torch
    return torch.float32 if dtype == "f32" else torch.bfloat16


def to_dev(arr, dtype):
    """float32 array whose values are exact in `dtype` -> device tensor of that dtype."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda().to(torch_dtype(dtype))


def to_host(t):
    return t.float().cpu().numpy().astype(np.float64)


def check_prefill_head(y_gpu, S_gpu, q, k, v, P, dtype, label=""):
    """Compare one head's GPU prefill output (and state) with the oracle.

    Returns (max row error, excluded rows, state error or None)."""
    y_ref, _, kappa = oracle.taylor_attention(q, k, v, P)
    # rows whose denominator cancels (kappa > KAPPA_MAX, even P only) may divide by
    # a rounded zero; every other row must be finite and within tolerance
    assert np.all(np.isfinite(y_gpu[kappa <= KAPPA_MAX])), f"{label}: non-finite well-conditioned row"
    err, excluded = max_row_rel_error(y_gpu, y_ref, kappa)
    assert err <= TOL[dtype], f"{label}: max row rel error {err:.3e} > {TOL[dtype]:.0e} (excluded {excluded})"
    s_err = None
    if S_gpu is not None:
        S_ref = oracle.state_ref(k, v, P)
        s_err = state_rel_error(S_gpu, S_ref)
        assert s_err <= TOL[dtype], f"{label}: state rel error {s_err:.3e}"
    return err, excluded, s_err
