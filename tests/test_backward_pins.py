"""Pins for the oracle's backward (oracle.taylor_attention_backward).

The gradients are checked against central finite differences of the oracle's
own forward (the loss L = sum(dy * y)), against automatic differentiation of a
forward written with torch float64 operations, and against the closed form of
the P = 1 case (uniform weights: y is the running mean of v).  Plausible
mistakes planted in a copy of the backward fail the finite-difference pin.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import taylor as ta


def _loss(q, k, v, dy, P):
    y, _, _ = oracle.taylor_attention(q, k, v, P)
    return float(np.sum(dy * y))


def _fd_grads(q, k, v, dy, P, h=1e-6):
    out = []
    for which in range(3):
        arrs = [q.copy(), k.copy(), v.copy()]
        g = np.zeros_like(arrs[which])
        for idx in np.ndindex(g.shape):
            plus = [a.copy() for a in arrs]
            minus = [a.copy() for a in arrs]
            plus[which][idx] += h
            minus[which][idx] -= h
            g[idx] = (_loss(*plus, dy, P) - _loss(*minus, dy, P)) / (2 * h)
        out.append(g)
    return out


def check_fd(backward) -> bool:
    rng = np.random.default_rng(41)
    for P in range(1, 6):
        n, dk, dv = 6, 3, 2
        q, k = rng.standard_normal((n, dk)), rng.standard_normal((n, dk))
        v, dy = rng.standard_normal((n, dv)), rng.standard_normal((n, dv))
        got = backward(q, k, v, dy, P)
        want = _fd_grads(q, k, v, dy, P)
        for g, w in zip(got, want):
            if not np.allclose(g, w, rtol=1e-6, atol=1e-8):
                return False
    return True


def test_backward_matches_finite_differences():
    assert check_fd(oracle.taylor_attention_backward)


@pytest.mark.parametrize("P", [2, 3, 4])
def test_backward_matches_torch_autograd(P):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(50 + P)
    n, dk, dv = 70, 8, 5
    q, k, v, dy = (rng.standard_normal(s) for s in ((n, dk), (n, dk), (n, dv), (n, dv)))
    tq, tk, tv = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (q, k, v))
    s = tq @ tk.T / math.sqrt(dk)
    w = sum(s ** p / math.factorial(p) for p in range(P))
    w = torch.tril(w)
    y = (w @ tv) / w.sum(dim=1, keepdim=True)
    (y * torch.tensor(dy)).sum().backward()
    got = oracle.taylor_attention_backward(q, k, v, dy, P)
    for g, t in zip(got, (tq, tk, tv)):
        np.testing.assert_allclose(g, t.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_backward_P1_is_running_mean():
    """P = 1: every weight is 1, y_T is the mean of v_0..v_T, so q and k get
    no gradient and dL/dv_t = sum_{T >= t} dy_T / (T + 1)."""
    rng = np.random.default_rng(3)
    n = 9
    q, k, v, dy = (rng.standard_normal((n, 4)) for _ in range(4))
    dq, dk, dv = oracle.taylor_attention_backward(q, k, v, dy, 1)
    assert np.all(dq == 0) and np.all(dk == 0)
    want = np.array([sum(dy[T] / (T + 1) for T in range(t, n)) for t in range(n)])
    np.testing.assert_allclose(dv, want, rtol=1e-14)


def test_backward_row_blocks_do_not_change_it():
    rng = np.random.default_rng(4)
    q, k, v, dy = (rng.standard_normal((40, 4)) for _ in range(4))
    a = oracle.taylor_attention_backward(q, k, v, dy, 4, block=512)
    b = oracle.taylor_attention_backward(q, k, v, dy, 4, block=7)
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- planted mistakes

def _variant(derivative_terms=-1, y_sign=1.0, mask_dk=True, dv_over_z=True):
    def backward(q, k, v, dy, P, block=512):
        n, d_k = q.shape
        c = math.sqrt(d_k)
        s = q @ k.T / c
        mask = np.arange(n)[None, :] <= np.arange(n)[:, None]
        w = np.where(mask, ta.taylor_poly(s, P), 0.0)
        dw_ds = np.where(mask, ta.taylor_poly(s, P + derivative_terms), 0.0)
        Z = w.sum(1)
        y = (w @ v) / Z[:, None]
        g = dy / Z[:, None]
        dL_dw = g @ v.T - y_sign * np.sum(g * y, 1, keepdims=True)
        dL_ds = np.where(mask, dL_dw * dw_ds, 0.0)
        dq = dL_ds @ k / c
        dk = (dL_ds if mask_dk else dL_dw * ta.taylor_poly(s, P + derivative_terms)).T @ q / c
        dv = w.T @ (g if dv_over_z else dy)
        return dq, dk, dv
    return backward


@pytest.mark.parametrize("name,kw", [
    ("derivative with the full series", dict(derivative_terms=0)),
    ("sign of the normaliser term", dict(y_sign=-1.0)),
    ("future queries in dk", dict(mask_dk=False)),
    ("dv not divided by Z", dict(dv_over_z=False)),
])
def test_backward_mutants_are_caught(name, kw):
    assert check_fd(_variant()), "the unmutated copy must pass"
    assert not check_fd(_variant(**kw)), name
