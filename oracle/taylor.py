"""Float64 CPU oracle for symmetry-aware Taylor attention (arXiv 2602.00294).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check of the entry
module and the CPU-baseline leg of the benchmark may import or run this code.
The GPU product path never calls it and shares no code with it: the feature
table, the weights and every reduction here are computed independently of the
HIP library.

Everything is float64 and deliberately plain.  Where the method has a direct
definition the oracle writes that definition out; the only library primitives
used as steps are matrix products and sums.

What is computed (sections of the paper in brackets):

* ``taylor_poly``      f_P(s) = sum_{p<P} s^p / p!, the truncated exponential
                        series used for every query-key pair
                        [Sec. 2.1 Taylor expansion; Sec. 2.4 truncation to P
                        terms].
* ``taylor_attention`` causal attention with exp replaced by f_P, computed
                        directly from its definition: weights
                        f_P(q_T . k_t / sqrt(d_k)) for t <= T (inclusive), then
                        numerator / denominator [App. A2, the causal output
                        y_T and its Taylor substitution].
* ``term_scale``        the root-sum-square size of a row's terms w_Tt v_t over
                        |Z_T|: the size that roundings of independent signs
                        add up to, below which a row's numerator has cancelled
                        by accident [App. A2, the causal output y_T].
* ``softmax_attention`` the exact causal softmax attention it approximates
                        [App. A2, first display].
* ``multi_indices`` / ``multiplicity`` / ``phi_ref``
                        the minimal symmetric monomial basis (upper
                        hyper-triangle i1 <= ... <= ip), the permutation counts
                        that form the diagonal of C_p, and the feature map with
                        the weights split evenly between query and key
                        [Sec. 2.3, Sec. 2.4 weighted inner product, App. A1].
* ``state_ref`` / ``readout_ref`` / ``recurrent_attention`` / ``decode_ref``
                        the accumulated states S = sum_t phi(k_t) (x) [v_t, 1]
                        and their readout, as the paper's linear-attention
                        recurrence [App. A2, accumulated feature states and
                        evaluation at the query].
* ``state_abs_ref``     the same sum over absolute values, sum_t |phi(k_t)| (x)
                        |[v_t, 1]|: the size of the terms that make up each
                        state entry, against which a rounded state is judged
                        [App. A2, accumulated feature states].
* ``taylor_attention_backward``
                        the gradients dL/dq, dL/dk, dL/dv of a loss through
                        the causal output, for a given dL/dy: the derivative
                        of the direct definition above, written out row by row
                        (the paper names training as the next step and gives
                        no backward; this is calculus on App. A2's output).
* ``feature_count`` / ``state_elems`` / ``flops_per_token``
                        the closed forms of Sec. 2.6 and Sec. 2.7.

Readings of points the paper leaves open (also listed in the design notes):

1. The weight alpha_p * C_p[m] is split symmetrically, so one map serves both
   queries and keys: phi_m(x) = sqrt(alpha_p * C_p[m]) * prod_j x[m_j]
   = x^m / (d^{p/4} sqrt(prod_j c_j!)).  The attention output does not depend
   on this choice; the feature vector and the state do.
2. Feature order: degree-major, and inside one degree the non-decreasing index
   tuples in lexicographic order (the order of the paper's d = p = 2 example).
   Indices are 0-based.
3. State layout: one matrix [D][d_v + 1] per head; column d_v holds the
   normaliser (the value vector extended by a constant 1).
4. The causal sum is inclusive (t <= T); a decode step updates the state with
   the new token before reading it out.
5. The scaling constant is c = sqrt(d_k), also when d_v != d_k.
6. No clamp or epsilon in the division; for even P the polynomial has a real
   root, so rows whose denominator nearly cancels are flagged through
   kappa_T = sum_t |f_Tt| / |sum_t f_Tt| instead of being altered.
"""
from __future__ import annotations

import itertools
import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "taylor_poly", "taylor_attention", "taylor_attention_rows", "term_scale", "taylor_attention_backward",
    "softmax_attention",
    "softmax_attention_rows", "multi_indices", "multiplicity", "alpha", "feature_weights",
    "phi_ref", "state_ref", "state_abs_ref", "readout_ref", "recurrent_attention", "decode_ref",
    "feature_count", "degree_count", "state_elems", "flops_per_token",
]


# --------------------------------------------------------------------------------------
# Closed forms (Sec. 2.3, Sec. 2.6, Sec. 2.7)
# --------------------------------------------------------------------------------------

def degree_count(d: int, p: int) -> int:
    """m_p = C(d + p - 1, p): unique monomials of degree p over d coordinates (Sec. 2.3)."""
    return math.comb(d + p - 1, p)


def feature_count(d: int, P: int) -> int:
    """D = C(d + P - 1, P - 1): features of degrees 0..P-1 (Sec. 2.6, hidden state size)."""
    return math.comb(d + P - 1, P - 1)


def state_elems(d_k: int, d_v: int, P: int) -> int:
    """(d_v + 1) * C(d_k + P - 1, P - 1): elements of the per-head state (Sec. 2.6)."""
    return (d_v + 1) * feature_count(d_k, P)


def flops_per_token(d_k: int, d_v: int, P: int) -> float:
    """Forward FLOPs per token, closed form of Sec. 2.7 (all Taylor terms)."""
    return (4 * d_v + 2 * (P * d_k + 1) / (d_k + 1) + 2) * feature_count(d_k, P)


# --------------------------------------------------------------------------------------
# Truncated Taylor series of exp (Sec. 2.1, Sec. 2.4 "Truncating for Approximation")
# --------------------------------------------------------------------------------------

def alpha(p: int, d_k: int) -> float:
    """alpha_p = 1 / (p! c^p) with c = sqrt(d_k) (Sec. 2.1)."""
    return 1.0 / (math.factorial(p) * math.sqrt(d_k) ** p)


def taylor_poly(s: np.ndarray, P: int) -> np.ndarray:
    """f_P(s) = sum_{p=0}^{P-1} s^p / p!, elementwise, float64.

    The powers are built term by term (term_p = term_{p-1} * s / p), which is
    s^p / p! without a separate factorial.
    """
    s = np.asarray(s, dtype=np.float64)
    total = np.zeros_like(s)
    term = np.ones_like(s)
    for p in range(P):
        if p > 0:
            term = term * s / p
        total = total + term
    return total


# --------------------------------------------------------------------------------------
# Direct causal attention: the definition, blocked only by query rows (App. A2)
# --------------------------------------------------------------------------------------

def _as64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def taylor_attention(q, k, v, P: int, block: int = 512):
    """Causal truncated-Taylor attention for one head, straight from its definition.

    q: [n, d_k], k: [n, d_k], v: [n, d_v] (any real dtype; upcast exactly to float64).
    Returns (y [n, d_v], Z [n], kappa [n]) where for each 0-based row T

        w_Tt  = f_P(q_T . k_t / sqrt(d_k))             for t <= T
        Z_T   = sum_t w_Tt
        y_T   = (sum_t w_Tt v_t) / Z_T
        kappa = sum_t |w_Tt| / |Z_T|                    (cancellation factor)
    """
    q, k, v = _as64(q), _as64(k), _as64(v)
    n, d_k = q.shape
    d_v = v.shape[1]
    c = math.sqrt(d_k)
    y = np.empty((n, d_v))
    Z = np.empty(n)
    kappa = np.empty(n)
    for r0 in range(0, n, block):
        r1 = min(n, r0 + block)
        s = (q[r0:r1] @ k[:r1].T) / c                       # [rows, r1]
        w = taylor_poly(s, P)
        rows = np.arange(r0, r1)[:, None]
        cols = np.arange(r1)[None, :]
        w = np.where(cols <= rows, w, 0.0)                  # inclusive causal mask
        num = w @ v[:r1]
        den = w.sum(axis=1)
        y[r0:r1] = num / den[:, None]
        Z[r0:r1] = den
        kappa[r0:r1] = np.abs(w).sum(axis=1) / np.abs(den)
    return y, Z, kappa


def taylor_attention_rows(q, k, v, P: int, rows: Sequence[int]):
    """The same definition evaluated only at the given 0-based query rows.

    Used for full-size parity checks, where the quadratic oracle cannot run on
    the whole sequence.  Returns (y [len(rows), d_v], Z, kappa).
    """
    q, k, v = _as64(q), _as64(k), _as64(v)
    d_k = q.shape[1]
    c = math.sqrt(d_k)
    rows = list(rows)
    y = np.empty((len(rows), v.shape[1]))
    Z = np.empty(len(rows))
    kappa = np.empty(len(rows))
    for i, T in enumerate(rows):
        s = (k[: T + 1] @ q[T]) / c
        w = taylor_poly(s, P)
        den = w.sum()
        y[i] = (w @ v[: T + 1]) / den
        Z[i] = den
        kappa[i] = np.abs(w).sum() / abs(den)
    return y, Z, kappa


def term_scale(q, k, v, P: int, rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """rho_T = sqrt(sum_{t <= T} w_Tt^2 ||v_t||^2) / |Z_T| per query row T
    (every row when rows is None), with w_Tt and Z_T as in taylor_attention.

    y_T is a sum of the terms w_Tt v_t / Z_T; roundings of independent signs in
    those terms add up to about rho_T times the unit roundoff, whatever the
    size of the sum.  A row whose numerator cancels by accident has
    ||y_T|| far below rho_T; the row error measure floors ||y_T|| at a fixed
    fraction of rho_T (metrics.row_rel_error)."""
    q, k, v = _as64(q), _as64(k), _as64(v)
    n, d_k = q.shape
    c = math.sqrt(d_k)
    vv = (v * v).sum(axis=1)                                # ||v_t||^2
    if rows is None:                                        # all rows, blocked by query rows
        out = np.empty(n)
        for r0 in range(0, n, 512):
            r1 = min(n, r0 + 512)
            w = taylor_poly((q[r0:r1] @ k[:r1].T) / c, P)
            w = np.where(np.arange(r1)[None, :] <= np.arange(r0, r1)[:, None], w, 0.0)
            out[r0:r1] = np.sqrt((w * w) @ vv[:r1]) / np.abs(w.sum(axis=1))
        return out
    rows = list(rows)
    out = np.empty(len(rows))
    for i, T in enumerate(rows):
        w = taylor_poly((k[: T + 1] @ q[T]) / c, P)
        out[i] = math.sqrt(float((w * w) @ vv[: T + 1])) / abs(w.sum())
    return out


def taylor_attention_backward(q, k, v, dy, P: int, block: int = 512):
    """Gradients of the causal truncated-Taylor attention of one head.

    q, k: [n, d_k], v: [n, d_v], dy = dL/dy: [n, d_v].  With, for t <= T,
        s_Tt = q_T . k_t / c,  w_Tt = f_P(s_Tt),  Z_T = sum_t w_Tt,
        y_T  = sum_t w_Tt v_t / Z_T,
    the chain rule gives
        dL/dw_Tt = dy_T . (v_t - y_T) / Z_T
        dL/ds_Tt = dL/dw_Tt * f_P'(s_Tt),  f_P' = f_{P-1}  (the series cut one term earlier)
        dL/dq_T  = sum_{t <= T} dL/ds_Tt k_t / c
        dL/dk_t  = sum_{T >= t} dL/ds_Tt q_T / c
        dL/dv_t  = sum_{T >= t} w_Tt dy_T / Z_T.
    Returns (dq [n, d_k], dk [n, d_k], dv [n, d_v]), float64."""
    q, k, v, dy = _as64(q), _as64(k), _as64(v), _as64(dy)
    n, d_k = q.shape
    c = math.sqrt(d_k)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for r0 in range(0, n, block):
        r1 = min(n, r0 + block)
        s = (q[r0:r1] @ k[:r1].T) / c                       # [rows, r1]
        rows = np.arange(r0, r1)[:, None]
        cols = np.arange(r1)[None, :]
        mask = cols <= rows                                  # inclusive causal mask
        w = np.where(mask, taylor_poly(s, P), 0.0)
        dw_ds = np.where(mask, taylor_poly(s, P - 1), 0.0)
        Z = w.sum(axis=1)
        y = (w @ v[:r1]) / Z[:, None]
        g = dy[r0:r1] / Z[:, None]                           # dL/dN_T
        dL_dw = g @ v[:r1].T - np.sum(g * y, axis=1, keepdims=True)
        dL_ds = np.where(mask, dL_dw * dw_ds, 0.0)
        dq[r0:r1] = (dL_ds @ k[:r1]) / c
        dk[:r1] += (dL_ds.T @ q[r0:r1]) / c
        dv[:r1] += w.T @ g
    return dq, dk, dv


def softmax_attention(q, k, v, block: int = 512) -> np.ndarray:
    """Exact causal softmax attention with c = sqrt(d_k), float64 (App. A2).

    The row maximum is subtracted before exponentiating; this changes nothing
    mathematically and keeps exp in range.
    """
    q, k, v = _as64(q), _as64(k), _as64(v)
    n, d_k = q.shape
    c = math.sqrt(d_k)
    y = np.empty((n, v.shape[1]))
    for r0 in range(0, n, block):
        r1 = min(n, r0 + block)
        s = (q[r0:r1] @ k[:r1].T) / c
        rows = np.arange(r0, r1)[:, None]
        cols = np.arange(r1)[None, :]
        s = np.where(cols <= rows, s, -np.inf)
        e = np.exp(s - s.max(axis=1, keepdims=True))
        y[r0:r1] = (e @ v[:r1]) / e.sum(axis=1, keepdims=True)
    return y


def softmax_attention_rows(q, k, v, rows: Sequence[int]) -> np.ndarray:
    """Exact causal softmax attention at selected 0-based query rows."""
    q, k, v = _as64(q), _as64(k), _as64(v)
    c = math.sqrt(q.shape[1])
    out = np.empty((len(rows), v.shape[1]))
    for i, T in enumerate(rows):
        s = (k[: T + 1] @ q[T]) / c
        e = np.exp(s - s.max())
        out[i] = (e @ v[: T + 1]) / e.sum()
    return out


# --------------------------------------------------------------------------------------
# Minimal symmetric basis and feature map (Sec. 2.3, Sec. 2.4, App. A1)
# --------------------------------------------------------------------------------------

def multi_indices(d: int, P: int) -> List[Tuple[int, ...]]:
    """All non-decreasing index tuples of lengths 0..P-1 over range(d).

    Degree-major; inside a degree, lexicographic order.  Degree 0 is the empty
    tuple, whose monomial is the empty product 1 (App. A1).
    """
    out: List[Tuple[int, ...]] = []
    for p in range(P):
        out.extend(itertools.combinations_with_replacement(range(d), p))
    return out


def multiplicity(m: Iterable[int]) -> int:
    """Diagonal entry of C_p for a sorted tuple m: the number of ordered index
    tuples that are permutations of m, i.e. p! / prod_j (count of index j)!."""
    m = tuple(m)
    counts = {}
    for i in m:
        counts[i] = counts.get(i, 0) + 1
    denom = 1
    for c in counts.values():
        denom *= math.factorial(c)
    return math.factorial(len(m)) // denom


def feature_weights(d: int, P: int) -> np.ndarray:
    """sqrt(alpha_p * C_p[m]) for every feature m, in feature order (reading 1)."""
    return np.array([math.sqrt(alpha(len(m), d) * multiplicity(m)) for m in multi_indices(d, P)])


def phi_ref(x, P: int) -> np.ndarray:
    """Feature map phi(x) for rows of x ([..., d] -> [..., D]), float64.

    phi_m(x) = sqrt(alpha_p C_p[m]) * prod_j x[m_j]; for m = () the product is 1.
    Then phi(q) . phi(k) = sum_p alpha_p <Phi_p(q), Phi_p(k)>_{C_p} = f_P(q.k/sqrt(d)).
    """
    x = _as64(x)
    d = x.shape[-1]
    idx = multi_indices(d, P)
    w = feature_weights(d, P)
    out = np.empty(x.shape[:-1] + (len(idx),))
    for f, m in enumerate(idx):
        prod = np.ones(x.shape[:-1])
        for i in m:
            prod = prod * x[..., i]
        out[..., f] = w[f] * prod
    return out


# --------------------------------------------------------------------------------------
# Linear-attention route through the accumulated state (App. A2)
# --------------------------------------------------------------------------------------

def _extend(v: np.ndarray) -> np.ndarray:
    """[v | 1]: values extended by the constant that accumulates the normaliser."""
    return np.concatenate([v, np.ones(v.shape[:-1] + (1,))], axis=-1)


def state_ref(k, v, P: int) -> np.ndarray:
    """S = sum_t phi(k_t) (x) [v_t, 1]  ->  [D, d_v + 1] (the Z_{p,T} and S_{p,T}
    of every degree stacked, normaliser in the last column)."""
    return phi_ref(k, P).T @ _extend(_as64(v))


def state_abs_ref(k, v, P: int) -> np.ndarray:
    """sum_t |phi(k_t)| (x) |[v_t, 1]|  ->  [D, d_v + 1].

    Entry (f, j) is the sum of the magnitudes of the terms whose sum is the
    state entry S[f, j].  A state accumulated in a precision with unit
    roundoff u (per term, plus the rounding of the running sums) is off by at
    most a small multiple of u times this entry, whatever the cancellation
    inside the sum; a misplaced row or column is off by the entry itself."""
    return np.abs(phi_ref(k, P)).T @ np.abs(_extend(_as64(v)))


def readout_ref(S, q, P: int) -> np.ndarray:
    """Readout at queries q ([m, d_k]) from a state S ([D, d_v + 1]): y = S_T / Z_T."""
    o = phi_ref(q, P) @ _as64(S)
    return o[..., :-1] / o[..., -1:]


def recurrent_attention(q, k, v, P: int) -> Tuple[np.ndarray, np.ndarray]:
    """Causal attention by the state recurrence, one token at a time.

    S_T = S_{T-1} + phi(k_T) (x) [v_T, 1], then y_T = readout at q_T.  Returns
    (y [n, d_v], final S).  Small inputs only.
    """
    q, k, v = _as64(q), _as64(k), _as64(v)
    fq, fk, ve = phi_ref(q, P), phi_ref(k, P), _extend(v)
    S = np.zeros((fk.shape[1], ve.shape[1]))
    y = np.empty((q.shape[0], v.shape[1]))
    for T in range(q.shape[0]):
        S = S + np.outer(fk[T], ve[T])
        o = fq[T] @ S
        y[T] = o[:-1] / o[-1]
    return y, S


def decode_ref(S0, q, k, v, P: int) -> Tuple[np.ndarray, np.ndarray]:
    """Sequential decode steps from state S0: update with (k_t, v_t), then read out q_t.

    q, k: [steps, d_k], v: [steps, d_v].  Returns (y [steps, d_v], final S).
    """
    q, k, v = _as64(q), _as64(k), _as64(v)
    S = np.array(S0, dtype=np.float64, copy=True)
    fq, fk, ve = phi_ref(q, P), phi_ref(k, P), _extend(v)
    y = np.empty((q.shape[0], v.shape[1]))
    for t in range(q.shape[0]):
        S += np.outer(fk[t], ve[t])
        o = fq[t] @ S
        y[t] = o[:-1] / o[-1]
    return y, S
