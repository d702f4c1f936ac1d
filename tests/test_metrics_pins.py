"""Pins for the comparison measures and the cancellation factor kappa, and a
check that the element-wise state comparison can fail where the whole-state
Frobenius comparison cannot.

Hand-computed arrays pin every measure of ``oracle.metrics``; kappa is pinned
by a worked two-token example and by the fact that an odd number of Taylor
terms gives a series with no real root (so every weight is positive and
kappa is exactly 1); ``state_abs_ref`` is pinned by brute force, by equality
with the state for non-negative inputs and by the triangle inequality.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import metrics as me
from oracle import taylor as ta


# ---------------------------------------------------------------- measures on hand-computed arrays

def test_row_rel_error_hand_values():
    y = np.array([[3.0, 4.0], [1.0, 0.0], [0.0, 2.0]])
    y_hat = np.array([[3.0, 4.0], [1.0, 1.0], [0.0, 3.0]])
    np.testing.assert_array_equal(me.row_rel_error(y_hat, y), [0.0, 1.0, 0.5])


def test_max_row_rel_error_counts_and_refuses_empty():
    y = np.array([[3.0, 4.0], [1.0, 0.0], [0.0, 2.0]])
    y_hat = np.array([[3.0, 4.0], [1.0, 1.0], [0.0, 3.0]])
    assert me.max_row_rel_error(y_hat, y) == (1.0, 0)
    # the row with error 1 is ill-conditioned and left out; one row excluded
    assert me.max_row_rel_error(y_hat, y, kappa=[1.0, 101.0, 1.0]) == (0.5, 1)
    assert me.max_row_rel_error(y_hat, y, kappa=[1.0, 100.0, 1.0]) == (1.0, 0)  # the bound is inclusive
    with pytest.raises(ValueError):
        me.max_row_rel_error(y_hat, y, kappa=[150.0, 101.0, 1e9])
    with pytest.raises(ValueError):
        me.max_row_rel_error(np.zeros((0, 2)), np.zeros((0, 2)))


def test_row_rel_error_floor_hand_values():
    """With term scales rho, ||y_T|| is floored at rho_T / 10: row 0 (norm 5)
    is left alone by rho = 20, row 1 (norm 1) is judged against 30 / 10 = 3,
    and row 2 (an exactly cancelled numerator, norm 0) against 50 / 10 = 5."""
    y = np.array([[3.0, 4.0], [1.0, 0.0], [0.0, 0.0]])
    y_hat = np.array([[3.0, 5.0], [1.0, 1.5], [0.0, 0.5]])
    assert me.CANCEL_FLOOR == 10.0
    np.testing.assert_allclose(me.row_rel_error(y_hat, y, scale=[20.0, 30.0, 50.0]), [0.2, 0.5, 0.1], rtol=1e-15)
    assert me.max_row_rel_error(y_hat, y, kappa=[1.0, 1.0, 1.0], scale=[20.0, 30.0, 50.0]) == (0.5, 0)
    # without scales the cancelled row has no finite relative error
    with np.errstate(divide="ignore"):
        assert math.isinf(me.row_rel_error(y_hat, y)[2])


def test_term_scale_closed_forms():
    """P = 1 makes every weight 1: rho_T = sqrt(sum_{t<=T} ||v_t||^2) / (T + 1).
    P = 2 makes the weights 1 + q_T.k_t / sqrt(d), written out here with a loop
    over tokens; both with and without a row list."""
    rng = np.random.default_rng(17)
    q, k, v = rng.standard_normal((9, 3)), rng.standard_normal((9, 3)), rng.standard_normal((9, 2))
    vv = np.cumsum((v ** 2).sum(axis=1))
    np.testing.assert_allclose(oracle.term_scale(q, k, v, 1), np.sqrt(vv) / np.arange(1, 10), rtol=1e-14)
    want = []
    for T in range(9):
        w = [1.0 + float(np.dot(q[T], k[t])) / math.sqrt(3.0) for t in range(T + 1)]
        want.append(math.sqrt(sum(w[t] ** 2 * float(np.dot(v[t], v[t])) for t in range(T + 1))) / abs(sum(w)))
    np.testing.assert_allclose(oracle.term_scale(q, k, v, 2), want, rtol=1e-13)
    np.testing.assert_allclose(oracle.term_scale(q, k, v, 2, rows=[8, 2]), [want[8], want[2]], rtol=1e-13)


def test_term_scale_floor_leaves_one_term_rows_alone():
    """A row with a single term (T = 0) has ||y_0|| = ||v_0|| = rho_0, ten
    times the floor, so the floor never binds there; for non-negative weights
    and values ||y_T|| >= rho_T (the norm of a sum of non-negative vectors is
    at least the root-sum-square of their norms), so it never binds either."""
    rng = np.random.default_rng(3)
    q, k = rng.standard_normal((40, 4)), rng.standard_normal((40, 4))
    v = np.abs(rng.standard_normal((40, 5)))
    y, _, _ = oracle.taylor_attention(q, k, v, 3)
    rho = oracle.term_scale(q, k, v, 3)
    assert np.all(np.linalg.norm(y, axis=1) >= rho * (1 - 1e-12))
    np.testing.assert_allclose(rho[0], np.linalg.norm(v[0]), rtol=1e-14)
    y_hat = y * (1 + 1e-3)
    np.testing.assert_array_equal(me.row_rel_error(y_hat, y, rho), me.row_rel_error(y_hat, y))


def test_state_rel_error_hand_value():
    assert me.state_rel_error([[3.0, 5.0]], [[3.0, 4.0]]) == pytest.approx(0.2, rel=1e-15)


def test_state_elem_error_hand_values():
    S = np.array([[1.0, -1.0], [0.0, 2.0]])
    S_abs = np.array([[5.0, 3.0], [0.0, 2.0]])
    assert me.state_elem_error([[1.5, -1.0], [0.0, 2.0]], S, S_abs) == pytest.approx(0.1, rel=1e-15)
    assert me.state_elem_error([[1.0, -1.3], [0.0, 2.0]], S, S_abs) == pytest.approx(0.1, rel=1e-12)
    assert me.state_elem_error(S, S, S_abs) == 0.0
    # an entry made of no terms must be exactly zero
    assert me.state_elem_error([[1.0, -1.0], [1e-30, 2.0]], S, S_abs) == math.inf
    assert me.state_elem_error([[1.0, np.nan], [0.0, 2.0]], S, S_abs) == math.inf


def test_log10_abs_diff_hand_values():
    np.testing.assert_allclose(me.log10_abs_diff([1.001, 5.0, 2.0], [1.0, 4.0, 2.0]), [-3.0, 0.0, -300.0],
                               rtol=0, atol=1e-9)


def test_tolerances():
    u32, ubf = 2.0 ** -24, 2.0 ** -8
    assert me.state_tol("f32", 256, 64, 4) == 2 * (64 + 4 + 16) * u32
    assert me.state_tol("f32", 256, 64, 4, steps=10) == 2 * (64 + 4 + 10 + 16) * u32
    assert me.state_tol("bf16", 8192, 64, 4) == 4 * ubf + 2 * (64 + 128 + 16) * u32
    assert me.state_tol("split", 65536, 64, 6) == 6 * ubf ** 2 + 2 * (64 + 1024 + 24) * u32
    assert me.state_tol("f32", 0, 64, 4) == 0.0
    assert me.y_tol("bf16", "bf16") == 2e-2 and me.y_tol("bf16", "f32") == 2e-2
    assert me.y_tol("f32", "f32") == 1e-4 and me.y_tol("f32", "bf16") == 2.0 ** -8
    assert me.y_tol("split", "f32") == 1e-4
    with pytest.raises(ValueError):
        me.state_tol("f16", 8, 8, 2)


# ---------------------------------------------------------------- kappa

def test_kappa_worked_example():
    """d = 1, P = 2 (f_2(s) = 1 + s): q = (1, 1), k = (0.5, -3), v = (2, 4).
    Row 0: w = [1.5], y = 2, Z = 1.5, kappa = 1.  Row 1: w = [1.5, -2],
    Z = -0.5, y = (1.5*2 - 2*4) / -0.5 = 10, kappa = 3.5 / 0.5 = 7."""
    q = np.array([[1.0], [1.0]])
    k = np.array([[0.5], [-3.0]])
    v = np.array([[2.0], [4.0]])
    y, Z, kappa = oracle.taylor_attention(q, k, v, 2)
    np.testing.assert_allclose(y[:, 0], [2.0, 10.0], rtol=1e-15)
    np.testing.assert_allclose(Z, [1.5, -0.5], rtol=1e-15)
    np.testing.assert_allclose(kappa, [1.0, 7.0], rtol=1e-15)
    yr, Zr, kr = oracle.taylor_attention_rows(q, k, v, 2, [0, 1])
    np.testing.assert_allclose(kr, [1.0, 7.0], rtol=1e-15)


@pytest.mark.parametrize("P", [1, 3, 5, 7])
def test_odd_P_series_is_positive_and_kappa_is_one(P):
    """f_P with P odd is the exponential series cut after an even degree; it has
    no real root (its minimum, where f_P' = f_{P-1} vanishes, equals
    s^(P-1)/(P-1)! > 0), so every weight is positive and kappa = 1 exactly."""
    s = np.linspace(-60.0, 60.0, 200001)
    assert np.all(oracle.taylor_poly(s, P) > 0)
    rng = np.random.default_rng(P)
    q, k, v = (3.0 * rng.standard_normal((80, 6)) for _ in range(3))
    _, _, kappa = oracle.taylor_attention(q, k, v, P)
    np.testing.assert_allclose(kappa, 1.0, rtol=0, atol=1e-14)


def test_even_P_kappa_exceeds_one_where_weights_turn_negative():
    rng = np.random.default_rng(3)
    q, k, v = (3.0 * rng.standard_normal((80, 6)) for _ in range(3))
    _, _, kappa = oracle.taylor_attention(q, k, v, 4)
    assert np.all(kappa >= 1.0 - 1e-14) and kappa.max() > 1.0


# ---------------------------------------------------------------- state magnitudes

def check_state_abs(mod) -> bool:
    rng = np.random.default_rng(17)
    # brute force on a tiny case: every monomial written out by hand
    d, P, n = 2, 3, 3
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, 2))
    c = math.sqrt(d)
    mono = [lambda x: 1.0, lambda x: x[0] / c ** 0.5, lambda x: x[1] / c ** 0.5,
            lambda x: x[0] * x[0] / (c * math.sqrt(2)), lambda x: x[0] * x[1] / c,
            lambda x: x[1] * x[1] / (c * math.sqrt(2))]
    brute = np.zeros((6, 3))
    for t in range(n):
        ve = [v[t, 0], v[t, 1], 1.0]
        for f, m in enumerate(mono):
            for j in range(3):
                brute[f, j] += abs(m(k[t])) * abs(ve[j])
    if not np.allclose(mod.state_abs_ref(k, v, P), brute, rtol=1e-13, atol=0):
        return False
    # equal to the state itself when no term is negative
    k, v = np.abs(rng.standard_normal((40, 4))), np.abs(rng.standard_normal((40, 3)))
    if not np.allclose(mod.state_abs_ref(k, v, 4), mod.state_ref(k, v, 4), rtol=1e-13, atol=0):
        return False
    # triangle inequality, strict somewhere for signed inputs
    k, v = rng.standard_normal((40, 4)), rng.standard_normal((40, 3))
    A, S = mod.state_abs_ref(k, v, 4), mod.state_ref(k, v, 4)
    return bool(np.all(A >= np.abs(S) * (1 - 1e-13)) and np.any(A > np.abs(S) * 1.5))


def test_state_abs_ref_pins():
    assert check_state_abs(ta)


def test_state_abs_ref_mutants_are_caught():
    real = ta.state_abs_ref

    def signed_values(k, v, P):
        return np.abs(ta.phi_ref(k, P)).T @ np.concatenate([v, np.ones((len(v), 1))], 1)

    def missing_weights(k, v, P):
        return real(k, v, P) * np.r_[1.0, np.ones(ta.feature_count(k.shape[1], P) - 1) * 2.0][:, None]

    class M:
        state_ref = staticmethod(ta.state_ref)

    for bad in (signed_values, missing_weights):
        M.state_abs_ref = staticmethod(bad)
        assert not check_state_abs(M), bad.__name__


# ---------------------------------------------------------------- the element-wise check can fail

def test_swapped_or_zeroed_top_rows_fail_elementwise_but_pass_frobenius():
    """d = 32, P = 4, bf16 N(0,1) keys and values, 8192 tokens (the benchmark's
    head shape and length).  Two degree-3 rows of the oracle's own state
    swapped, or its eight largest degree-3 rows zeroed, stay within 2e-2 in the
    whole-head Frobenius measure (the degree-0 row dominates it) but fail the
    element-wise bound of a bfloat16-operand path several times over."""
    import sata_synth as syn
    d, P, n = 32, 4, 8192
    _, k, v = syn.make_head(3, 0, 0, n, d, d, "bf16")
    S = oracle.state_ref(k, v, P)
    S_abs = oracle.state_abs_ref(k, v, P)
    tol = me.state_tol("bf16", n, 64, P)
    assert me.state_elem_error(S, S, S_abs) == 0.0
    top = np.arange(1 + d + d * (d + 1) // 2, S.shape[0])
    norms = np.linalg.norm(S[top], axis=1)
    a, b = top[np.argsort(norms)[-2:]]
    swapped = S.copy()
    swapped[[a, b]] = S[[b, a]]
    zeroed = S.copy()
    zeroed[top[np.argsort(norms)[-8:]]] = 0.0
    for bad in (swapped, zeroed):
        assert me.state_rel_error(bad, S) < 2e-2
        assert me.state_elem_error(bad, S, S_abs) > 4 * tol
