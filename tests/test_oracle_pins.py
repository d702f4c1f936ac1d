"""Pins for the float64 oracle: each check ties it to something other than itself.

Every check below compares the oracle with a fact fixed by the paper or by
mathematics: the printed worked example, closed forms, brute force over all
ordered index tuples, exact rational arithmetic, special cases that reduce to
textbook routines, a library softmax attention, and the Lagrange remainder
bound.  ``test_mutants_are_caught`` plants plausible mistakes in the oracle
(on the CPU) and shows that some pin fails for each of them.
"""
import collections
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import taylor as ta

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- counts (Sec. 2.3, 2.6)

def check_counts(mod) -> bool:
    for d in range(1, 9):
        for P in range(1, 7):
            idx = mod.multi_indices(d, P)
            if len(idx) != math.comb(d + P - 1, P - 1) or len(set(idx)) != len(idx):
                return False
            # brute force: distinct sorted tuples among all d^p ordered tuples
            for p in range(P):
                brute = {tuple(sorted(t)) for t in itertools.product(range(d), repeat=p)}
                if sorted(brute) != [m for m in idx if len(m) == p]:
                    return False
    return True


def test_feature_counts_against_brute_force():
    assert check_counts(ta)


def test_spot_feature_counts():
    # C(d+P-1, P-1) at the head sizes of the workloads (closed form, Sec. 2.6)
    assert [oracle.feature_count(d, 4) for d in (8, 16, 32, 64)] == [165, 969, 6545, 47905]
    assert [oracle.feature_count(16, P) for P in (2, 3, 4, 5, 6)] == [17, 153, 969, 4845, 20349]
    assert len(ta.multi_indices(32, 4)) == 6545


def test_state_size_closed_form():
    for dk, dv, P in [(8, 8, 4), (16, 16, 4), (32, 32, 4), (5, 3, 6), (64, 64, 4)]:
        per_degree = sum((dv + 1) * math.comb(dk + p - 1, p) for p in range(P))
        assert oracle.state_elems(dk, dv, P) == per_degree == (dv + 1) * oracle.feature_count(dk, P)


def test_flops_closed_form_equals_per_degree_sum():
    # Sec. 2.7 gives the per-degree count and its closed-form sum; they must agree.
    for dk, dv, P in [(8, 8, 4), (16, 16, 2), (16, 16, 6), (32, 32, 4), (7, 3, 5)]:
        per_degree = sum((4 * dv + 2 * p + 4) * math.comb(dk + p - 1, p) for p in range(P))
        assert oracle.flops_per_token(dk, dv, P) == pytest.approx(per_degree, rel=1e-12)


# ---------------------------------------------------------------- worked example, degree 0

def test_worked_example_d2_p2(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "worked_example_d2_p2.json")))
    basis = [m for m in ta.multi_indices(g["d"], g["p"] + 1) if len(m) == g["p"]]
    assert [list(m) for m in basis] == g["basis_zero_based"]
    assert [ta.multiplicity(m) for m in basis] == g["coefficients"]


def test_degree_zero(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "degree_zero.json")))
    for d in (1, 3, 16):
        idx = ta.multi_indices(d, 3)
        assert sum(1 for m in idx if len(m) == 0) == g["m_0"]
        assert idx[0] == ()
        phi = ta.phi_ref(_rng(d).standard_normal((4, d)), 3)
        assert np.all(phi[:, 0] == g["Phi_0"])


# ---------------------------------------------------------------- multiplicities, exact identity

def check_multiplicity(mod) -> bool:
    for d in range(1, 5):
        for p in range(0, 5):
            counts = collections.Counter(tuple(sorted(t)) for t in itertools.product(range(d), repeat=p))
            for m, c in counts.items():
                if mod.multiplicity(m) != c:
                    return False
    return True


def test_multiplicity_counts_permutations():
    assert check_multiplicity(ta)


def test_exact_rational_power_identity():
    """(q.k)^p == sum over the minimal basis of C_p[m] q^m k^m == sum over all d^p
    ordered tuples, in exact rational arithmetic (Sec. 2.2, eq. for (q^T k)^p)."""
    rng = _rng(3)
    for d in range(1, 5):
        for p in range(0, 5):
            q = [Fraction(int(a), int(b)) for a, b in zip(rng.integers(-5, 6, d), rng.integers(1, 4, d))]
            k = [Fraction(int(a), int(b)) for a, b in zip(rng.integers(-5, 6, d), rng.integers(1, 4, d))]
            dot = sum(a * b for a, b in zip(q, k))
            brute = Fraction(0)
            for t in itertools.product(range(d), repeat=p):
                term = Fraction(1)
                for i in t:
                    term *= q[i] * k[i]
                brute += term
            basis = Fraction(0)
            for m in ta.multi_indices(d, p + 1):
                if len(m) != p:
                    continue
                term = Fraction(ta.multiplicity(m))
                for i in m:
                    term *= q[i] * k[i]
                basis += term
            assert dot ** p == brute == basis


def test_exact_rational_truncated_series():
    """With d in {1, 4} the constant c = sqrt(d) is rational, so the truncated
    series sum_p alpha_p <Phi_p(q), Phi_p(k)>_{C_p} can be checked exactly
    against sum_p (q.k/c)^p / p! (Sec. 2.4, truncated expansion)."""
    rng = _rng(4)
    for d, c in ((1, 1), (4, 2)):
        for P in range(1, 7):
            q = [Fraction(int(a), 2) for a in rng.integers(-4, 5, d)]
            k = [Fraction(int(a), 2) for a in rng.integers(-4, 5, d)]
            s = sum(a * b for a, b in zip(q, k)) / c
            want = sum(s ** p / math.factorial(p) for p in range(P))
            got = Fraction(0)
            for m in ta.multi_indices(d, P):
                p = len(m)
                term = Fraction(ta.multiplicity(m), math.factorial(p) * c ** p)
                for i in m:
                    term *= q[i] * k[i]
                got += term
            assert got == want


# ---------------------------------------------------------------- feature map identity

def check_phi_identity(mod) -> bool:
    rng = _rng(5)
    for d in range(1, 7):
        for P in range(1, 8):
            q = rng.standard_normal((6, d))
            k = rng.standard_normal((6, d))
            got = np.sum(mod.phi_ref(q, P) * mod.phi_ref(k, P), axis=1)
            for i in range(6):
                s = float(q[i] @ k[i]) / math.sqrt(d)
                want = math.fsum(s ** p / math.factorial(p) for p in range(P))
                if not abs(got[i] - want) <= 1e-13 * max(1.0, abs(want)) * 10:
                    return False
    return True


def test_phi_inner_product_is_truncated_exp():
    assert check_phi_identity(ta)


def test_hierarchy_prefix_property():
    """Every degree-(p-1) monomial divides some degree-p monomial (Sec. 2.4
    footnote); in index-tuple form the shorter tuple is a prefix of a longer one."""
    for d in (1, 3, 7):
        idx = ta.multi_indices(d, 5)
        by_deg = collections.defaultdict(set)
        for m in idx:
            by_deg[len(m)].add(m)
        for p in range(1, 5):
            prefixes = {m[:-1] for m in by_deg[p]}
            assert by_deg[p - 1] <= prefixes


# ---------------------------------------------------------------- Taylor polynomial

def check_lagrange(mod) -> bool:
    rng = _rng(6)
    s = np.concatenate([rng.uniform(-3, 3, 2000), [0.0, 1e-3, -1e-3]])
    for P in range(1, 9):
        err = np.abs(np.exp(s) - mod.taylor_poly(s, P))
        bound = np.abs(s) ** P / math.factorial(P) * np.exp(np.maximum(s, 0.0))
        if not np.all(err <= bound * (1 + 1e-9) + 1e-15):
            return False
    return True


def test_lagrange_remainder_bound():
    assert check_lagrange(ta)


# ---------------------------------------------------------------- special cases of attention

def check_special_cases(mod) -> bool:
    rng = _rng(7)
    n, dk, dv = 37, 5, 3
    q, k, v = rng.standard_normal((n, dk)), rng.standard_normal((n, dk)), rng.standard_normal((n, dv))
    cum_mean = np.cumsum(v, axis=0) / np.arange(1, n + 1)[:, None]
    # P = 1: every weight is 1, so y is the running mean of v
    y1, _, _ = mod.taylor_attention(q, k, v, 1, block=8)
    if not np.allclose(y1, cum_mean, rtol=0, atol=1e-13):
        return False
    for P in range(1, 7):
        # q = 0: every weight is f_P(0) = 1
        y0, _, _ = mod.taylor_attention(np.zeros_like(q), k, v, P, block=16)
        if not np.allclose(y0, cum_mean, rtol=0, atol=1e-13):
            return False
        # first row: only t = T = 0 contributes
        yp, _, _ = mod.taylor_attention(q, k, v, P, block=16)
        if not np.allclose(yp[0], v[0], rtol=0, atol=1e-14):
            return False
    return True


def test_special_cases():
    assert check_special_cases(ta)


def test_p2_is_linear_attention_with_affine_features():
    """P = 2 is plain linear attention (Katharopoulos et al.) with the feature
    map psi(x) = [1, x / d^(1/4)]; evaluated here by prefix sums of outer products."""
    rng = _rng(8)
    n, dk, dv = 53, 6, 4
    q, k, v = rng.standard_normal((n, dk)), rng.standard_normal((n, dk)), rng.standard_normal((n, dv))
    psi = lambda x: np.concatenate([np.ones((x.shape[0], 1)), x / dk ** 0.25], axis=1)
    kv = np.cumsum(psi(k)[:, :, None] * v[:, None, :], axis=0)    # [n, 1+dk, dv]
    ks = np.cumsum(psi(k), axis=0)                                  # [n, 1+dk]
    want = np.einsum("nf,nfv->nv", psi(q), kv) / np.einsum("nf,nf->n", psi(q), ks)[:, None]
    got, _, _ = ta.taylor_attention(q, k, v, 2)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-13)


def check_two_routes(mod) -> bool:
    rng = _rng(9)
    for (n, dk, dv, P) in [(29, 3, 5, 1), (41, 4, 2, 2), (33, 5, 3, 3), (47, 3, 4, 4), (19, 2, 3, 6)]:
        q = rng.standard_normal((n, dk))
        k = rng.standard_normal((n, dk))
        v = rng.standard_normal((n, dv))
        y_direct, _, kappa = mod.taylor_attention(q, k, v, P, block=7)
        y_rec, S = mod.recurrent_attention(q, k, v, P)
        keep = kappa < 100
        if not np.allclose(y_direct[keep], y_rec[keep], rtol=1e-10, atol=1e-12):
            return False
        if not np.allclose(S, mod.state_ref(k, v, P), rtol=1e-12, atol=1e-12):
            return False
    return True


def test_direct_definition_equals_state_recurrence():
    """Two independent routes: the quadratic definition and the linear-attention
    recurrence over phi and the accumulated state (App. A2)."""
    assert check_two_routes(ta)


def test_decode_continues_prefill_state():
    rng = _rng(10)
    n1, n2, dk, dv, P = 30, 12, 4, 3, 4
    q = rng.standard_normal((n1 + n2, dk))
    k = rng.standard_normal((n1 + n2, dk))
    v = rng.standard_normal((n1 + n2, dv))
    S1 = ta.state_ref(k[:n1], v[:n1], P)
    y_dec, S2 = ta.decode_ref(S1, q[n1:], k[n1:], v[n1:], P)
    y_all, _, _ = ta.taylor_attention(q, k, v, P)
    np.testing.assert_allclose(y_dec, y_all[n1:], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(S2, ta.state_ref(k, v, P), rtol=1e-12, atol=1e-12)
    # the readout of the final state at the last query is the last output row
    np.testing.assert_allclose(ta.readout_ref(S2, q[-1:], P)[0], y_all[-1], rtol=1e-10)


def test_rows_variant_matches_full():
    rng = _rng(11)
    n, dk, dv, P = 300, 8, 8, 4
    q, k, v = rng.standard_normal((n, dk)), rng.standard_normal((n, dk)), rng.standard_normal((n, dv))
    y, Z, kap = ta.taylor_attention(q, k, v, P, block=64)
    rows = [0, 1, 63, 64, 150, 299]
    yr, Zr, kr = ta.taylor_attention_rows(q, k, v, P, rows)
    np.testing.assert_allclose(yr, y[rows], rtol=1e-12)
    np.testing.assert_allclose(Zr, Z[rows], rtol=1e-12)
    np.testing.assert_allclose(kr, kap[rows], rtol=1e-12)
    ys = ta.softmax_attention(q, k, v, block=64)
    np.testing.assert_allclose(ta.softmax_attention_rows(q, k, v, rows), ys[rows], rtol=1e-12)


# ---------------------------------------------------------------- softmax reference and convergence

def check_softmax_library(mod) -> bool:
    torch = pytest.importorskip("torch")
    rng = _rng(12)
    n, dk, dv = 70, 6, 5
    q, k, v = rng.standard_normal((n, dk)), rng.standard_normal((n, dk)), rng.standard_normal((n, dv))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None],
        is_causal=True).numpy()[0]
    return bool(np.allclose(mod.softmax_attention(q, k, v, block=16), ref, rtol=1e-12, atol=1e-13))


def test_softmax_matches_library_attention():
    assert check_softmax_library(ta)


def check_convergence(mod) -> bool:
    rng = _rng(13)
    n, d = 256, 16
    q, k, v = rng.standard_normal((n, d)), rng.standard_normal((n, d)), rng.standard_normal((n, d))
    ys = mod.softmax_attention(q, k, v)
    med = []
    for P in range(1, 8):
        y, _, _ = mod.taylor_attention(q, k, v, P)
        med.append(float(np.median(np.log10(np.abs(y - ys)[64:] + 1e-300))))
    y30, _, _ = mod.taylor_attention(q, k, v, 30)
    return all(b < a for a, b in zip(med, med[1:])) and float(np.max(np.abs(y30 - ys))) < 1e-11


def test_error_against_softmax_shrinks_with_P():
    """Each added Taylor term lowers the error against exact softmax (Sec. 3.1),
    and with many terms the truncated series reproduces softmax."""
    assert check_convergence(ta)


# ---------------------------------------------------------------- planted mistakes

class _Mutant:
    """A copy of the oracle namespace with one function replaced."""

    def __init__(self, **overrides):
        self.__dict__.update({k: getattr(ta, k) for k in ta.__all__})
        self.__dict__.update(overrides)
        # route internal calls through the replaced functions
        for name in ("taylor_attention", "recurrent_attention", "state_ref", "phi_ref", "softmax_attention"):
            if name not in overrides:
                setattr(self, name, _rebind(getattr(ta, name), self))


def _rebind(fn, ns):
    import types
    g = dict(fn.__globals__)
    g.update({k: getattr(ns, k) for k in ta.__all__ if hasattr(ns, k)})
    return types.FunctionType(fn.__code__, g, fn.__name__, fn.__defaults__, fn.__closure__)


def _poly_dropped_term(s, P):
    return ta.taylor_poly(s, P) - (np.asarray(s, float) ** (P - 1) / math.factorial(P - 1) if P > 1 else 0)


def _poly_wrong_sign(s, P):
    return ta.taylor_poly(-np.asarray(s, float), P)


def _multiplicity_missing(m):
    return 1


def _weights_no_alpha(d, P):
    return np.array([math.sqrt(ta.multiplicity(m)) for m in ta.multi_indices(d, P)])


def _exclusive_mask_attention(q, k, v, P, block=512):
    q, k, v = (np.asarray(a, float) for a in (q, k, v))
    n = q.shape[0]
    s = q @ k.T / math.sqrt(q.shape[1])
    w = ta.taylor_poly(s, P) * (np.arange(n)[None, :] < np.arange(n)[:, None])
    den = w.sum(1)
    return (w @ v) / den[:, None], den, np.abs(w).sum(1) / np.abs(den)


def _wrong_scale_attention(q, k, v, P, block=512):
    q, k, v = (np.asarray(a, float) for a in (q, k, v))
    n = q.shape[0]
    s = q @ k.T / q.shape[1]
    w = ta.taylor_poly(s, P) * (np.arange(n)[None, :] <= np.arange(n)[:, None])
    den = w.sum(1)
    return (w @ v) / den[:, None], den, np.abs(w).sum(1) / np.abs(den)


def _transposed_value_state(k, v, P):
    S = ta.state_ref(k, v, P)
    return S[:, ::-1].copy()


PINS = [check_counts, check_multiplicity, check_phi_identity, check_lagrange,
        check_special_cases, check_two_routes, check_softmax_library, check_convergence]


def _caught(mutant) -> bool:
    for pin in PINS:
        try:
            if not pin(mutant):
                return True
        except Exception:
            return True
    return False


@pytest.mark.parametrize("name,overrides", [
    ("dropped Taylor term", dict(taylor_poly=_poly_dropped_term)),
    ("wrong sign in the series", dict(taylor_poly=_poly_wrong_sign)),
    ("multiplicity left out", dict(multiplicity=_multiplicity_missing)),
    ("alpha_p left out of the weights", dict(feature_weights=_weights_no_alpha)),
    ("exclusive causal mask", dict(taylor_attention=_exclusive_mask_attention)),
    ("scale d_k instead of sqrt(d_k)", dict(taylor_attention=_wrong_scale_attention)),
    ("state columns permuted", dict(state_ref=_transposed_value_state)),
])
def test_mutants_are_caught(name, overrides):
    assert all(pin(ta) for pin in PINS)
    assert _caught(_Mutant(**overrides)), name
