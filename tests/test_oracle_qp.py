"""Pins of the oracle's column-QP functions (closed form, KKT, objective).

The closed form of Eq. (10)-(11) is checked against things other than itself:
exact rational arithmetic on the KKT system of Eq. (5)-(6), a dense LU solve of
the same system, a hand-worked 2x2 example, optimality under random feasible
perturbations, and special cases whose answer is known without solving.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _spd(rng, d, cond=10.0):
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    ev = np.geomspace(1.0, cond, d)
    return (Q * ev) @ Q.T


def _exact_kkt(H, w0, keep):
    """Solve [[2H, E^T], [E, 0]] [dw; nu] = [0; -w0_S] in exact rationals."""
    d = len(w0)
    S = [i for i in range(d) if not keep[i]]
    n = d + len(S)
    A = [[Fraction(0)] * (n + 1) for _ in range(n)]
    for i in range(d):
        for j in range(d):
            A[i][j] = 2 * Fraction(H[i][j])
    for r, i in enumerate(S):
        A[i][d + r] = Fraction(1)
        A[d + r][i] = Fraction(1)
        A[d + r][n] = -Fraction(w0[i])
    for c in range(n):  # Gauss-Jordan with exact pivots
        p = next(r for r in range(c, n) if A[r][c] != 0)
        A[c], A[p] = A[p], A[c]
        piv = A[c][c]
        A[c] = [v / piv for v in A[c]]
        for r in range(n):
            if r != c and A[r][c] != 0:
                f = A[r][c]
                A[r] = [a - f * b for a, b in zip(A[r], A[c])]
    dw = [A[i][n] for i in range(d)]
    return [Fraction(w0[i]) + dw[i] for i in range(d)]


def test_closed_form_matches_exact_rational_kkt():
    rng = np.random.default_rng(1)
    for d in (3, 4, 6):
        for _ in range(3):
            X = rng.integers(-3, 4, size=(d + 3, d)).astype(float)
            H = X.T @ X + np.eye(d)           # integer SPD matrix
            w0 = rng.integers(-5, 6, size=d).astype(float)
            keep = rng.integers(0, 2, size=d).astype(np.uint8)
            exact = _exact_kkt(H.astype(int).tolist(), w0.astype(int).tolist(), keep)
            W = oracle.closed_form(H, w0[None, :], keep[None, :])[0]
            np.testing.assert_allclose(W, [float(v) for v in exact], rtol=1e-12, atol=1e-12)


def test_closed_form_matches_dense_kkt_lu():
    rng = np.random.default_rng(2)
    for d in (2, 5, 9, 16):
        H = _spd(rng, d, cond=50.0)
        W0 = rng.standard_normal((7, d))
        M = (rng.random((7, d)) < 0.5).astype(np.uint8)
        M[0] = 1
        M[1] = 0
        a = oracle.closed_form(H, W0, M)
        b = oracle.kkt_solve(H, W0, M)
        np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)


def test_hand_worked_2x2():
    g = json.load(open(os.path.join(GOLDEN, "qp_2x2.json")))
    H = np.array(g["H"])
    w0 = np.array([g["w0"]])
    m = np.array([g["mask"]], dtype=np.uint8)
    W = oracle.closed_form(H, w0, m)
    np.testing.assert_allclose(W[0], g["closed_form"]["w"], rtol=0, atol=1e-15)
    assert oracle.objective(H, w0, W)[0] == pytest.approx(g["closed_form"]["f_opt"], rel=1e-15)
    x0 = np.where(m != 0, w0, 0.0)
    assert oracle.objective(H, w0, x0)[0] == pytest.approx(g["closed_form"]["f_initial"], rel=1e-15)


def test_objective_definition_on_small_integers():
    H = np.array([[2.0, -1.0, 0.0], [-1.0, 2.0, -1.0], [0.0, -1.0, 2.0]])
    W0 = np.array([[1.0, 2.0, 3.0]])
    W = np.array([[0.0, 2.0, 4.0]])
    # dw = [-1, 0, 1]; H dw = [-2, 0, 2]; dw . H dw = 4
    assert oracle.objective(H, W0, W)[0] == 4.0


def test_random_feasible_perturbations_never_lower_objective():
    rng = np.random.default_rng(3)
    d = 24
    H = _spd(rng, d, cond=1e3)
    W0 = rng.standard_normal((5, d))
    M = (rng.random((5, d)) < 0.5).astype(np.uint8)
    W = oracle.closed_form(H, W0, M)
    f = oracle.objective(H, W0, W)
    for _ in range(200):
        step = rng.standard_normal((5, d)) * 10.0 ** rng.uniform(-6, 0)
        step[M == 0] = 0.0
        assert np.all(oracle.objective(H, W0, W + step) >= f - 1e-12 * np.abs(f))


def test_special_cases():
    rng = np.random.default_rng(4)
    d = 12
    H = _spd(rng, d, cond=100.0)
    W0 = rng.standard_normal((4, d))
    ones = np.ones((4, d), np.uint8)
    zeros = np.zeros((4, d), np.uint8)
    np.testing.assert_array_equal(oracle.closed_form(H, W0, ones), W0)
    np.testing.assert_array_equal(oracle.closed_form(H, W0, zeros), np.zeros_like(W0))
    # Diagonal H decouples the entries: the update is plain zeroing (Wanda).
    Hd = np.diag(rng.uniform(1, 5, d))
    M = (rng.random((4, d)) < 0.5).astype(np.uint8)
    np.testing.assert_allclose(oracle.closed_form(Hd, W0, M), np.where(M != 0, W0, 0.0),
                               rtol=0, atol=1e-15)
    # Scaling W0 scales W; scaling H leaves W unchanged.
    W = oracle.closed_form(H, W0, M)
    np.testing.assert_allclose(oracle.closed_form(H, 3.0 * W0, M), 3.0 * W, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(oracle.closed_form(7.0 * H, W0, M), W, rtol=1e-12, atol=1e-13)
    # Consistent permutation of the inputs permutes the result.
    p = rng.permutation(d)
    Wp = oracle.closed_form(H[np.ix_(p, p)], W0[:, p], M[:, p])
    np.testing.assert_allclose(Wp, W[:, p], rtol=1e-12, atol=1e-13)
    # Columns are independent: solving a subset gives the same rows.
    np.testing.assert_array_equal(oracle.closed_form(H, W0[1:3], M[1:3]), W[1:3])


def test_pruned_entries_are_positive_zero():
    rng = np.random.default_rng(5)
    d = 10
    H = _spd(rng, d)
    W0 = -np.abs(rng.standard_normal((3, d)))   # negative weights: -0.0 would show
    M = (rng.random((3, d)) < 0.5).astype(np.uint8)
    for W in (oracle.closed_form(H, W0, M), oracle.kkt_solve(H, W0, M)):
        bits = W[M == 0].view(np.uint64)
        assert np.all(bits == 0)
