"""Pins of the oracle's Lanczos estimate of lambda_max (the solver's step size).

Each test checks the recurrence against something it does not compute itself:
the three-term recurrence of the discrete Chebyshev (Gram) polynomials, the
Rayleigh-Ritz value of an explicitly built Krylov basis, a hand-worked 2x2
case, LAPACK eigenvalues of matrices with known spectra, and the interlacing
bound of Ritz values.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _known_spectrum(d, ev, seed):
    U, _ = np.linalg.qr(np.random.default_rng(seed).standard_normal((d, d)))
    return (U * ev) @ U.T


def test_lanczos_gram_polynomial_recurrence():
    # With H = diag(1..n) and the all-ones start, Lanczos is the Stieltjes
    # procedure for the uniform weight on the nodes 1..n: its coefficients are
    # those of the discrete Chebyshev (Gram) polynomials,
    # alpha_j = (n+1)/2 and beta_j^2 = j^2 (n^2 - j^2) / (4 (4 j^2 - 1)).
    for n in (5, 12, 31):
        H = np.diag(np.arange(1.0, n + 1))
        th, steps, a, b = oracle.lanczos(H, np.ones(n), max_steps=n, tol=0.0, tridiagonal=True)
        j = np.arange(1.0, n)
        assert steps == n and a.shape == (n,) and b.shape == (n - 1,)
        np.testing.assert_allclose(a, (n + 1) / 2, rtol=0, atol=1e-12 * n)
        np.testing.assert_allclose(b ** 2, j ** 2 * (n ** 2 - j ** 2) / (4 * (4 * j ** 2 - 1)),
                                   rtol=1e-12)
        assert th == pytest.approx(n, rel=1e-13)


def test_lanczos_hand_worked_2x2():
    # H = [[4, 1], [1, 3]] from q_1 = e_1: alpha_1 = 4, w = H e_1 - 4 e_1 = e_2,
    # beta_1 = 1, alpha_2 = 3, so T_2 = H and theta_2 = (7 + sqrt 5) / 2.
    g = json.load(open(os.path.join(GOLDEN, "qp_2x2.json")))
    H = np.array(g["H"])
    th1, s1, a1, b1 = oracle.lanczos(H, np.array([2.0, 0.0]), max_steps=1, tol=0.0,
                                     tridiagonal=True)
    assert s1 == 1 and th1 == 4.0 and list(a1) == [4.0]
    th, s, a, b = oracle.lanczos(H, np.array([2.0, 0.0]), max_steps=2, tol=0.0, tridiagonal=True)
    assert s == 2 and list(a) == [4.0, 3.0] and list(b) == [1.0]
    assert th == pytest.approx(g["spectral"]["lambda_max"], rel=1e-15)


def test_lanczos_is_rayleigh_ritz_on_the_krylov_space():
    # theta_m is the largest eigenvalue of Q^T H Q for an orthonormal basis Q
    # of span{v, Hv, ..., H^(m-1) v}, here built from the powers directly.
    rng = np.random.default_rng(5)
    A = rng.standard_normal((11, 11))
    H = A @ A.T + 0.5 * np.eye(11)
    v = rng.standard_normal(11)
    for m in range(1, 7):
        K = np.stack([np.linalg.matrix_power(H, k) @ v for k in range(m)], axis=1)
        Q, _ = np.linalg.qr(K)
        ref = np.linalg.eigvalsh(Q.T @ H @ Q)[-1]
        th, steps = oracle.lanczos(H, v, max_steps=m, tol=0.0)
        assert steps == m
        assert th == pytest.approx(ref, rel=1e-12)


def test_lanczos_ritz_values_increase_and_stay_below_lambda_max():
    ev = np.concatenate([np.linspace(1.0, 2.0, 60), [2.05, 2.1]])
    H = _known_spectrum(62, ev, seed=8)
    v0 = np.random.default_rng(9).standard_normal(62)
    prev = -np.inf
    for m in range(1, 30):
        th, _ = oracle.lanczos(H, v0, max_steps=m, tol=0.0)
        assert th >= prev - 1e-13 * abs(th)
        assert th <= 2.1 * (1 + 1e-13)
        prev = th
    assert prev == pytest.approx(2.1, rel=1e-8)


def test_lanczos_breakdown_on_two_eigenvalues():
    # Two distinct eigenvalues: K_2 is invariant, beta_2 vanishes and theta_2
    # is the largest eigenvalue.
    ev = np.concatenate([np.full(20, 3.0), np.full(12, 7.0)])
    H = _known_spectrum(32, ev, seed=4)
    th, steps, a, b = oracle.lanczos(H, np.random.default_rng(2).standard_normal(32),
                                     max_steps=10, tol=0.0, tridiagonal=True)
    assert steps == 2 and b.shape == (1,)
    assert th == pytest.approx(7.0, rel=1e-13)
    # A multiple of the identity breaks down at the first step.
    th, steps = oracle.lanczos(2.5 * np.eye(9), np.arange(1.0, 10.0), max_steps=10, tol=0.0)
    assert steps == 1 and th == pytest.approx(2.5, rel=1e-15)


def test_lanczos_layers_against_lapack():
    for cfg, chunks in ((workloads.TINY, 1), (workloads.GPT2_FC, 2)):
        H, _ = oracle.damp(oracle.hessian([workloads.x_to_f64(workloads.x_chunk(cfg, c))
                                           for c in range(chunks)]), cfg.rel_damp)
        lam = np.linalg.eigvalsh(H)[-1]
        th, steps = oracle.lanczos(H, workloads.power_start(cfg.d), 256, 1e-12)
        assert th == pytest.approx(lam, rel=1e-10)
        assert th <= lam * (1 + 1e-13)
        assert steps < 256


def test_lanczos_beats_subspace_iteration_without_a_gap():
    # Evenly spread spectrum with no gap at the top: block-16 subspace
    # iteration converges as (lambda_17 / lambda_1)^k, Lanczos as a Chebyshev
    # polynomial of the step count.
    ev = np.linspace(1.0, 3.0, 400)
    H = _known_spectrum(400, ev, seed=21)
    th, steps = oracle.lanczos(H, workloads.power_start(400), 400, 1e-10)
    assert th == pytest.approx(3.0, rel=1e-6)
    sub, passes = oracle.subspace_iteration(H, workloads.power_start_block(400, 16), steps, 1e-10)
    assert passes == steps and abs(sub - 3.0) > 10 * abs(th - 3.0)


def test_lanczos_change_test_tolerance_without_a_gap():
    # Evenly spread spectrum: the Ritz value keeps rising by small amounts
    # long before it converges, so the change test at tol 1e-6 stops about
    # 1e-5 short of lambda_max, and tol 1e-7 (the step-size default) within
    # 1e-6 of it.
    d = 2048
    H = np.diag(np.linspace(1.0, 3.0, d))
    v0 = np.random.default_rng(5).standard_normal(d)
    th6, _ = oracle.lanczos(H, v0, 256, 1e-6)
    th7, _ = oracle.lanczos(H, v0, 256, 1e-7)
    assert (3.0 - th6) / 3.0 > 5e-6
    assert 0.0 <= (3.0 - th7) / 3.0 < 1e-6
