"""Pins of the oracle's Hessian, damping and power iteration."""
import json
import os

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hessian_matches_brute_force_loops():
    rng = np.random.default_rng(0)
    X = rng.integers(-4, 5, size=(13, 6)).astype(np.float32)
    H = oracle.hessian([X])
    n, d = X.shape
    for i in range(d):
        for j in range(d):
            s = 0
            for t in range(n):
                s += int(X[t, i]) * int(X[t, j])
            assert H[i, j] == s


def test_incremental_accumulation_equals_stacked_product():
    # Section 3.4: summing y_i^T y_i over sequences equals Y^T Y of the stack.
    rng = np.random.default_rng(1)
    X = rng.integers(-8, 9, size=(96, 10)).astype(np.float64)
    full = oracle.hessian([X])
    parts = oracle.hessian([X[:7], X[7:40], X[40:41], X[41:]])
    np.testing.assert_array_equal(full, parts)
    np.testing.assert_array_equal(full, full.T)
    assert np.linalg.eigvalsh(full).min() >= -1e-9


def test_hessian_of_bf16_storage_is_exact():
    cfg = workloads.GPT2_FC.with_tokens(64)
    bits = workloads.x_chunk(cfg, 0)[:, :16]
    x = workloads.x_to_f64(bits)
    H = oracle.hessian([x])
    # bf16 products are exact in fp64 and 64 of them are summed exactly.
    i, j = 3, 11
    ref = sum(float(a) * float(b) for a, b in zip(x[:, i], x[:, j]))
    assert H[i, j] == ref


def test_damping_closed_form():
    rng = np.random.default_rng(2)
    X = rng.standard_normal((50, 8))
    H = oracle.hessian([X])
    Hd, lam = oracle.damp(H, 0.01)
    tr = sum(H[i, i] for i in range(8))
    assert lam == pytest.approx(0.01 * tr / 8, rel=1e-15)
    np.testing.assert_array_equal(Hd - np.diag(np.diag(Hd)), H - np.diag(np.diag(H)))
    np.testing.assert_allclose(np.linalg.eigvalsh(Hd), np.linalg.eigvalsh(H) + lam, rtol=1e-12)


def test_power_iteration_against_lapack():
    rng = np.random.default_rng(3)
    Q, _ = np.linalg.qr(rng.standard_normal((40, 40)))
    ev = np.concatenate([np.linspace(1, 5, 39), [10.0]])
    H = (Q * ev) @ Q.T
    v0 = rng.standard_normal(40)
    lam, it = oracle.power_iteration(H, v0, max_iters=2000, tol=1e-14)
    assert lam == pytest.approx(np.linalg.eigvalsh(H)[-1], rel=1e-10)
    assert lam <= np.linalg.eigvalsh(H)[-1] * (1 + 1e-14)  # Rayleigh quotient bound


def test_power_iteration_eigenvector_start_and_golden():
    g = json.load(open(os.path.join(GOLDEN, "qp_2x2.json")))
    H = np.array(g["H"])
    w, V = np.linalg.eigh(H)
    lam, it = oracle.power_iteration(H, V[:, -1], max_iters=10, tol=1e-15)
    assert it == 2
    assert lam == pytest.approx(g["spectral"]["lambda_max"], rel=1e-14)
    lam2, _ = oracle.power_iteration(H, np.array([1.0, 0.3]), max_iters=500, tol=1e-15)
    assert lam2 == pytest.approx(g["spectral"]["lambda_max"], rel=1e-13)


def test_power_iteration_tiny_config():
    cfg = workloads.TINY
    H, _ = oracle.damp(oracle.hessian([workloads.x_chunk(cfg, 0)]), cfg.rel_damp)
    lam, it = oracle.power_iteration(H, workloads.power_start(cfg.d), 1000, 1e-12)
    assert lam == pytest.approx(np.linalg.eigvalsh(H)[-1], rel=1e-9)


def _known_spectrum(d, top, rest_lo, rest_hi, seed):
    rng = np.random.default_rng(seed)
    U, _ = np.linalg.qr(rng.standard_normal((d, d)))
    ev = np.concatenate([np.linspace(rest_lo, rest_hi, d - len(top)), top])
    return (U * ev) @ U.T, U, ev


def test_subspace_iteration_clustered_top_against_lapack():
    # Eight top eigenvalues within 1e-3 of each other (as outlier channels
    # make them), the rest in [0.5, 1]: the block of 16 captures the whole
    # cluster and converges in a few iterations; the plain power iteration
    # is still far off after 100.
    top = 10.0 - 1e-4 * np.arange(8)
    H, U, ev = _known_spectrum(96, top, 0.5, 1.0, seed=11)
    lam_max = np.linalg.eigvalsh(H)[-1]
    assert lam_max == pytest.approx(10.0, rel=1e-13)
    V0 = np.random.default_rng(12).standard_normal((16, 96))
    th, it = oracle.subspace_iteration(H, V0, max_iters=100, tol=1e-14)
    assert th == pytest.approx(lam_max, rel=1e-12)
    assert th <= lam_max * (1 + 1e-14)  # Ritz values never exceed lambda_max
    assert it <= 12
    rho, it1 = oracle.power_iteration(H, V0[0], max_iters=100, tol=1e-14)
    assert it1 == 100 and abs(rho - lam_max) > 1e-6 * lam_max


def test_subspace_iteration_block_one_is_power_iteration():
    cfg = workloads.TINY
    H, _ = oracle.damp(oracle.hessian([workloads.x_chunk(cfg, 0)]), cfg.rel_damp)
    v0 = workloads.power_start(cfg.d)
    for tol in (1e-6, 1e-12):
        a, ia = oracle.power_iteration(H, v0, 1000, tol)
        b, ib = oracle.subspace_iteration(H, v0[None, :], 1000, tol)
        assert ia == ib
        assert b == pytest.approx(a, rel=1e-13)


def test_subspace_iteration_golden_2x2_and_invariant_start():
    g = json.load(open(os.path.join(GOLDEN, "qp_2x2.json")))
    H = np.array(g["H"])
    # A block as wide as the matrix spans everything: the first Ritz value is
    # already lambda_max; the second iteration confirms it.
    th, it = oracle.subspace_iteration(H, np.array([[1.0, 0.0], [0.0, 1.0]]), 10, 1e-15)
    assert it == 2
    assert th == pytest.approx(g["spectral"]["lambda_max"], rel=1e-14)
    # Starting on the invariant subspace of the top 4 eigenvectors.
    Hk, U, ev = _known_spectrum(40, np.array([7.0, 6.0, 5.0, 4.0]), 1.0, 2.0, seed=3)
    th, it = oracle.subspace_iteration(Hk, U[:, -4:].T, 10, 1e-15)
    assert it == 2 and th == pytest.approx(7.0, rel=1e-13)


def test_subspace_iteration_layers_and_zero():
    for cfg, chunks in ((workloads.TINY, 1), (workloads.GPT2_FC, 2)):
        H, _ = oracle.damp(oracle.hessian([workloads.x_to_f64(workloads.x_chunk(cfg, c))
                                           for c in range(chunks)]), cfg.rel_damp)
        th, it = oracle.subspace_iteration(H, workloads.power_start_block(cfg.d, 16),
                                           1000, 1e-12)
        lam = np.linalg.eigvalsh(H)[-1]
        assert th == pytest.approx(lam, rel=1e-10)
        assert th <= lam * (1 + 1e-13)
    th, it = oracle.subspace_iteration(np.zeros((8, 8)), np.ones((3, 8)), 10, 1e-6)
    assert th == 0.0 and it == 1


def test_power_start_block_rows():
    B = workloads.power_start_block(100, 4)
    assert B.shape == (4, 100) and B.dtype == np.float32
    np.testing.assert_array_equal(B[0], workloads.power_start(100))
    assert np.linalg.matrix_rank(B.astype(np.float64)) == 4
