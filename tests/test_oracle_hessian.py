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
