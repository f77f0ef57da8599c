"""Pins of the oracle's conjugate-gradient solve of the unconstrained form
(Eq. (7)-(11)): H_KK x_K = (H w0)_K per column."""
import json
import os

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _spd(d, seed, cond=50.0):
    rng = np.random.default_rng(seed)
    U, _ = np.linalg.qr(rng.standard_normal((d, d)))
    return (U * np.geomspace(1.0, cond, d)) @ U.T


def test_finite_termination_reaches_the_closed_form():
    # In exact arithmetic CG solves an s x s system in at most s steps; in
    # fp64 on a well-conditioned 12 x 12 system that is exact to ~1e-12.
    d = 12
    H = _spd(d, 1)
    rng = np.random.default_rng(2)
    W0 = rng.standard_normal((9, d))
    M = (rng.random((9, d)) < 0.6).astype(np.uint8)
    M[0] = 1
    M[1] = 0
    r = oracle.cg(H, W0, M, oracle.SolverOptions(max_iters=d, fixed_iters=True))
    ref = oracle.closed_form(H, W0, M)
    np.testing.assert_allclose(r.W, ref, rtol=0, atol=1e-10 * np.abs(ref).max())
    assert np.all(r.W[M == 0] == 0.0)


def test_golden_2x2_is_solved_in_one_step():
    # One kept entry: the system is 1 x 1 and the first CG step is exact.
    g = json.load(open(os.path.join(GOLDEN, "qp_2x2.json")))
    H, w0, m = np.array(g["H"]), np.array(g["w0"]), np.array(g["mask"], dtype=np.uint8)
    r = oracle.cg(H, w0[None, :], m[None, :], oracle.SolverOptions(max_iters=1, fixed_iters=True))
    np.testing.assert_allclose(r.W[0], g["closed_form"]["w"], rtol=1e-15, atol=1e-15)
    assert r.f_final[0] == pytest.approx(g["closed_form"]["f_opt"], rel=1e-14)


def test_directions_are_conjugate_and_the_energy_error_falls():
    d = 30
    H = _spd(d, 3, cond=1e3)
    rng = np.random.default_rng(4)
    W0 = rng.standard_normal((1, d))
    M = (rng.random((1, d)) < 0.7).astype(np.uint8)
    K = np.flatnonzero(M[0])
    x_star = oracle.closed_form(H, W0, M)[0]
    ps, errs = [], []

    def obs(t, x, p):
        ps.append(p[0].copy())
        e = x[0] - x_star
        errs.append(float(e @ H @ e))

    oracle.cg(H, W0, M, oracle.SolverOptions(max_iters=8, fixed_iters=True), observer=obs)
    A = H[np.ix_(K, K)]
    P = np.array([p[K] for p in ps[:-1]])
    G = P @ A @ P.T
    off = G - np.diag(np.diag(G))
    assert np.max(np.abs(off)) <= 1e-9 * np.max(np.abs(np.diag(G)))
    assert all(b <= a * (1 + 1e-12) for a, b in zip(errs, errs[1:]))


def test_degenerate_masks_and_tight_mode():
    cfg = workloads.TINY
    H, _ = oracle.damp(oracle.hessian([workloads.x_chunk(cfg, 0)]), cfg.rel_damp)
    W0 = workloads.w0(cfg)
    M = workloads.layer_mask(cfg, W0, np.diag(H))
    tight = oracle.SolverOptions(eps_rel=1e-12, eps_abs=0.0, check_every=8, max_iters=2000)
    r = oracle.cg(H, W0, np.ones_like(M), tight)
    assert np.array_equal(r.W, W0) and np.all(r.iters == 0) and r.converged.all()
    r = oracle.cg(H, W0, np.zeros_like(M), tight)
    assert np.all(r.W == 0.0) and np.all(r.iters == 0)
    r = oracle.cg(H, W0, M, tight)
    ref = oracle.closed_form(H, W0, M)
    assert np.linalg.norm(r.W - ref) / np.linalg.norm(ref) <= 1e-10
    assert r.converged.all() and r.iters.max() <= 64
