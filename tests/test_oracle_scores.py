"""Pins of the oracle's termination scores (Appendix D tolerances; Eq. (6)).

Every paper-mode stopping check and every restart is decided by r_d (the
norm of the gradient on the kept entries), the gap |z^T g|, KKT, the primal
and dual objectives P and D and the scale ||2 H w0||. These tests pin each of
them against something other than the oracle's own formulas: values worked by
hand on the 2 x 2 case (tests/golden/qp_2x2.json), finite differences of the
objective of Eq. (6), the Lagrangian dual function of Eq. (6) evaluated at
its own minimiser, and the flip of the termination decision exactly at the
hand-derived tolerance.
"""
import json
import os

import numpy as np
import pytest

import oracle
from oracle.optima_oracle import _score

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "qp_2x2.json")))


def _two_by_two(mask):
    H = np.array(GOLD["H"], dtype=np.float64)
    w0 = np.array(GOLD["w0"], dtype=np.float64)[None, :]
    keep = np.array(mask)[None, :] != 0
    return H, w0, keep


@pytest.mark.parametrize("key,mask", [("start_point_scores", GOLD["mask"]),
                                      ("start_point_scores_other_mask", [0, 1])])
def test_start_point_scores_match_hand_values(key, mask):
    gs = GOLD[key]
    H, w0, keep = _two_by_two(mask)
    x0 = np.where(keep, w0, 0.0)
    np.testing.assert_array_equal(x0[0], gs["x0"])
    s = _score(H, w0, keep, x0)
    assert s["rd"][0] == pytest.approx(gs["rd"], rel=1e-15)
    assert s["gap"][0] == pytest.approx(gs["gap"], rel=1e-15)
    assert s["f"][0] == pytest.approx(gs["P"], rel=1e-15)
    assert s["zHz"][0] == pytest.approx(gs["zHz"], rel=1e-15)
    assert s["kkt"][0] == pytest.approx(np.hypot(gs["rd"], gs["gap"]), rel=1e-15)
    if "kkt" in gs:
        assert s["kkt"][0] == pytest.approx(gs["kkt"], rel=1e-15)
    _, c_norm, w0Hw0 = oracle.anchor_terms(H, w0)
    assert c_norm[0] == pytest.approx(GOLD["start_point_scores"]["c_norm"], rel=1e-15)
    assert w0Hw0[0] == pytest.approx(GOLD["start_point_scores"]["w0Hw0"], rel=1e-15)
    _, P, D = oracle.termination(s, c_norm, w0Hw0, oracle.SolverOptions())
    assert P[0] == pytest.approx(gs["P"], rel=1e-15)
    assert D[0] == pytest.approx(gs["D"], rel=1e-15)


@pytest.mark.parametrize("key,mask", [("start_point_scores", GOLD["mask"]),
                                      ("start_point_scores_other_mask", [0, 1])])
@pytest.mark.parametrize("side", [-1, 1])
def test_start_point_stops_exactly_above_the_hand_threshold(key, mask, side):
    # With eps_abs = 0 the start point passes the test iff eps_rel reaches the
    # hand-derived threshold: 4/sqrt(340) where r_d binds, 1/3 where the gap
    # binds (that case fixes P and D). Checked on the decision function and
    # through a whole rapdhg run (a column that passes stops at iteration 0).
    gs = GOLD[key]
    eps = gs["eps_rel_threshold"] * (1.0 + side * 0.02)
    opts = oracle.SolverOptions(eps_rel=eps, eps_abs=0.0, max_iters=5000)
    H, w0, keep = _two_by_two(mask)
    x0 = np.where(keep, w0, 0.0)
    _, c_norm, w0Hw0 = oracle.anchor_terms(H, w0)
    conv, _, _ = oracle.termination(_score(H, w0, keep, x0), c_norm, w0Hw0, opts)
    assert bool(conv[0]) == (side > 0)
    lam = float(np.linalg.eigvalsh(H)[-1])
    r = oracle.rapdhg(H, w0, keep.astype(np.uint8), lam, opts)
    assert (r.iters[0] == 0) == (side > 0)
    assert r.converged[0]


def test_duality_at_the_two_by_two_optimum():
    gd = GOLD["duality_at_optimum"]
    H, w0, keep = _two_by_two(GOLD["mask"])
    w = oracle.closed_form(H, w0, keep.astype(np.uint8))
    np.testing.assert_allclose(w[0], gd["w_opt"], rtol=1e-15)
    s = _score(H, w0, keep, w)
    _, c_norm, w0Hw0 = oracle.anchor_terms(H, w0)
    _, P, D = oracle.termination(s, c_norm, w0Hw0, oracle.SolverOptions())
    assert s["zHz"][0] == pytest.approx(gd["zHz"], rel=1e-15)
    assert D[0] == pytest.approx(gd["D"], rel=1e-15)
    assert P[0] == pytest.approx(gd["D"], rel=1e-15)
    assert s["gap"][0] == pytest.approx(0.0, abs=1e-14)
    # q(lam) = -lam^2/11 - 2 lam by hand; its maximiser is g*_1.
    lam = np.linspace(-20.0, -2.0, 1801)
    q = -lam ** 2 / 11.0 - 2.0 * lam
    assert lam[np.argmax(q)] == pytest.approx(gd["lam_opt"], abs=1e-12)
    assert q.max() == pytest.approx(gd["q_opt"], rel=1e-15)


def _random_problem(seed, d=9, n=5):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((d, d))
    H = A @ A.T + 0.5 * np.eye(d)
    W0 = rng.standard_normal((n, d))
    keep = rng.random((n, d)) < 0.55
    keep[:, 0] = True
    keep[:, 1] = False
    Z = np.where(keep, rng.standard_normal((n, d)), 0.0)  # feasible points
    return H, W0, keep, Z


def _fd_gradient(H, w0, z, h=1e-3):
    """Central differences of the objective of Eq. (6) (exact up to rounding
    for a quadratic)."""
    d = z.size
    g = np.empty(d)
    for i in range(d):
        e = np.zeros(d)
        e[i] = h
        fp = oracle.objective(H, w0[None], (z + e)[None])[0]
        fm = oracle.objective(H, w0[None], (z - e)[None])[0]
        g[i] = (fp - fm) / (2.0 * h)
    return g


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_rd_gap_and_scale_from_finite_differences(seed):
    H, W0, keep, Z = _random_problem(seed)
    s = _score(H, W0, keep, Z)
    _, c_norm, _ = oracle.anchor_terms(H, W0)
    for j in range(W0.shape[0]):
        g = _fd_gradient(H, W0[j], Z[j])
        assert s["rd"][j] == pytest.approx(np.linalg.norm(g[keep[j]]), rel=1e-7)
        assert s["gap"][j] == pytest.approx(abs(Z[j] @ g), rel=1e-7, abs=1e-9)
        # ||2 H w0|| is the gradient's norm at w = 0.
        g0 = _fd_gradient(H, W0[j], np.zeros_like(Z[j]))
        assert c_norm[j] == pytest.approx(np.linalg.norm(g0), rel=1e-7)


def test_rd_with_a_scaling_is_the_original_gradient():
    # In the scaled coordinates y = D^-1 w (Hessian D H D, anchors D^-1 w0)
    # r_d is still the norm of the original problem's gradient on K.
    H, W0, keep, Z = _random_problem(4)
    Dg = np.exp(np.random.default_rng(8).standard_normal(H.shape[0]))
    Hs = H * np.outer(Dg, Dg)
    s = _score(Hs, W0 / Dg[None, :], keep, Z / Dg[None, :], Dg)
    _, c_norm, _ = oracle.anchor_terms(Hs, W0 / Dg[None, :], Dg)
    for j in range(W0.shape[0]):
        g = _fd_gradient(H, W0[j], Z[j])
        assert s["rd"][j] == pytest.approx(np.linalg.norm(g[keep[j]]), rel=1e-7)
        assert s["gap"][j] == pytest.approx(abs(Z[j] @ g), rel=1e-7, abs=1e-9)
        assert s["f"][j] == pytest.approx(oracle.objective(H, W0[j:j + 1], Z[j:j + 1])[0],
                                          rel=1e-12)
        g0 = _fd_gradient(H, W0[j], np.zeros_like(Z[j]))
        assert c_norm[j] == pytest.approx(np.linalg.norm(g0), rel=1e-7)


def _lagrangian_dual(H, w0, pruned, lam):
    """q(lam) = min over w of (w - w0)^T H (w - w0) - lam^T w_P, evaluated
    at the minimiser w = w0 + H^-1 E_P^T lam / 2 (stationarity of the
    Lagrangian of Eq. (6))."""
    d = w0.size
    E = np.zeros((pruned.size, d))
    E[np.arange(pruned.size), pruned] = 1.0
    w = w0 + 0.5 * np.linalg.solve(H, E.T @ lam)
    return oracle.objective(H, w0[None], w[None])[0] - lam @ w[pruned]


@pytest.mark.parametrize("seed", [5, 6])
def test_dual_objective_against_the_lagrangian_dual(seed):
    H, W0, keep, Z = _random_problem(seed)
    Wst = oracle.closed_form(H, W0, keep.astype(np.uint8))
    _, c_norm, w0Hw0 = oracle.anchor_terms(H, W0)
    s_opt = _score(H, W0, keep, Wst)
    _, P_opt, D_opt = oracle.termination(s_opt, c_norm, w0Hw0, oracle.SolverOptions())
    s_z = _score(H, W0, keep, Z)
    _, P_z, D_z = oracle.termination(s_z, c_norm, w0Hw0, oracle.SolverOptions())
    rng = np.random.default_rng(seed + 100)
    for j in range(W0.shape[0]):
        pruned = np.flatnonzero(~keep[j])
        g = _fd_gradient(H, W0[j], Wst[j])
        q_star = _lagrangian_dual(H, W0[j], pruned, g[pruned])
        # Strong duality at the optimum: P = D = q(lam*) = f*, zero gap.
        assert P_opt[j] == pytest.approx(q_star, rel=1e-8)
        assert D_opt[j] == pytest.approx(q_star, rel=1e-8)
        # Weak duality: any multipliers give a lower bound of every feasible P.
        for _ in range(5):
            lam = g[pruned] + rng.standard_normal(pruned.size)
            assert _lagrangian_dual(H, W0[j], pruned, lam) <= P_opt[j] * (1 + 1e-12)
        # At any feasible point the gap is |P - D|.
        assert s_z["gap"][j] == pytest.approx(abs(P_z[j] - D_z[j]), rel=1e-10)
