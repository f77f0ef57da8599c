"""Pins of the shared diagonal (Jacobi) preconditioning in the oracle."""
import numpy as np
import pytest

import oracle
import workloads


def _layer():
    cfg = workloads.GPT2_FC.with_tokens(4096).with_cols(24)
    X = workloads.x_all(cfg)
    H, _ = oracle.damp(oracle.hessian([workloads.x_to_f64(X)]), cfg.rel_damp)
    W0 = workloads.w0(cfg).astype(np.float64)
    M = workloads.layer_mask(cfg, W0, np.diag(H))
    return H, W0, M


def test_unit_diagonal_and_symmetry():
    H, _, _ = _layer()
    Hs, D = oracle.jacobi_scale(H)
    np.testing.assert_allclose(np.diag(Hs), 1.0, rtol=1e-14)
    assert np.array_equal(Hs, Hs.T)
    np.testing.assert_allclose(Hs / np.outer(D, D), H, rtol=1e-14)


@pytest.mark.parametrize("solver", ["rapdhg", "cg"])
def test_scaled_solves_reach_the_original_closed_form(solver):
    # The scaled problem's optimum maps back to the original one (Eq. (10)-(11)
    # is invariant under w = D y); the solve runs on D H D and reports in the
    # original coordinates.
    H, W0, M = _layer()
    Hs, D = oracle.jacobi_scale(H)
    tight = oracle.SolverOptions(eps_rel=1e-11, eps_abs=0.0, max_iters=5000, check_every=8)
    if solver == "rapdhg":
        lam = np.linalg.eigvalsh(Hs)[-1]
        r = oracle.rapdhg(Hs, W0, M, lam, tight, scale=D)
    else:
        r = oracle.cg(Hs, W0, M, tight, scale=D)
    ref = oracle.closed_form(H, W0, M)
    assert np.linalg.norm(r.W - ref) / np.linalg.norm(ref) <= 1e-9
    assert np.all(r.W[M == 0] == 0.0)
    # Reported objectives are the original problem's.
    np.testing.assert_allclose(r.f_final, oracle.objective(H, W0, r.W), rtol=1e-9)
    np.testing.assert_allclose(r.f_initial, oracle.objective(H, W0, np.where(M, W0, 0.0)),
                               rtol=1e-12)


def test_unit_scale_changes_nothing():
    H, W0, M = _layer()
    lam = np.linalg.eigvalsh(H)[-1]
    o = oracle.SolverOptions(max_iters=200, fixed_iters=True)
    a = oracle.rapdhg(H, W0, M, lam, o)
    b = oracle.rapdhg(H, W0, M, lam, o, scale=np.ones(H.shape[0]))
    assert np.array_equal(a.W, b.W) and np.array_equal(a.kkt_final, b.kkt_final)
    c = oracle.cg(H, W0, M, o)
    e = oracle.cg(H, W0, M, o, scale=np.ones(H.shape[0]))
    assert np.array_equal(c.W, e.W)
