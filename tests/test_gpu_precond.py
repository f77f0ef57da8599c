"""GPU parity of the shared diagonal (Jacobi) preconditioning:
optima_hessian_jacobi and optima_qp_solve_batched with opts.col_scale.

The solver runs on D H D and reports in the original coordinates; parity is
against the oracle's scaled solvers on the same (device-scaled, fp32) matrix
and against the closed form of the original problem.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import dev, to_dev, gpu_spectral, gpu_solve, rel_fro, log
from test_gpu_solver import PRECISIONS, _oracle_layer, _assert_w_and_f, _assert_zero_pattern

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


def _scaled(L, H):
    """Device Jacobi scaling of the fp32 matrix H: (scaled H on the device,
    its fp64 copy, D on the device, D in fp64)."""
    Hd = to_dev(H)
    Dd = torch.empty(H.shape[0], dtype=torch.float32, device=dev())
    L.optima_hessian_jacobi(Hd, Dd)
    torch.cuda.synchronize()
    return Hd, Hd.cpu().numpy().astype(np.float64), Dd, Dd.cpu().numpy().astype(np.float64)


@pytest.fixture(scope="module")
def tiny():
    return _oracle_layer(workloads.TINY)


@pytest.fixture(scope="module")
def qproj_layer():
    return _oracle_layer(workloads.Q_PROJ.with_tokens(8 * 2048))


def test_jacobi_kernel(L, qproj_layer):
    H = qproj_layer[0]
    Hd, Hs, Dd, D = _scaled(L, H)
    Hs_o, D_o = oracle.jacobi_scale(H)
    np.testing.assert_allclose(D, D_o, rtol=6e-8)
    assert np.array_equal(Hs, Hs.T), "D H D must stay exactly symmetric"
    assert rel_fro(Hs, Hs_o) <= 3e-7
    np.testing.assert_allclose(np.diag(Hs), 1.0, rtol=3e-7)
    # Non-positive diagonal entries keep a unit scale.
    Z = np.eye(8)
    Z[3, 3] = 0.0
    Z[5, 5] = -2.0
    _, Zs, _, Dz = _scaled(L, Z)
    assert Dz[3] == 1.0 and Dz[5] == 1.0 and Zs[5, 5] == -2.0


@pytest.mark.parametrize("prec", PRECISIONS)
@pytest.mark.parametrize("T", [10, 200])
def test_scaled_rapdhg_trajectory(L, tiny, T, prec):
    H, W0, M, _ = tiny
    Hd, Hs, Dd, D = _scaled(L, H)
    lam = float(np.float32(np.linalg.eigvalsh(Hs)[-1]))
    opts = L.SolverOpts.default(max_iters=T, fixed_iters=1, precision=prec, col_scale=Dd)
    Wg, st, _ = gpu_solve(L, Hd, to_dev(np.array([lam])), W0, M, opts)
    ref = oracle.rapdhg(Hs, W0, M, lam, oracle.SolverOptions(max_iters=T, fixed_iters=True),
                        scale=D)
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    r = rel_fro(Wg, ref.W)
    log(f"  scaled rapdhg T={T}: W rel_fro vs oracle {r:.3e}")
    assert r <= (1e-5 if prec == 0 else 1e-4)
    np.testing.assert_allclose(st["f_final"], ref.f_final, rtol=1e-4)


@pytest.mark.parametrize("prec", PRECISIONS)
@pytest.mark.parametrize("method", ["rapdhg", "cg"])
def test_scaled_solves_reach_the_original_optimum(L, qproj_layer, method, prec):
    # q_proj shape (d = 4096, 2:4), H from 16384 tokens: after scaling, both
    # methods reach the original closed form in a few hundred iterations.
    cfg = workloads.Q_PROJ.with_tokens(8 * 2048)
    H, W0, M, _ = qproj_layer
    Hd, Hs, Dd, D = _scaled(L, H)
    if method == "rapdhg":
        lm, _ = gpu_spectral(L, Hd, workloads.power_start_block(cfg.d, 16))
        opts = L.SolverOpts.default(max_iters=600, fixed_iters=1, precision=prec, col_scale=Dd)
    else:
        lm = None
        opts = L.SolverOpts.default(method=L.METHOD_CG, max_iters=120, fixed_iters=1,
                                    precision=prec, col_scale=Dd)
    Wg, st, info = gpu_solve(L, Hd, lm, W0, M, opts)
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    cols = np.arange(0, cfg.n_cols, cfg.n_cols // 32)
    _assert_w_and_f(H, W0[cols], M[cols], Wg[cols], oracle.closed_form(H, W0[cols], M[cols]),
                    label=f"scaled {method} q_proj")


def test_scaling_cuts_paper_mode_iterations(L, qproj_layer):
    # Table 8 tolerances on the q_proj shape: the scaled solve stops earlier
    # and ends closer to the optimum.
    cfg = workloads.Q_PROJ.with_tokens(8 * 2048)
    H, W0, M, lam = qproj_layer
    lm0 = to_dev(np.array([lam]))
    Wp, sp, ip = gpu_solve(L, to_dev(H), lm0, W0, M, L.SolverOpts.default())
    Hd, Hs, Dd, D = _scaled(L, H)
    lm, _ = gpu_spectral(L, Hd, workloads.power_start_block(cfg.d, 16))
    Ws, ss, is_ = gpu_solve(L, Hd, lm, W0, M, L.SolverOpts.default(col_scale=Dd))
    cols = np.arange(0, cfg.n_cols, cfg.n_cols // 32)
    ref = oracle.closed_form(H, W0[cols], M[cols])
    ep = rel_fro(Wp.cpu().numpy()[cols], ref)
    es = rel_fro(Ws.cpu().numpy()[cols], ref)
    log(f"  paper mode: plain {ip['iterations']} iterations (W err {ep:.2e}), "
        f"scaled {is_['iterations']} iterations (W err {es:.2e})")
    assert is_["iterations"] <= ip["iterations"] and es < ep
    assert ss["converged"].all()


def test_scale_error_paths(L, tiny):
    H, W0, M, lam = tiny
    Hd, W0d, Md = to_dev(H), to_dev(W0), to_dev(M, torch.uint8)
    out = torch.empty_like(W0d)
    bad = torch.ones(H.shape[0], dtype=torch.float32, device=dev())
    bad[7] = 0.0
    with pytest.raises(L.OptimaError) as e:
        L.optima_qp_solve_batched(Hd, to_dev(np.array([lam])), W0d, Md, out,
                                  opts=L.SolverOpts.default(col_scale=bad))
    assert e.value.status == -3
    with pytest.raises(ValueError):
        L.optima_qp_solve_batched(Hd, to_dev(np.array([lam])), W0d, Md, out,
                                  opts=L.SolverOpts.default(col_scale=bad[:5]))
