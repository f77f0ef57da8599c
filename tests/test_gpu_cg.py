"""GPU parity of the conjugate-gradient solve of the unconstrained form
(Eq. (7)-(11); optima_qp_solve_batched with method = OPTIMA_METHOD_CG).

Same bars as the rAPDHG solve: zero pattern bit-exact, W within 1e-4 relative
Frobenius of the oracle, per-column objective within 1e-5. Trajectories are
compared with oracle.cg after a fixed number of iterations; converged results
with the closed form of Eq. (10)-(11).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import dev, to_dev, gpu_solve, rel_fro, log
from test_gpu_solver import (PRECISIONS, _oracle_layer, _assert_w_and_f, _assert_zero_pattern)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


def _cg(L, **kw):
    return L.SolverOpts.default(method=L.METHOD_CG, **kw)


@pytest.fixture(scope="module")
def tiny():
    return _oracle_layer(workloads.TINY)


@pytest.mark.parametrize("prec", PRECISIONS)
@pytest.mark.parametrize("T", [1, 3, 10, 30])
def test_cg_trajectory_tiny(L, tiny, T, prec):
    H, W0, M, _ = tiny
    Wg, st, info = gpu_solve(L, to_dev(H), None, W0, M,
                             _cg(L, max_iters=T, fixed_iters=1, precision=prec))
    ref = oracle.cg(H, W0, M, oracle.SolverOptions(max_iters=T, fixed_iters=True)).W
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    r = rel_fro(Wg, ref)
    log(f"  cg T={T} prec={prec}: W rel_fro vs oracle cg {r:.3e}")
    assert r <= (1e-5 if prec == 0 else 1e-4)
    assert info["iterations"] == T and np.all(st["iters"][M.any(axis=1) & ~M.all(axis=1)] == T)


@pytest.mark.parametrize("prec", PRECISIONS)
def test_cg_tight_tiny(L, tiny, prec):
    H, W0, M, _ = tiny
    Wg, st, info = gpu_solve(L, to_dev(H), None, W0, M,
                             _cg(L, eps_rel=1e-7, eps_abs=0.0, check_every=8, max_iters=2000,
                                 precision=prec))
    _assert_w_and_f(H, W0, M, Wg.cpu().numpy(), oracle.closed_form(H, W0, M), label="cg tiny")
    log(f"  iterations {info['iterations']}, converged {st['converged'].mean():.2f}")
    assert info["iterations"] <= 200


@pytest.mark.parametrize("prec", PRECISIONS)
def test_cg_paper_mode_tiny(L, tiny, prec):
    # Table 8 tolerances, checked every 8 iterations: the stopping check and
    # the iterate agree with the oracle's CG.
    H, W0, M, _ = tiny
    Wg, st, _ = gpu_solve(L, to_dev(H), None, W0, M, _cg(L, check_every=8, precision=prec))
    ref = oracle.cg(H, W0, M, oracle.SolverOptions(check_every=8))
    same = np.mean(st["iters"] == ref.iters)
    log(f"  paper mode: same stopping check for {same:.3f} of the columns")
    assert same >= 0.95 and st["converged"].all()
    agree = st["iters"] == ref.iters
    assert rel_fro(Wg.cpu().numpy()[agree], ref.W[agree]) <= 1e-4


@pytest.fixture(scope="module")
def gpt2_layer():
    return _oracle_layer(workloads.GPT2_FC)


@pytest.mark.parametrize("prec", PRECISIONS)
def test_cg_gpt2_shape(L, gpt2_layer, prec):
    cfg = workloads.GPT2_FC
    H, W0, M, _ = gpt2_layer
    Wg, st, info = gpu_solve(L, to_dev(H), None, W0, M,
                             _cg(L, max_iters=600, fixed_iters=1, precision=prec))
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    cols = np.arange(0, cfg.n_cols, cfg.n_cols // 96)
    _assert_w_and_f(H, W0[cols], M[cols], Wg[cols], oracle.closed_form(H, W0[cols], M[cols]),
                    label="cg gpt2 fc")


@pytest.fixture(scope="module")
def qproj_layer():
    return _oracle_layer(workloads.Q_PROJ.with_tokens(8 * 2048))


@pytest.mark.parametrize("prec", PRECISIONS)
def test_cg_qproj_shape(L, qproj_layer, prec):
    cfg = workloads.Q_PROJ.with_tokens(8 * 2048)
    H, W0, M, _ = qproj_layer
    Wg, st, info = gpu_solve(L, to_dev(H), None, W0, M,
                             _cg(L, max_iters=300, fixed_iters=1, precision=prec))
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    cols = np.arange(0, cfg.n_cols, cfg.n_cols // 32)
    _assert_w_and_f(H, W0[cols], M[cols], Wg[cols], oracle.closed_form(H, W0[cols], M[cols]),
                    label="cg q_proj")


def test_cg_degenerate_masks(L, tiny):
    H, W0, M, _ = tiny
    Hd = to_dev(H)
    tight = dict(eps_rel=1e-7, eps_abs=0.0, check_every=8, max_iters=500)
    Wg, st, info = gpu_solve(L, Hd, None, W0, np.ones_like(M), _cg(L, **tight))
    assert np.array_equal(Wg.cpu().numpy(), W0) and np.all(st["iters"] == 0)
    Wg, st, _ = gpu_solve(L, Hd, None, W0, np.zeros_like(M), _cg(L, **tight))
    assert np.all(Wg.cpu().numpy().view(np.uint32) == 0)
    Mx = M.copy()
    Mx[::3] = 1
    Mx[1::3] = 0
    Wg, st, _ = gpu_solve(L, Hd, None, W0, Mx, _cg(L, **tight))
    Wg = Wg.cpu().numpy()
    assert np.array_equal(Wg[::3], W0[::3])
    assert np.all(Wg[1::3].view(np.uint32) == 0)
    _assert_w_and_f(H, W0[2::3], Mx[2::3], Wg[2::3], oracle.closed_form(H, W0, Mx)[2::3],
                    label="cg mixed masks")


def test_cg_error_paths(L, tiny):
    H, W0, M, lam = tiny
    Hd, W0d, Md = to_dev(H), to_dev(W0), to_dev(M, torch.uint8)
    out = torch.empty_like(W0d)
    with pytest.raises(L.OptimaError) as e:
        L.optima_qp_solve_batched(Hd, None, W0d, Md, out, opts=L.SolverOpts.default(method=7))
    assert e.value.status == -1
    # rAPDHG still needs the step size.
    with pytest.raises(L.OptimaError) as e:
        L.optima_qp_solve_batched(Hd, None, W0d, Md, out, opts=L.SolverOpts.default())
    assert e.value.status == -1
