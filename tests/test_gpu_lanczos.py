"""GPU parity of the Lanczos spectral-norm entry point (optima_spectral_lanczos).

The device keeps the Krylov basis in fp32 and every sum in fp64; the oracle
runs the same recurrence in fp64 on the same fp32 matrix. Ritz values from an
fp32 basis carry relative errors of a few 1e-7, so the per-step values must
agree within 2e-6 and the converged value lie within 1e-5 of LAPACK's
lambda_max (tol 1e-6 stops on the change of the Ritz value, not on its error).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import dev, to_dev, gpu_spectral, f32_exact, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


def gpu_lanczos(L, H: torch.Tensor, v0: np.ndarray, max_steps=256, tol=1e-6):
    lm = torch.empty(1, dtype=torch.float32, device=dev())
    st = torch.full((1,), -1, dtype=torch.int32, device=dev())
    L.optima_spectral_lanczos(H, to_dev(v0), lm, max_steps=max_steps, tol=tol, steps=st)
    torch.cuda.synchronize()
    return float(lm.item()), int(st.item())


def _layer_h(cfg, tokens):
    c = cfg.with_tokens(tokens) if tokens else cfg
    H, _ = oracle.damp(oracle.hessian(workloads.x_to_f64(workloads.x_chunk(c, k))
                                      for k in range(c.n_chunks)), c.rel_damp)
    return f32_exact(H)


@pytest.mark.parametrize("cfg,tokens", [(workloads.TINY, None), (workloads.GPT2_FC, 8192),
                                        (workloads.Q_PROJ, 4096)])
def test_lanczos_parity_layers(L, cfg, tokens):
    log(f"lanczos {cfg.name}")
    Hin = _layer_h(cfg, tokens)
    top = np.linalg.eigvalsh(Hin)[-1]
    v0 = workloads.power_start(cfg.d)
    lam_g, st_g = gpu_lanczos(L, to_dev(Hin), v0)
    lam_o, st_o = oracle.lanczos(Hin, v0, 256, 1e-6)
    log(f"  gpu {lam_g:.8e} ({st_g} steps) oracle {lam_o:.8e} ({st_o} steps) eig {top:.8e}")
    assert lam_g <= top * (1 + 2e-6)
    assert lam_g == pytest.approx(top, rel=1e-5)
    assert lam_g == pytest.approx(lam_o, rel=1e-5)
    assert abs(st_g - st_o) <= 2


@pytest.mark.parametrize("d", [64, 131, 1000])
def test_lanczos_trajectory_matches_oracle(L, d):
    # Fixed step counts (tol 0): the Ritz value after each of the first steps,
    # on ragged sizes (scalar loads when d % 4 != 0, partial row blocks).
    rng = np.random.default_rng(d)
    A = rng.standard_normal((2 * d + 3, d))
    Hin = f32_exact(A.T @ A + 0.05 * d * np.eye(d))
    v0 = rng.standard_normal(d).astype(np.float32)
    Hd = to_dev(Hin)
    for m in (1, 2, 3, 5, 8, 13):
        lam_g, st_g = gpu_lanczos(L, Hd, v0, max_steps=m, tol=0.0)
        lam_o, st_o = oracle.lanczos(Hin, v0, m, 0.0)
        log(f"  d={d} m={m}: gpu {lam_g:.9e} oracle {lam_o:.9e}")
        assert st_g == st_o == m
        assert lam_g == pytest.approx(lam_o, rel=2e-6)


def test_lanczos_gram_polynomial_matrix(L):
    # diag(1..n) from the all-ones start: the Ritz values are the largest
    # zeros of the discrete Chebyshev polynomials, and n steps span the
    # whole space (theta_n = n).
    n = 48
    Hin = np.diag(np.arange(1.0, n + 1)).astype(np.float32)
    v0 = np.ones(n, dtype=np.float32)
    for m in (1, 2, 4, 10, n):
        lam_g, st_g = gpu_lanczos(L, to_dev(Hin), v0, max_steps=m, tol=0.0)
        lam_o, _ = oracle.lanczos(Hin, v0, m, 0.0)
        log(f"  m={m}: gpu {lam_g:.9e} ({st_g}) oracle {lam_o:.9e}")
        assert lam_g == pytest.approx(lam_o, rel=2e-6)
    assert lam_g == pytest.approx(float(n), rel=1e-6)


def test_lanczos_breakdown_and_degenerate(L):
    d = 96
    rng = np.random.default_rng(4)
    U, _ = np.linalg.qr(rng.standard_normal((d, d)))
    ev = np.concatenate([np.full(60, 3.0), np.full(36, 7.0)])
    Hin = f32_exact((U * ev) @ U.T)
    v0 = rng.standard_normal(d).astype(np.float32)
    lam_g, st_g = gpu_lanczos(L, to_dev(Hin), v0, max_steps=20, tol=0.0)
    log(f"  two eigenvalues: {lam_g:.9e} ({st_g} steps)")
    assert st_g == 2  # beta_2 is at rounding level: the Krylov space is invariant
    assert lam_g == pytest.approx(7.0, rel=1e-6)
    # A multiple of the identity: beta_1 is at rounding level.
    lam_g, st_g = gpu_lanczos(L, to_dev(2.5 * np.eye(d, dtype=np.float32)), v0)
    assert st_g == 1 and lam_g == pytest.approx(2.5, rel=1e-7)
    # Zero matrix, zero start vector, NaN in H.
    Z = to_dev(np.zeros((d, d), dtype=np.float32))
    lam_g, st_g = gpu_lanczos(L, Z, v0)
    assert lam_g == 0.0 and st_g == 1
    lam_g, st_g = gpu_lanczos(L, to_dev(Hin), np.zeros(d, dtype=np.float32))
    assert lam_g == 0.0 and st_g == 0
    Hn = np.eye(d, dtype=np.float32)
    Hn[5, 7] = np.nan
    lam_g, _ = gpu_lanczos(L, to_dev(Hn), v0)
    assert np.isnan(lam_g)
    # 1 x 1 and more steps than rows.
    lam_g, st_g = gpu_lanczos(L, to_dev(np.array([[4.5]], dtype=np.float32)),
                              np.array([1.0], dtype=np.float32))
    assert lam_g == 4.5 and st_g == 1
    Hs = f32_exact(np.array([[4.0, 1.0], [1.0, 3.0]]))
    lam_g, st_g = gpu_lanczos(L, to_dev(Hs), np.array([2.0, 0.0], dtype=np.float32), tol=0.0)
    assert st_g == 2 and lam_g == pytest.approx((7 + np.sqrt(5)) / 2, rel=1e-7)


def test_lanczos_argument_errors(L):
    H = to_dev(np.eye(8, dtype=np.float32))
    lm = torch.empty(1, dtype=torch.float32, device=dev())
    for steps in (0, L.LANCZOS_MAX_STEPS + 1):
        with pytest.raises(L.OptimaError) as e:
            L.optima_spectral_lanczos(H, to_dev(np.ones(8)), lm, max_steps=steps)
        assert e.value.status == -1
    with pytest.raises(L.OptimaError) as e:
        L.optima_spectral_lanczos(H, to_dev(np.ones(8)), lm, tol=-1.0)
    assert e.value.status == -1
    small = torch.empty(16, dtype=torch.uint8, device=dev())
    with pytest.raises(L.OptimaError) as e:
        L.optima_spectral_lanczos(H, to_dev(np.ones(8)), lm, ws=small)
    assert e.value.status == -4


def test_lanczos_without_a_gap_needs_fewer_passes(L):
    # Evenly spread spectrum (no gap at the top), d = 2048. The Ritz value
    # creeps up by small amounts long before it has converged, so the change
    # test needs tol 1e-7 here (1e-6 stops about 3e-4 short); the block-16
    # subspace iteration at tol 1e-6 takes twice the passes and stops further
    # from lambda_max.
    d = 2048
    rng = np.random.default_rng(33)
    U, _ = np.linalg.qr(rng.standard_normal((d, d)))
    ev = np.linspace(1.0, 3.0, d)
    Hin = f32_exact((U * ev) @ U.T)
    top = np.linalg.eigvalsh(Hin)[-1]
    Hd = to_dev(Hin)
    lam_l, st_l = gpu_lanczos(L, Hd, workloads.power_start(d), tol=1e-7)
    lm, it_s = gpu_spectral(L, Hd, workloads.power_start_block(d, 16), max_iters=1000, tol=1e-6)
    lam_s = float(lm.item())
    log(f"  lanczos {lam_l:.8e} ({st_l} steps), subspace {lam_s:.8e} ({it_s} passes), "
        f"eig {top:.8e}")
    assert lam_l == pytest.approx(top, rel=1e-5)
    assert st_l < it_s
    assert 10 * abs(lam_l - top) < abs(lam_s - top)


def test_lanczos_maximum_steps_and_more_steps_than_rows(L):
    # 256 steps (the largest basis and coefficient arrays, the last
    # coefficient block of 64 waves): H = diag(1..2 evenly over 8192 values),
    # stored dense, whose top Ritz value is still rising at step 256.
    d = 8192
    Hin = np.diag(np.linspace(1.0, 2.0, d)).astype(np.float32)
    rng = np.random.default_rng(12)
    v0 = rng.standard_normal(d).astype(np.float32)
    lam_g, st_g = gpu_lanczos(L, to_dev(Hin), v0, max_steps=L.LANCZOS_MAX_STEPS, tol=0.0)
    lam_o, st_o = oracle.lanczos(Hin.astype(np.float64), v0, L.LANCZOS_MAX_STEPS, 0.0)
    log(f"  256 steps: gpu {lam_g:.9e} ({st_g}) oracle {lam_o:.9e} ({st_o})")
    assert st_g == st_o == L.LANCZOS_MAX_STEPS
    assert lam_g == pytest.approx(lam_o, rel=2e-6)
    assert 2.0 * (1 - 1e-5) < lam_g <= 2.0 * (1 + 1e-7)
    # max_steps above d: the run ends by d steps (the Krylov space is then the
    # whole space, or invariant earlier) at lambda_max.
    d = 40
    Hs = f32_exact((lambda A: A @ A.T + np.eye(d))(rng.standard_normal((d, d))))
    lam_g, st_g = gpu_lanczos(L, to_dev(Hs), rng.standard_normal(d).astype(np.float32),
                              max_steps=L.LANCZOS_MAX_STEPS, tol=0.0)
    log(f"  d=40: gpu {lam_g:.9e} ({st_g} steps)")
    assert st_g <= d
    assert lam_g == pytest.approx(np.linalg.eigvalsh(Hs)[-1], rel=2e-6)
