"""GPU parity of the batched column-QP solve (optima_qp_solve_batched).

Both sides get the same fp32 Hessian values (formed by the oracle and rounded
to fp32) and the same step constant, so solver error is separated from Hessian
error. Bars: masks/zero pattern bit-exact; W within 1e-4 relative Frobenius of
the oracle; per-column objective (recomputed in fp64 by the oracle from each
returned W) within 1e-5 relative.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import (dev, to_dev, to_dev_x, gpu_layer_hessian, gpu_spectral, gpu_solve, rel_fro,
                      f32_exact, log)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


def _oracle_layer(cfg):
    chunks = (workloads.x_to_f64(workloads.x_chunk(cfg, c)) for c in range(cfg.n_chunks))
    H, _ = oracle.damp(oracle.hessian(chunks), cfg.rel_damp)
    H = f32_exact(H)
    W0 = workloads.w0(cfg)
    cs = workloads.col_sq_norms(cfg)
    M = workloads.layer_mask(cfg, W0, cs)
    lam, _ = oracle.power_iteration(H, workloads.power_start(cfg.d), 2000, 1e-9)
    lam = float(np.float32(lam))
    return H, W0, M, lam


def _assert_zero_pattern(W: np.ndarray, M: np.ndarray):
    assert W.dtype == np.float32
    assert np.all(W[M == 0].view(np.uint32) == 0), "pruned entries must be +0.0"


def _assert_w_and_f(H, W0, M, Wg, Wref, col_rel=1e-4, f_rel=1e-5, label=""):
    _assert_zero_pattern(Wg, M)
    r = rel_fro(Wg, Wref)
    fg = oracle.objective(H, W0, Wg)
    fr = oracle.objective(H, W0, Wref)
    fe = float(np.max(np.abs(fg - fr) / np.maximum(np.abs(fr), 1e-300)))
    log(f"  {label} W rel_fro={r:.3e}  max f rel={fe:.3e}")
    assert r <= col_rel
    assert fe <= f_rel


def _opts(L, **kw):
    return L.SolverOpts.default(**kw)


# Both arithmetic paths of the H-product must meet the same parity bar.
PRECISIONS = [pytest.param(0, id="fp32"), pytest.param(1, id="bf16x3")]


@pytest.mark.parametrize("prec", PRECISIONS)
def test_tiny_fixed_1000_matches_oracle_and_closed_form(L, prec):
    cfg = workloads.TINY
    H, W0, M, lam = _oracle_layer(cfg)
    o = oracle.rapdhg(H, W0, M, lam, oracle.SolverOptions(max_iters=1000, fixed_iters=True))
    ref = oracle.closed_form(H, W0, M)
    Wg, st, info = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                             _opts(L, max_iters=1000, fixed_iters=1, precision=prec))
    Wg = Wg.cpu().numpy()
    _assert_w_and_f(H, W0, M, Wg, o.W, label="vs oracle rapdhg")
    _assert_w_and_f(H, W0, M, Wg, ref, label="vs closed form")
    assert np.all(st["iters"] == 1000)
    assert info["iterations"] == 1000
    np.testing.assert_allclose(st["f_initial"], o.f_initial, rtol=1e-5)
    assert np.all(st["restarts"] > 0)


@pytest.mark.parametrize("prec", PRECISIONS)
@pytest.mark.parametrize("T", [1, 2, 7, 40, 63])
def test_trajectory_before_first_check(L, T, prec):
    # No check happens before iteration 64, so both sides follow the same
    # continuous map; only rounding separates them (fp32: 2^-24 per product;
    # bf16x3: up to 3 * 2^-16 per product).
    cfg = workloads.TINY
    H, W0, M, lam = _oracle_layer(cfg)
    o = oracle.rapdhg(H, W0, M, lam, oracle.SolverOptions(max_iters=T, fixed_iters=True))
    Wg, st, _ = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                          _opts(L, max_iters=T, fixed_iters=1, precision=prec))
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    per_col = np.linalg.norm(Wg - o.W, axis=1) / np.linalg.norm(o.W, axis=1)
    log(f"  T={T} worst column rel={per_col.max():.3e}")
    assert per_col.max() <= (1e-5 if prec == 0 else 1e-4)
    assert np.all(st["iters"] == T)


@pytest.mark.parametrize("prec", PRECISIONS)
@pytest.mark.parametrize("T", [8, 16, 24])
def test_restarts_and_final_kkt_match_oracle(L, T, prec):
    # Fixed mode with a check every 8 iterations: every check before T takes
    # restart decisions (PDLP-style decay tests and the monotone safeguard)
    # from the scores r_d, gap and KKT, and the final check reports the KKT of
    # the candidate. Per column the device's restart count must equal the
    # oracle's, and its final KKT must agree within a bound derived from the
    # arithmetic: with g = 2 H (x - w0),
    #   |dKKT| <= |d r_d| + |d gap| <= (1 + ||x||) ||dg|| + ||dx|| ||g||,
    #   ||dg|| <= 2 ||H||_2 ||dx|| + 2 eps (|| |H| |x| || + || |H| |w0| ||),
    # where dx is the measured difference of the two outputs (the trajectories
    # round differently) and eps the relative error of one H-product (fp32:
    # d 2^-24; bf16x3: 3 2^-16 plus that), doubled for the maintained sums.
    cfg = workloads.TINY
    H, W0, M, lam = _oracle_layer(cfg)
    o = oracle.rapdhg(H, W0, M, lam,
                      oracle.SolverOptions(max_iters=T, fixed_iters=True, check_every=8))
    Wg, st, _ = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                          _opts(L, max_iters=T, fixed_iters=1, check_every=8, precision=prec))
    Wg = Wg.cpu().numpy().astype(np.float64)
    d = cfg.d
    eps = d * 2.0 ** -24 + (3 * 2.0 ** -16 if prec == 1 else 0.0)
    absH = np.abs(H)
    hnorm = float(np.linalg.eigvalsh(H)[-1])
    dx = np.linalg.norm(Wg - o.W, axis=1)
    prod = np.linalg.norm(np.abs(o.W) @ absH, axis=1) + np.linalg.norm(np.abs(W0) @ absH, axis=1)
    dg = 2.0 * hnorm * dx + 4.0 * eps * prod
    g = 2.0 * (o.W - W0) @ H
    tol = (1.0 + np.linalg.norm(o.W, axis=1)) * dg + dx * np.linalg.norm(g, axis=1)
    err = np.abs(st["kkt_final"].astype(np.float64) - o.kkt_final)
    log(f"  T={T}: restarts {np.bincount(o.restarts)}; kkt_final max rel err "
        f"{np.max(err / o.kkt_final):.2e}, max err / bound {np.max(err / tol):.2e}")
    np.testing.assert_array_equal(st["restarts"], o.restarts)
    assert np.all(err <= tol + 2.0 ** -23 * o.kkt_final)
    assert np.all(st["iters"] == T)


def test_paper_mode_tiny(L):
    cfg = workloads.TINY
    H, W0, M, lam = _oracle_layer(cfg)
    o = oracle.rapdhg(H, W0, M, lam, oracle.SolverOptions())
    Wg, st, info = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M, _opts(L))
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    same = st["iters"] == o.iters
    log(f"  same stopping check on {same.mean():.2%} of columns; iters {np.unique(st['iters'])}")
    assert same.mean() >= 0.95
    assert st["converged"].all()
    _assert_w_and_f(H, W0[same], M[same], Wg[same], o.W[same], label="paper mode")


def test_full_pipeline_tiny(L):
    # Hessian, damping, spectral norm and solve all on the GPU vs the oracle's
    # own pipeline (fp64 throughout).
    cfg = workloads.TINY
    X = workloads.x_all(cfg)
    W0 = workloads.w0(cfg)
    M = workloads.layer_mask(cfg, W0, workloads.col_sq_norms(cfg, X))
    H, lamd = gpu_layer_hessian(L, to_dev_x(X), cfg.rel_damp)
    lm, _ = gpu_spectral(L, H, workloads.power_start(cfg.d))
    Wg, st, _ = gpu_solve(L, H, lm, W0, M, _opts(L, max_iters=1000, fixed_iters=1))
    Ho, _ = oracle.damp(oracle.hessian([X]), cfg.rel_damp)
    ref = oracle.closed_form(Ho, W0, M)
    _assert_w_and_f(Ho, W0, M, Wg.cpu().numpy(), ref, label="pipeline")


@pytest.mark.parametrize("prec", PRECISIONS)
def test_degenerate_masks_and_zero_iterations(L, prec):
    cfg = workloads.TINY
    H, W0, M, lam = _oracle_layer(cfg)
    Hd, lmd = to_dev(H), to_dev(np.array([lam]))
    ones = np.ones_like(M)
    Wg, st, info = gpu_solve(L, Hd, lmd, W0, ones,
                             _opts(L, eps_rel=1e-6, eps_abs=0.0, precision=prec))
    assert np.array_equal(Wg.cpu().numpy(), W0)
    assert np.all(st["iters"] == 0) and st["converged"].all() and info["iterations"] == 0
    Wg, st, _ = gpu_solve(L, Hd, lmd, W0, np.zeros_like(M),
                          _opts(L, eps_rel=1e-6, eps_abs=0.0, precision=prec))
    assert np.all(Wg.cpu().numpy().view(np.uint32) == 0) and np.all(st["iters"] == 0)
    Wg, st, _ = gpu_solve(L, Hd, lmd, W0, M, _opts(L, max_iters=0, precision=prec))
    np.testing.assert_array_equal(Wg.cpu().numpy(), np.where(M != 0, W0, 0.0).astype(np.float32))
    assert np.all(st["iters"] == 0)
    # A mix: some columns all-kept, some all-pruned, the rest masked.
    Mx = M.copy()
    Mx[::3] = 1
    Mx[1::3] = 0
    Wg, st, _ = gpu_solve(L, Hd, lmd, W0, Mx,
                          _opts(L, max_iters=1000, fixed_iters=1, precision=prec))
    Wg = Wg.cpu().numpy()
    # Fixed mode keeps iterating the all-kept columns, which sit at their
    # optimum: only the rounding of the products and of the averaging steps
    # may move them. bf16x3 products carry up to 3 * 2^-16 relative error per
    # term, so their drift stays within the W parity bar instead of fp32's.
    drift = 1e-5 if prec == 0 else 1e-4
    assert rel_fro(Wg[::3], W0[::3]) <= drift
    assert np.all(Wg[1::3].view(np.uint32) == 0)
    ref = oracle.closed_form(H, W0, Mx)
    _assert_w_and_f(H, W0[2::3], Mx[2::3], Wg[2::3], ref[2::3], label="mixed masks")


@pytest.mark.parametrize("prec", PRECISIONS)
def test_columns_are_independent(L, prec):
    # A column's result does not depend on the rest of the batch. The product
    # may split its contraction differently for different batch sizes, so
    # the agreement is up to fp32 rounding; runs with the same batch are
    # bitwise reproducible.
    cfg = workloads.TINY
    H, W0, M, lam = _oracle_layer(cfg)
    Hd, lmd = to_dev(H), to_dev(np.array([lam]))
    opts = _opts(L, max_iters=2000, fixed_iters=1, precision=prec)
    full, _, _ = gpu_solve(L, Hd, lmd, W0, M, opts)
    again, _, _ = gpu_solve(L, Hd, lmd, W0, M, opts)
    assert torch.equal(full, again)
    full = full.cpu().numpy()
    for sl in (slice(5, 6), slice(10, 30), slice(0, 64, 7)):
        part, _, _ = gpu_solve(L, Hd, lmd, W0[sl], M[sl], opts)
        assert rel_fro(part.cpu().numpy(), full[sl]) <= 1e-5


@pytest.mark.parametrize("prec", PRECISIONS)
def test_ragged_shapes_multi_tile(L, prec):
    # d not a multiple of the 128-wide tile, columns spanning several row
    # tiles with a ragged tail.
    rng = np.random.default_rng(5)
    for d, n in ((100, 3), (200, 130), (300, 257)):
        log(f"  ragged d={d} n={n}")
        X = rng.standard_normal((4 * d, d)).astype(np.float32)
        X[:, :3] *= 10
        H, _ = oracle.damp(oracle.hessian([X]), 0.01)
        H = f32_exact(H)
        W0 = (rng.standard_normal((n, d)) * 0.02).astype(np.float32)
        M = (rng.random((n, d)) < 0.5).astype(np.uint8)
        lam = float(np.float32(np.linalg.eigvalsh(H)[-1]))
        Wg, st, _ = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                              _opts(L, max_iters=3000, fixed_iters=1, precision=prec))
        _assert_w_and_f(H, W0, M, Wg.cpu().numpy(), oracle.closed_form(H, W0, M),
                        label=f"d={d} n={n}")


@pytest.fixture(scope="module")
def gpt2_layer():
    return _oracle_layer(workloads.GPT2_FC)


@pytest.mark.parametrize("prec", PRECISIONS)
def test_gpt2_shape_tight(L, gpt2_layer, prec):
    cfg = workloads.GPT2_FC
    log("gpt2 fc: oracle Hessian over the full token set")
    H, W0, M, lam = gpt2_layer
    Wg, st, info = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                             _opts(L, max_iters=4000, fixed_iters=1, precision=prec))
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    cols = np.arange(0, cfg.n_cols, cfg.n_cols // 96)
    ref = oracle.closed_form(H, W0[cols], M[cols])
    _assert_w_and_f(H, W0[cols], M[cols], Wg[cols], ref, label="gpt2 fc")


@pytest.fixture(scope="module")
def qproj_layer():
    return _oracle_layer(workloads.Q_PROJ.with_tokens(8 * 2048))


@pytest.mark.parametrize("prec", PRECISIONS)
def test_qproj_shape_tight(L, qproj_layer, prec):
    # The benchmark's launch shape (d = 4096, 4096 columns, 2:4 mask) on a
    # Hessian from 16384 tokens; 32 sampled columns against the closed form.
    cfg = workloads.Q_PROJ.with_tokens(8 * 2048)
    log("q_proj: oracle Hessian over 16384 tokens")
    H, W0, M, lam = qproj_layer
    Wg, st, info = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                             _opts(L, max_iters=5000, fixed_iters=1, precision=prec))
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    cols = np.arange(0, cfg.n_cols, cfg.n_cols // 32)
    ref = oracle.closed_form(H, W0[cols], M[cols])
    _assert_w_and_f(H, W0[cols], M[cols], Wg[cols], ref, label="q_proj")


def test_qproj_sparse_and_dense_paper_mode(L, qproj_layer):
    # The benchmark's solve (2:4 mask, paper tolerances) with the 2:4-sparse
    # iteration products and with the dense bf16x3 ones: the same stopping
    # check on nearly every column, all columns converged, and the results
    # within the W bar of each other.
    H, W0, M, lam = qproj_layer
    Hd, lmd = to_dev(H), to_dev(np.array([lam]))
    Ws, sts, infs = gpu_solve(L, Hd, lmd, W0, M, _opts(L))
    Wd, std, infd = gpu_solve(L, Hd, lmd, W0, M, _opts(L, sparse=0))
    assert infs["sparse_products"] == 1 and infd["sparse_products"] == 0
    Ws, Wd = Ws.cpu().numpy(), Wd.cpu().numpy()
    _assert_zero_pattern(Ws, M)
    same = sts["iters"] == std["iters"]
    log(f"  same stopping check on {same.mean():.2%} of columns; "
        f"iterations {np.unique(sts['iters'])}")
    assert same.mean() >= 0.95
    assert sts["converged"].all() and std["converged"].all()
    assert rel_fro(Ws[same], Wd[same]) <= 1e-4


def test_error_paths(L):
    cfg = workloads.TINY
    H, W0, M, lam = _oracle_layer(cfg)
    Hd, lmd = to_dev(H), to_dev(np.array([lam]))
    W0d, Md = to_dev(W0), to_dev(M, torch.uint8)
    out = torch.empty_like(W0d)
    # A non-finite H: scanned while the split planes are built (bf16x3) or
    # in a pass of its own (fp32).
    for prec in (L.PREC_FP32, L.PREC_BF16X3):
        for (i, j, v) in ((2, 5, float("inf")), (cfg.d - 1, cfg.d - 1, float("nan"))):
            Hn = Hd.clone()
            Hn[i, j] = v
            with pytest.raises(L.OptimaError) as e:
                L.optima_qp_solve_batched(Hn, lmd, W0d, Md, out, opts=_opts(L, precision=prec))
            assert e.value.status == -3
        # a width that needs padding: the scan runs with the padded copy
        rng = np.random.default_rng(5)
        A = rng.standard_normal((300, 100))
        Hr = to_dev(f32_exact(A.T @ A + np.eye(100)))
        Hr[99, 0] = float("nan")
        Wr = to_dev((rng.standard_normal((3, 100)) * 0.02).astype(np.float32))
        Mr = to_dev(np.ones((3, 100), dtype=np.uint8), torch.uint8)
        with pytest.raises(L.OptimaError) as e:
            L.optima_qp_solve_batched(Hr, lmd, Wr, Mr, torch.empty_like(Wr),
                                      opts=_opts(L, precision=prec))
        assert e.value.status == -3
    with pytest.raises(L.OptimaError) as e:
        L.optima_qp_solve_batched(Hd, torch.zeros_like(lmd), W0d, Md, out)
    assert e.value.status == -3
    with pytest.raises(L.OptimaError) as e:
        L.optima_qp_solve_batched(Hd, lmd, W0d, Md, out, opts=_opts(L, precision=7))
    assert e.value.status == -5
    small = torch.empty(16, dtype=torch.uint8, device=dev())
    with pytest.raises(L.OptimaError) as e:
        L.optima_qp_solve_batched(Hd, lmd, W0d, Md, out, ws=small)
    assert e.value.status == -4
    with pytest.raises(L.OptimaError) as e:
        L.optima_qp_solve_batched(Hd, lmd, W0d, Md, W0d)
    assert e.value.status == -1


@pytest.mark.parametrize("prec", PRECISIONS)
@pytest.mark.parametrize("n", [1, 5, 8, 9])
def test_few_columns_match_closed_form(L, prec, n):
    # At most 8 active columns take the HBM-streaming bf16x3 product (H's
    # planes read once per iteration; fp32 solves keep the MFMA tiles);
    # 9 take the tiles. Both reach the closed form; the columns of the
    # small batch agree with the same columns solved in a full batch.
    cfg = workloads.TINY
    H, W0, M, lam = _oracle_layer(cfg)
    Hd, lmd = to_dev(H), to_dev(np.array([lam]))
    opts = _opts(L, max_iters=1000, fixed_iters=1, precision=prec)
    Wg, st, _ = gpu_solve(L, Hd, lmd, W0[:n], M[:n], opts)
    Wg = Wg.cpu().numpy()
    _assert_w_and_f(H, W0[:n], M[:n], Wg, oracle.closed_form(H, W0[:n], M[:n]),
                    label=f"{n} columns")
    full, _, _ = gpu_solve(L, Hd, lmd, W0, M, opts)
    assert rel_fro(Wg, full.cpu().numpy()[:n]) <= 1e-5
