"""GPU parity of the Hessian, damping and spectral-norm entry points.

Every case runs the HIP library through its C ABI and compares with the CPU
oracle on the same seeded inputs. Tolerances: fp32 accumulation of exact
products gives a relative Frobenius error well under 1e-5 for H; every entry
must lie within 2e-5 sqrt(H_ii H_jj) of the fp64 value.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import (dev, to_dev, to_dev_x, gpu_layer_hessian, gpu_spectral, rel_fro, f32_exact,
                      log)

pytestmark = pytest.mark.gpu

@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


def _check_h(Hg: np.ndarray, Ho: np.ndarray, rel=1e-5, ent=2e-5):
    assert np.array_equal(Hg, Hg.T), "H must be exactly symmetric"
    r = rel_fro(Hg, Ho)
    dg = np.sqrt(np.abs(np.outer(np.diag(Ho), np.diag(Ho))))
    worst = float(np.max(np.abs(Hg - Ho) / (dg + 1e-30)))
    log(f"  H rel_fro={r:.3e} worst_entry={worst:.3e}")
    assert r <= rel
    assert worst <= ent


@pytest.mark.parametrize("case", [
    ("tiny_f32", workloads.TINY, None),
    ("bf16_ragged", workloads.GPT2_FC, (3000, 200)),
    ("f32_ragged", workloads.TINY, (77, 5)),
    ("bf16_one_tile", workloads.Q_PROJ, (130, 128)),
    # bf16 with d % 256 == 0: token rows read in place (direct path)
    ("bf16_direct_one_tile_tail", workloads.Q_PROJ, (130, 256)),
    ("bf16_direct_tail_only", workloads.Q_PROJ, (50, 512)),
    ("bf16_direct_exact_stages", workloads.GPT2_FC, (640, 768)),
    ("bf16_direct_split", workloads.Q_PROJ, (8256, 1024)),
    # one tile over 100 full stages in 32 token splits of 3 or 4 stages (6 or 8
    # ring buffers: the unrolled body and its two-step remainder) plus a 37-row
    # tail (two buffers: the remainder alone)
    ("bf16_direct_ring_lengths", workloads.Q_PROJ, (6437, 256)),
])
def test_hessian_parity_small(L, case):
    name, cfg, shape = case
    log(f"hessian parity {name}")
    X = workloads.x_all(cfg.with_tokens(shape[0]) if shape else cfg)
    if shape:
        X = np.ascontiguousarray(X[:, :shape[1]])
    Xd = to_dev_x(X)
    H = torch.empty((X.shape[1], X.shape[1]), dtype=torch.float32, device=dev())
    L.optima_hessian_accumulate(Xd, H)
    Ho = oracle.hessian([workloads.x_to_f64(X)])
    _check_h(H.cpu().numpy().astype(np.float64), Ho)


def test_hessian_accumulate_in_sequences(L):
    # Section 3.4: per-sequence accumulation equals the stacked product.
    cfg = workloads.GPT2_FC.with_tokens(5 * 2048)
    X = workloads.x_all(cfg)[:, :300].copy()
    Xd = to_dev_x(X)
    H = torch.full((300, 300), 123.0, dtype=torch.float32, device=dev())
    for c in range(5):
        L.optima_hessian_accumulate(Xd[c * 2048:(c + 1) * 2048], H, accumulate=c > 0)
    Ho = oracle.hessian([workloads.x_to_f64(X[c * 2048:(c + 1) * 2048]) for c in range(5)])
    _check_h(H.cpu().numpy().astype(np.float64), Ho)
    H0 = torch.full((300, 300), 7.0, dtype=torch.float32, device=dev())
    L.optima_hessian_accumulate(Xd[:0], H0, accumulate=True)
    assert torch.all(H0 == 7.0)
    L.optima_hessian_accumulate(Xd[:0], H0, accumulate=False)
    assert torch.all(H0 == 0.0)


def test_hessian_direct_accumulate_in_sequences(L):
    # The direct path: sequences of 2048 tokens and a ragged 100-token one,
    # accumulated into an H that starts non-zero.
    cfg = workloads.Q_PROJ.with_tokens(3 * 2048)
    X = np.ascontiguousarray(workloads.x_all(cfg)[:, :512])
    X = np.concatenate([X, X[:100]])
    Xd = to_dev_x(X)
    H = torch.full((512, 512), 5.0, dtype=torch.float32, device=dev())
    bounds = [0, 2048, 4096, 6144, 6244]
    for c in range(4):
        L.optima_hessian_accumulate(Xd[bounds[c]:bounds[c + 1]], H, accumulate=True)
    Ho = oracle.hessian([workloads.x_to_f64(X[bounds[c]:bounds[c + 1]]) for c in range(4)])
    _check_h(H.cpu().numpy().astype(np.float64), Ho + 5.0)


def test_hessian_gpt2_full_size(L):
    cfg = workloads.GPT2_FC
    log("hessian gpt2 full size: generating X")
    X = workloads.x_all(cfg)
    Xd = to_dev_x(X)
    H = torch.empty((cfg.d, cfg.d), dtype=torch.float32, device=dev())
    L.optima_hessian_accumulate(Xd, H)
    torch.cuda.synchronize()
    log("  oracle")
    Ho = oracle.hessian(workloads.x_to_f64(X[c * cfg.chunk:(c + 1) * cfg.chunk])
                        for c in range(cfg.n_chunks))
    _check_h(H.cpu().numpy().astype(np.float64), Ho)


def test_hessian_qproj_full_size_sampled(L):
    # Full 262144 x 4096 bf16 layer in one call (the benchmark's launch);
    # the oracle forms the 256 x 256 block of H over a sample of features.
    cfg = workloads.Q_PROJ
    log("hessian q_proj full size: generating X")
    X = workloads.x_all(cfg)
    Xd = to_dev_x(X)
    H = torch.empty((cfg.d, cfg.d), dtype=torch.float32, device=dev())
    L.optima_hessian_accumulate(Xd, H)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    cols = np.sort(np.unique(np.concatenate([
        workloads.outlier_channels(cfg), rng.choice(cfg.d, 248, replace=False), [0, cfg.d - 1]])))
    log(f"  oracle on {cols.size} features")
    Ho = oracle.hessian(workloads.x_to_f64(X[c * cfg.chunk:(c + 1) * cfg.chunk][:, cols])
                        for c in range(cfg.n_chunks))
    Hg = H.cpu().numpy().astype(np.float64)
    assert np.array_equal(Hg, Hg.T)
    _check_h(Hg[np.ix_(cols, cols)], Ho)
    # The step size at the benchmark's shape: damping and the block-16
    # subspace iteration on the device's H, against LAPACK and the oracle's
    # subspace iteration on the same (fp32) matrix.
    lam = torch.empty(1, dtype=torch.float32, device=dev())
    L.optima_hessian_damp(H, cfg.rel_damp, lam)
    V0 = workloads.power_start_block(cfg.d, 16)
    lm, it = gpu_spectral(L, H, V0, max_iters=1000, tol=1e-6)
    Hd = H.cpu().numpy().astype(np.float64)
    top = np.linalg.eigvalsh(Hd)[-1]
    th_o, it_o = oracle.subspace_iteration(Hd, V0, 1000, 1e-6)
    lam_g = float(lm.item())
    log(f"  q_proj lambda_max gpu {lam_g:.8e} ({it} it) oracle {th_o:.8e} ({it_o} it) "
        f"eig {top:.8e}")
    assert lam_g == pytest.approx(top, rel=2e-6)
    assert lam_g == pytest.approx(th_o, rel=2e-6)
    assert abs(it - it_o) <= 1 and it <= 8


def test_damp_parity(L):
    cfg = workloads.TINY
    Ho, lam_o = oracle.damp(oracle.hessian([workloads.x_chunk(cfg, 0)]), 0.0)
    Hin = f32_exact(Ho)
    H = to_dev(Hin)
    lam = torch.empty(1, dtype=torch.float32, device=dev())
    L.optima_hessian_damp(H, 0.01, lam)
    Hd_o, lam_ref = oracle.damp(Hin, 0.01)
    assert float(lam.item()) == pytest.approx(lam_ref, rel=1e-6)
    Hg = H.cpu().numpy().astype(np.float64)
    np.testing.assert_array_equal(Hg - np.diag(np.diag(Hg)), Hin - np.diag(np.diag(Hin)))
    np.testing.assert_allclose(np.diag(Hg), np.diag(Hd_o), rtol=1e-7)
    # Non-finite trace: H untouched, lambda = NaN.
    Hn = to_dev(Hin)
    Hn[3, 3] = float("nan")
    L.optima_hessian_damp(Hn, 0.01, lam)
    assert torch.isnan(lam).item()
    assert float(Hn[4, 4].item()) == float(Hin[4, 4].astype(np.float32))


@pytest.mark.parametrize("block", [1, 16])
@pytest.mark.parametrize("cfg,tokens", [(workloads.TINY, None), (workloads.Q_PROJ, 4096),
                                        (workloads.GPT2_FC, 8192)])
def test_spectral_norm_parity(L, cfg, tokens, block):
    c = cfg.with_tokens(tokens) if tokens else cfg
    log(f"spectral {cfg.name} block {block}")
    Ho, _ = oracle.damp(oracle.hessian(workloads.x_to_f64(workloads.x_chunk(c, k))
                                       for k in range(c.n_chunks)), c.rel_damp)
    Hin = f32_exact(Ho)
    top = np.linalg.eigvalsh(Hin)[-1]
    if block == 1:
        v0 = workloads.power_start(c.d)
        lm, it = gpu_spectral(L, to_dev(Hin), v0, max_iters=1000, tol=1e-6)
        lam_o, it_o = oracle.power_iteration(Hin, v0, 1000, 1e-6)
        # The power iteration stops on a small change of rho, which may
        # still be short of lambda_max when the top eigenvalues cluster.
        near, rel = 1e-3, 1e-4
    else:
        V0 = workloads.power_start_block(c.d, block)
        lm, it = gpu_spectral(L, to_dev(Hin), V0, max_iters=1000, tol=1e-6)
        lam_o, it_o = oracle.subspace_iteration(Hin, V0, 1000, 1e-6)
        near, rel = 2e-6, 2e-6
        assert abs(it - it_o) <= 2
    lam_g = float(lm.item())
    log(f"  gpu {lam_g:.8e} ({it} it)  oracle {lam_o:.8e} ({it_o} it)  eig {top:.8e}")
    assert lam_g <= top * (1 + 1e-5)
    assert lam_g >= top * (1 - near)
    assert lam_g == pytest.approx(lam_o, rel=rel)


@pytest.mark.parametrize("d,block", [(100, 2), (100, 16), (200, 5), (8, 16), (1, 3)])
def test_spectral_block_shapes(L, d, block):
    # Ragged d (scalar loads when d % 4 != 0, padded row blocks), blocks wider
    # than the matrix (the extra directions are dependent and dropped).
    log(f"spectral shapes d={d} block={block}")
    rng = np.random.default_rng(d * 100 + block)
    A = rng.standard_normal((3 * d + 5, d))
    Hin = f32_exact(A.T @ A + 0.1 * np.eye(d))
    top = np.linalg.eigvalsh(Hin)[-1]
    V0 = rng.standard_normal((block, d)).astype(np.float32)
    lm, it = gpu_spectral(L, to_dev(Hin), V0, max_iters=500, tol=1e-6)
    lam_o, it_o = oracle.subspace_iteration(Hin, V0, 500, 1e-6)
    lam_g = float(lm.item())
    log(f"  gpu {lam_g:.8e} ({it} it) oracle {lam_o:.8e} ({it_o} it) eig {top:.8e}")
    assert lam_g == pytest.approx(top, rel=1e-5)
    assert lam_g == pytest.approx(lam_o, rel=1e-5)
    if block >= d:
        assert it == 2  # the block spans everything: the first Ritz value is exact


def test_spectral_block_clustered_top(L):
    # Eight top eigenvalues 2 % apart, far above the rest (outlier
    # channels): the block of 16 finishes in a few passes where the power
    # iteration needs hundreds.
    d = 512
    rng = np.random.default_rng(21)
    U, _ = np.linalg.qr(rng.standard_normal((d, d)))
    ev = np.concatenate([np.linspace(0.5, 1.0, d - 8), 100.0 * (1 - 0.02 * np.arange(8))])
    Hin = f32_exact((U * ev) @ U.T)
    top = np.linalg.eigvalsh(Hin)[-1]
    V0 = workloads.power_start_block(d, 16)
    lm, it = gpu_spectral(L, to_dev(Hin), V0, max_iters=1000, tol=1e-6)
    lm1, it1 = gpu_spectral(L, to_dev(Hin), V0[0], max_iters=1000, tol=1e-6)
    log(f"  block 16: {float(lm.item()):.8e} ({it} it); power: {float(lm1.item()):.8e} "
        f"({it1} it); eig {top:.8e}")
    assert float(lm.item()) == pytest.approx(top, rel=1e-6)
    assert it <= 6 and it1 >= 50


def test_spectral_degenerate(L):
    d = 64
    Z = to_dev(np.zeros((d, d), dtype=np.float32))
    V0 = workloads.power_start_block(d, 4)
    lm, it = gpu_spectral(L, Z, V0)
    assert float(lm.item()) == 0.0 and it == 1
    Hn = np.eye(d, dtype=np.float32)
    Hn[5, 7] = np.nan
    lm, it = gpu_spectral(L, to_dev(Hn), V0)
    assert np.isnan(float(lm.item()))
    # More start vectors than the library's maximum block: rejected by the
    # C entry point's validation.
    with pytest.raises(L.OptimaError) as e:
        gpu_spectral(L, Z, np.zeros((17, d), dtype=np.float32))
    assert e.value.status == -1
