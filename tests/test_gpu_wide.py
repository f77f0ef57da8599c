"""GPU parity of the dense products on the 256 x 128 tile (d >= 8192).

Long contractions (d >= 8192, at least 256 active columns) run the dense
bf16x3 products on 256 x 128 tiles. d = 8192 with 300 columns gives two row
tiles, the second ragged, and a split of the contraction into two ranges
(partial sums plus the split epilogue), so every piece of that path runs.

H = B B^T / r + I with B an 8192 x 512 Gaussian matrix: symmetric positive
definite and cheap to form on the host.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import dev, to_dev, gpu_solve, rel_fro, f32_exact, log

pytestmark = pytest.mark.gpu

D, N_COLS, RANK = 8192, 300, 512


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


@pytest.fixture(scope="module")
def problem(L):
    rng = np.random.default_rng(81)
    B = rng.standard_normal((D, RANK))
    H = f32_exact(B @ B.T / RANK + np.eye(D))
    W0 = (rng.standard_normal((N_COLS, D)) * 0.02).astype(np.float32)
    score = np.abs(W0) * rng.uniform(0.5, 1.5, D)[None, :]
    keep = np.argsort(-score, axis=1, kind="stable")[:, :D // 2]
    M = np.zeros((N_COLS, D), dtype=np.uint8)
    np.put_along_axis(M, keep, 1, axis=1)
    Hd = to_dev(H)
    lm = torch.empty(1, dtype=torch.float32, device=dev())
    L.optima_spectral_lanczos(Hd, to_dev(rng.standard_normal(D).astype(np.float32)), lm)
    lam = float(lm.item())
    log(f"wide: lambda_max {lam:.6e} (above 1: the identity term)")
    assert lam > 1.0
    return H, Hd, lm, lam, W0, M


def test_wide_trajectory_matches_oracle(L, problem):
    # Ten iterations before any check: the iterates of the bf16x3 wide tile
    # against the oracle's fp64 ones.
    H, Hd, lm, lam, W0, M = problem
    T = 10
    Wg, st, info = gpu_solve(L, Hd, lm, W0, M,
                             L.SolverOpts.default(max_iters=T, fixed_iters=1, check_every=64,
                                                  precision=L.PREC_BF16X3))
    r = oracle.rapdhg(H, W0, M, lam, oracle.SolverOptions(max_iters=T, fixed_iters=True))
    Wg = Wg.cpu().numpy()
    assert np.all(Wg[M == 0].view(np.uint32) == 0)
    rel = rel_fro(Wg, r.W)
    per_col = max(rel_fro(Wg[j], r.W[j]) for j in range(0, N_COLS, 37))
    log(f"  T={T}: W rel_fro {rel:.3e}, worst sampled column {per_col:.3e}")
    assert rel <= 1e-5 and per_col <= 1e-5


def test_wide_tight_reaches_closed_form_and_fp32(L, problem):
    H, Hd, lm, lam, W0, M = problem
    opts = dict(max_iters=3000, fixed_iters=1)
    Wb, _, _ = gpu_solve(L, Hd, lm, W0, M, L.SolverOpts.default(precision=L.PREC_BF16X3, **opts))
    Wf, _, _ = gpu_solve(L, Hd, lm, W0, M, L.SolverOpts.default(precision=L.PREC_FP32, **opts))
    Wb, Wf = Wb.cpu().numpy(), Wf.cpu().numpy()
    # 32 columns spread over both row tiles, the ragged second one included.
    cols = np.unique(np.linspace(0, N_COLS - 1, 32).astype(int))
    assert cols.size == 32 and np.sum(cols >= 256) >= 4
    ref = oracle.closed_form(H, W0[cols], M[cols])
    fb = oracle.objective(H, W0[cols], Wb[cols])
    fr = oracle.objective(H, W0[cols], ref)
    log(f"  closed form: W rel_fro {rel_fro(Wb[cols], ref):.3e}, "
        f"f rel {np.max(np.abs(fb - fr) / fr):.3e}; bf16x3 vs fp32 {rel_fro(Wb, Wf):.3e}")
    assert rel_fro(Wb[cols], ref) <= 1e-4
    assert np.max(np.abs(fb - fr) / fr) <= 1e-5
    assert rel_fro(Wb, Wf) <= 1e-4
