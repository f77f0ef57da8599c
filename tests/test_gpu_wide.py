"""GPU parity of the dense products on the 256 x 128 tile.

Long contractions (d >= 8192, at least 256 active columns) and large batches
(d >= 4096, at least 4096 active columns) run the dense bf16x3 products on
256 x 128 tiles. d = 8192 with 300 columns gives two row tiles, the second
ragged, and a split of the contraction into two ranges (partial sums plus the
split epilogue), so every piece of that path runs. d = 4096 with 4396 columns
gives 18 row tiles, the last with 44 rows, and no split. d = 9216 with 256
columns runs three ranges of 96 stages: the three-buffer loop ends without a
remainder (the other shapes leave one or two stages).

H = B B^T / r + I with B a d x 512 Gaussian matrix: symmetric positive
definite and cheap to form on the host.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import dev, to_dev, gpu_solve, rel_fro, f32_exact, log

pytestmark = pytest.mark.gpu

RANK = 512
# (d, columns, seed)
SHAPES = {"long": (8192, 300, 81), "batch": (4096, 4396, 82), "split3": (9216, 256, 83)}


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


_PROBLEMS = {}


def _problem(L, shape):
    if shape not in _PROBLEMS:
        _PROBLEMS[shape] = _make_problem(L, shape)
    return _PROBLEMS[shape]


def _make_problem(L, shape):
    D, N_COLS, seed = SHAPES[shape]
    rng = np.random.default_rng(seed)
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
    log(f"wide {shape}: d {D}, {N_COLS} columns, lambda_max {lam:.6e} (above 1: the identity term)")
    assert lam > 1.0
    return H, Hd, lm, lam, W0, M


@pytest.fixture(scope="module")
def problem(L):
    return _problem(L, "long")


@pytest.mark.parametrize("shape", ["long", "batch", "split3"])
def test_wide_trajectory_matches_oracle(L, shape):
    # Ten iterations before any check: the iterates of the bf16x3 wide tile
    # against the oracle's fp64 ones. With fixed iterations the columns do not
    # interact, so past the first shape the oracle runs a sample of columns:
    # 32 spread over the batch and the last 8 (in the ragged last row tile).
    H, Hd, lm, lam, W0, M = _problem(L, shape)
    n_cols = W0.shape[0]
    T = 10
    Wg, st, info = gpu_solve(L, Hd, lm, W0, M,
                             L.SolverOpts.default(max_iters=T, fixed_iters=1, check_every=64,
                                                  precision=L.PREC_BF16X3))
    cols = (np.arange(n_cols) if shape == "long" else
            np.unique(np.concatenate([np.linspace(0, n_cols - 1, 32).astype(int),
                                      np.arange(n_cols - 8, n_cols)])))
    r = oracle.rapdhg(H, W0[cols], M[cols], lam,
                      oracle.SolverOptions(max_iters=T, fixed_iters=True))
    Wg = Wg.cpu().numpy()
    assert np.all(Wg[M == 0].view(np.uint32) == 0)
    rel = rel_fro(Wg[cols], r.W)
    per_col = max(rel_fro(Wg[j], r.W[i]) for i, j in enumerate(cols) if i % 7 == 0 or j >= n_cols - 8)
    log(f"  T={T}: W rel_fro {rel:.3e} over {cols.size} columns, worst checked column {per_col:.3e}")
    assert rel <= 1e-5 and per_col <= 1e-5


def test_wide_tight_reaches_closed_form_and_fp32(L, problem):
    H, Hd, lm, lam, W0, M = problem
    D, N_COLS, _ = SHAPES["long"]
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
