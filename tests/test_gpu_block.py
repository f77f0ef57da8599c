"""The streamed Llama-3-8B-shaped decoder block (four calibration streams,
seven matrices: q/k/v/o 4096 -> 4096/1024/1024/4096, gate/up 4096 -> 14336,
down 14336 -> 4096; 50 % unstructured masks), on 8192 tokens per stream.

Per stream: the device Hessian; per matrix: the device Wanda mask from the
undamped Hessian's diagonal (bit-exact against the oracle on the same values),
the CG solve against the closed form on sampled columns, and the paper-mode
rAPDHG solve (all columns converge, pruned entries +0.0, no column ends above
its start objective).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import dev, to_dev, to_dev_x, gpu_spectral, gpu_solve, log
from test_gpu_solver import _assert_w_and_f, _assert_zero_pattern

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


@pytest.mark.parametrize("stream", list(workloads.BLOCK_STREAMS))
def test_block_stream(L, stream):
    scfg = workloads.BLOCK_STREAMS[stream].with_tokens(4 * 2048)
    mats = [lc for lc, st in workloads.BLOCK_LAYERS if st == stream]
    d = scfg.d
    log(f"block stream {stream}: d={d}, matrices {[lc.name for lc in mats]}")
    X = workloads.x_all(scfg)
    H = torch.empty((d, d), dtype=torch.float32, device=dev())
    L.optima_hessian_accumulate(to_dev_x(X), H)
    diag = np.diag(H.cpu().numpy()).astype(np.float64)
    masks = {}
    for lc in mats:
        W0 = workloads.w0(lc)
        M = torch.empty((lc.n_cols, d), dtype=torch.uint8, device=dev())
        L.optima_wanda_mask(to_dev(W0), H, M, L.MASK_UNSTRUCTURED, lc.sparsity, col_sq_stride=d + 1)
        M = M.cpu().numpy()
        np.testing.assert_array_equal(M, oracle.wanda_mask(W0, diag, "unstructured", lc.sparsity))
        masks[lc.name] = (W0, M)
    lam = torch.empty(1, dtype=torch.float32, device=dev())
    L.optima_hessian_damp(H, scfg.rel_damp, lam)
    Hd = H.cpu().numpy().astype(np.float64)
    lm, _ = gpu_spectral(L, H, workloads.power_start_block(d, 16))
    for lc in mats:
        W0, M = masks[lc.name]
        Wc, st, _ = gpu_solve(L, H, None, W0, M, L.SolverOpts.default(
            method=L.METHOD_CG, max_iters=200, fixed_iters=1))
        Wc = Wc.cpu().numpy()
        _assert_zero_pattern(Wc, M)
        cols = np.linspace(0, lc.n_cols - 1, 4 if d > 8192 else 8).astype(int)
        _assert_w_and_f(Hd, W0[cols], M[cols], Wc[cols], oracle.closed_form(Hd, W0[cols], M[cols]),
                        label=f"{lc.name} cg")
        Wr, st, info = gpu_solve(L, H, lm, W0, M, L.SolverOpts.default())
        Wr = Wr.cpu().numpy()
        _assert_zero_pattern(Wr, M)
        assert st["converged"].all()
        assert np.all(st["f_final"] <= st["f_initial"] * (1 + 1e-6))
        log(f"  {lc.name}: paper-mode rAPDHG {info['iterations']} iterations")
