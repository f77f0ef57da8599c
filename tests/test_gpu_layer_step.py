"""Whole layer steps at full size, checked on sampled outputs.

q_proj is the step bench.py times. GPT-2 fc and down_proj run the same sequence on the dense
(non-2:4) products under 50 % and 60 % unstructured masks; down_proj's step size falls through
to Lanczos, and its products run on the 256 x 128 tile. The q_proj step is:
* H from all 262144 bf16 tokens (Student-t, 8 outlier channels);
* damping;
* the step size (block-16 iteration, Lanczos when that has not converged in 8 passes);
* the paper-mode rAPDHG solve of 4096 columns under the 2:4 Wanda mask, with the 2:4-sparse
  bf16x3 products.

The oracle cannot redo the whole layer in seconds. It takes the device's damped H (fp32 values,
copied back) and recomputes:
* the step size;
* the paper-mode solve of sampled columns, from the same H and lambda_max.

The sampled columns come from every stopping check: up to 8 from each, up to 32 from the last
(on q_proj that is every column of the few-column phase). Both sides must stop at the same check on nearly every sampled column and,
where they do, agree to the W and objective bars.
"""
import numpy as np
import pytest
import torch

import workloads
from gpu_util import (dev, to_dev, to_dev_x, gpu_solve, paper_mode_parity, check_step_size,
                      log)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


@pytest.mark.parametrize("CFG", [workloads.Q_PROJ, workloads.GPT2_FC, workloads.DOWN_PROJ],
                         ids=lambda c: c.name)
def test_full_step_sampled(L, CFG):
    from paper_2512_13886_amd.pipeline import BLOCK_PASSES, spectral_step_size
    log(f"{CFG.name} step: generating {CFG.n_tok} x {CFG.d} tokens")
    X = workloads.x_all(CFG)
    W0 = workloads.w0(CFG)
    M = workloads.layer_mask(CFG, W0, workloads.col_sq_norms(CFG, X))
    Xd = to_dev_x(X)
    del X
    H = torch.empty((CFG.d, CFG.d), dtype=torch.float32, device=dev())
    L.optima_hessian_accumulate(Xd, H)
    del Xd
    lam = torch.empty(1, dtype=torch.float32, device=dev())
    L.optima_hessian_damp(H, CFG.rel_damp, lam)
    V0 = workloads.power_start_block(CFG.d, 16)
    lm = torch.empty(1, dtype=torch.float32, device=dev())
    rep = spectral_step_size(H, to_dev(V0), lm)
    Wg, st, info = gpu_solve(L, H, lm, W0, M, L.SolverOpts.default())
    assert info["sparse_products"] == (1 if CFG.mask_kind == "2:4" else 0)
    Hd = H.cpu().numpy().astype(np.float64)
    del H
    lam_g = float(lm.item())

    check_step_size(Hd, V0, rep, lam_g, BLOCK_PASSES, label=CFG.name)

    # Every column converges, pruned entries are +0.0 and no column ends above
    # its start objective.
    Wg = Wg.cpu().numpy()
    assert st["converged"].all()
    assert np.all(Wg[M == 0].view(np.uint32) == 0)
    assert np.all(st["f_final"] <= st["f_initial"] * (1 + 1e-6))

    paper_mode_parity(Hd, W0, M, Wg, st, lam_g, label=CFG.name)
