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

import oracle
import workloads
from gpu_util import dev, to_dev, to_dev_x, gpu_solve, rel_fro, log

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

    # The step size against the oracle's run of the method the policy took:
    # the block iteration where it converged within its passes, else Lanczos.
    if rep["method"] == "subspace":
        th, n_o = oracle.subspace_iteration(Hd, V0, BLOCK_PASSES, 1e-6)
        n_g = rep["block_passes"]
    else:
        th, n_o = oracle.lanczos(Hd, V0[0], 256, 1e-7)
        n_g = rep["lanczos_steps"]
    log(f"  lambda_max gpu {lam_g:.8e} ({rep['method']}, {n_g}) oracle {th:.8e} ({n_o})")
    assert lam_g == pytest.approx(th, rel=1e-5 if rep["method"] == "lanczos" else 2e-6)
    assert abs(n_g - n_o) <= 2

    # Every column converges, pruned entries are +0.0 and no column ends above
    # its start objective.
    Wg = Wg.cpu().numpy()
    assert st["converged"].all()
    assert np.all(Wg[M == 0].view(np.uint32) == 0)
    assert np.all(st["f_final"] <= st["f_initial"] * (1 + 1e-6))

    # Sampled columns: up to 8 from each stopping check, up to 32 of the longest.
    rng = np.random.default_rng(7)
    cols = []
    for k in np.unique(st["iters"]):
        idx = np.flatnonzero(st["iters"] == k)
        n = 32 if k == st["iters"].max() else 8
        cols.extend(int(c) for c in rng.choice(idx, min(n, idx.size), replace=False))
    cols = np.array(sorted(set(cols)))
    log(f"  checks {dict(zip(*np.unique(st['iters'], return_counts=True)))}; "
        f"{cols.size} sampled columns")
    r = oracle.rapdhg(Hd, W0[cols], M[cols], lam_g, oracle.SolverOptions())
    same = r.iters == st["iters"][cols]
    log(f"  same stopping check on {same.sum()}/{cols.size}")
    assert same.mean() >= 0.9
    assert r.converged.all()
    w_rel = rel_fro(Wg[cols][same], r.W[same])
    fg = oracle.objective(Hd, W0[cols], Wg[cols])[same]
    fo = oracle.objective(Hd, W0[cols], r.W)[same]
    f_rel = float(np.max(np.abs(fg - fo) / np.abs(fo)))
    log(f"  W rel_fro {w_rel:.3e}, max f rel {f_rel:.3e}")
    assert w_rel <= 1e-4
    assert f_rel <= 1e-5
