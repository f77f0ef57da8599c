"""Helpers shared by the GPU tests: device upload of the seeded inputs and the
library pipeline (Hessian -> damping -> spectral norm -> solve) through the
C-ABI binding."""
from __future__ import annotations

import numpy as np
import torch

import workloads


def dev():
    return torch.device("cuda:0")


def to_dev_x(x_storage: np.ndarray) -> torch.Tensor:
    """X in storage form (fp32 values or bf16 bits) as a device tensor."""
    if x_storage.dtype == np.uint16:
        t = torch.from_numpy(x_storage.view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x_storage, dtype=np.float32))
    return t.to(dev())


def to_dev(a: np.ndarray, dtype=torch.float32) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev(), dtype=dtype)


def gpu_layer_hessian(lib, X_dev: torch.Tensor, rel_damp: float):
    d = X_dev.shape[1]
    H = torch.empty((d, d), dtype=torch.float32, device=dev())
    lib.optima_hessian_accumulate(X_dev, H, accumulate=False)
    lam = torch.empty(1, dtype=torch.float32, device=dev())
    lib.optima_hessian_damp(H, rel_damp, lam)
    return H, lam


def gpu_spectral(lib, H: torch.Tensor, v0: np.ndarray, max_iters=1000, tol=1e-6):
    lm = torch.empty(1, dtype=torch.float32, device=dev())
    it = torch.zeros(1, dtype=torch.int32, device=dev())
    lib.optima_spectral_norm(H, to_dev(v0), lm, max_iters=max_iters, tol=tol, iters=it)
    return lm, int(it.item())


def gpu_solve(lib, H: torch.Tensor, lm: torch.Tensor, W0: np.ndarray | torch.Tensor,
              mask: np.ndarray | torch.Tensor, opts):
    W0_d = W0 if isinstance(W0, torch.Tensor) else to_dev(W0)
    m_d = mask if isinstance(mask, torch.Tensor) else to_dev(mask, torch.uint8)
    n = W0_d.shape[0]
    W = torch.empty_like(W0_d)
    stats = {"iters": torch.zeros(n, dtype=torch.int32, device=dev()),
             "restarts": torch.zeros(n, dtype=torch.int32, device=dev()),
             "converged": torch.zeros(n, dtype=torch.uint8, device=dev()),
             "f_initial": torch.zeros(n, dtype=torch.float32, device=dev()),
             "f_final": torch.zeros(n, dtype=torch.float32, device=dev()),
             "kkt_final": torch.zeros(n, dtype=torch.float32, device=dev())}
    info = lib.optima_qp_solve_batched(H, lm, W0_d, m_d, W, opts=opts, stats=stats)
    torch.cuda.synchronize()
    return W, {k: v.cpu().numpy() for k, v in stats.items()}, info


def rel_fro(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def f32_exact(H64: np.ndarray) -> np.ndarray:
    """fp32 rounding of an oracle matrix, returned as fp64 values."""
    return H64.astype(np.float32).astype(np.float64)


def log(msg: str):
    print(msg, flush=True)


def paper_mode_parity(Hd: np.ndarray, W0: np.ndarray, M: np.ndarray, Wg: np.ndarray, st: dict,
                      lam: float, per_check: int = 8, last: int = 32, seed: int = 7,
                      label: str = "") -> None:
    """A paper-mode solve on the device against the oracle's on sampled columns.

    Samples up to `per_check` columns of every stopping check and up to `last`
    of the last one, solves them with the oracle from the same H (fp64 values
    of the device's fp32 matrix) and lambda_max, and requires the same stopping
    check on at least 90 % of them and, where it agrees, W within 1e-4
    (relative Frobenius) and every objective within 1e-5.
    """
    import oracle
    rng = np.random.default_rng(seed)
    cols = []
    for k in np.unique(st["iters"]):
        idx = np.flatnonzero(st["iters"] == k)
        n = last if k == st["iters"].max() else per_check
        cols.extend(int(c) for c in rng.choice(idx, min(n, idx.size), replace=False))
    cols = np.array(sorted(set(cols)))
    r = oracle.rapdhg(Hd, W0[cols], M[cols], lam, oracle.SolverOptions())
    same = r.iters == st["iters"][cols]
    w_rel = rel_fro(Wg[cols][same], r.W[same])
    fg = oracle.objective(Hd, W0[cols], Wg[cols])[same]
    fo = oracle.objective(Hd, W0[cols], r.W)[same]
    f_rel = float(np.max(np.abs(fg - fo) / np.abs(fo)))
    log(f"  {label}: checks {dict(zip(*np.unique(st['iters'], return_counts=True)))}; same check "
        f"on {same.sum()}/{cols.size} sampled; W rel_fro {w_rel:.3e}, max f rel {f_rel:.3e}")
    assert same.mean() >= 0.9
    assert r.converged.all()
    assert w_rel <= 1e-4
    assert f_rel <= 1e-5


def check_step_size(Hd: np.ndarray, V0: np.ndarray, rep: dict, lam: float, block_passes: int,
                    label: str = "") -> None:
    """lambda_max from the step-size policy against the oracle's run of the
    method the policy took (the block iteration where it converged within its
    passes, else Lanczos from the block's first vector)."""
    import oracle
    if rep["method"] == "subspace":
        th, n_o = oracle.subspace_iteration(Hd, V0, block_passes, 1e-6)
        n_g, rel = rep["block_passes"], 2e-6
    else:
        th, n_o = oracle.lanczos(Hd, V0[0], 256, 1e-7)
        n_g, rel = rep["lanczos_steps"], 1e-5
    log(f"  {label} lambda_max gpu {lam:.8e} ({rep['method']}, {n_g}) oracle {th:.8e} ({n_o})")
    assert abs(lam - th) <= rel * abs(th)
    assert abs(n_g - n_o) <= 2
