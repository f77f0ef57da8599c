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
