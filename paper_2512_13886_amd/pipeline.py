"""The layer loop of Algorithm 1 over a chain of linear layers.

For every layer, in order, on the device through the C ABI:
  1. H = X^T X over the calibration tokens X (the layer's inputs, already the
     outputs of the pruned layers before it);
  2. the Wanda mask from the undamped diagonal of H;
  3. damping, the step size (spectral_step_size below) and the batched
     column QPs (paper tolerances unless `opts` says otherwise);
  4. the skip rule of Appendix D, read as: more than half of the columns
     unconverged, or sum f_final > sum f_initial. A skipped layer keeps the
     mask-only (Wanda) weights;
  5. the layer-wise error of Section 4: the squared output error against the
     dense layer, of the kept weights and of Wanda's;
  6. X <- bf16(act(X W^T)) with the kept weights, the next layer's inputs.

This module only sequences library calls and allocates with torch; every step
above runs in the HIP kernels. The skip decision is host logic on the
per-column statistics the solve returns.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable

import torch

from . import _lib as L


@dataclass
class LayerReport:
    d_in: int
    d_out: int
    iterations: int
    converged: int
    skipped: bool
    err_kept: float       # sum of squared output errors of the kept weights vs dense
    err_wanda: float      # the same for the mask-only weights
    ms: dict = field(default_factory=dict)
    # per-column statistics of the solve (host arrays): iters, converged,
    # f_initial, f_final
    columns: dict = field(default_factory=dict)

    @property
    def error_ratio(self) -> float:
        """MSE(Y_kept, Y_dense) / MSE(Y_wanda, Y_dense) (Section 4)."""
        return self.err_kept / self.err_wanda if self.err_wanda > 0 else float("nan")


# Passes of the block iteration before the step size falls back to Lanczos.
BLOCK_PASSES = 8


def spectral_step_size(H: torch.Tensor, V0: torch.Tensor, lambda_max: torch.Tensor,
                       block_passes: int = BLOCK_PASSES, tol_block: float = 1e-6,
                       tol_lanczos: float = 1e-7) -> dict:
    """lambda_max(H) for the solver's step size, into lambda_max (device).

    Outlier channels put a cluster of eigenvalues far above the rest; the
    block subspace iteration from the start block V0 [b, d] captures it and
    converges in a handful of passes. Without such a gap (near-isotropic
    inputs, or H after diagonal scaling) it crawls, and the Lanczos process
    from V0[0] gets there in far fewer passes over H. So: at most
    `block_passes` block passes, then Lanczos if they did not converge.
    Returns {"method", "block_passes", "lanczos_steps"}.
    """
    it = torch.zeros(1, dtype=torch.int32, device=H.device)
    L.optima_spectral_norm(H, V0, lambda_max, max_iters=block_passes, tol=tol_block, iters=it)
    passes = int(it.item())
    rep = {"method": "subspace", "block_passes": passes, "lanczos_steps": 0}
    if passes >= block_passes:
        st = torch.zeros(1, dtype=torch.int32, device=H.device)
        v0 = V0[0] if V0.dim() == 2 else V0
        L.optima_spectral_lanczos(H, v0.contiguous(), lambda_max, tol=tol_lanczos, steps=st)
        rep.update(method="lanczos", lanczos_steps=int(st.item()))
    return rep


def skip_layer(converged: torch.Tensor, f_initial: torch.Tensor, f_final: torch.Tensor) -> bool:
    """Appendix D's skip rule on the statistics of one layer's solve."""
    conv = converged.cpu().numpy() != 0
    n = conv.size
    f0 = f_initial.cpu().double().sum().item()
    f1 = f_final.cpu().double().sum().item()
    return bool(n and ((n - int(conv.sum())) * 2 > n or f1 > f0))


def prune_chain(X0: torch.Tensor, weights: list, start: Callable[[int], torch.Tensor],
                sparsity: float = 0.5, rel_damp: float = 0.01, act: int = L.ACT_SILU,
                opts: L.SolverOpts | None = None, timed: bool = False):
    """Algorithm 1 over a chain of layers.

    X0: bfloat16 [n_tok, d_0] calibration inputs of the first layer.
    weights: float32 [d_{l+1}, d_l] dense weights, layer by layer.
    start: d -> float32 [block, d] start vectors of the step-size iteration.
    Returns (kept weights, masks, reports, activations after the last layer);
    the masks are the updated masks of Algorithm 1, unchanged by the update.
    """
    X = X0
    dev = X0.device
    out_w, out_m, reports = [], [], []
    for W0 in weights:
        d_out, d_in = W0.shape
        if X.shape[1] != d_in:
            raise ValueError("layer widths do not chain")
        n_tok = X.shape[0]
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)] if timed else None
        if timed:
            ev[0].record()
        H = torch.empty((d_in, d_in), dtype=torch.float32, device=dev)
        L.optima_hessian_accumulate(X, H)
        M = torch.empty((d_out, d_in), dtype=torch.uint8, device=dev)
        L.optima_wanda_mask(W0, H, M, L.MASK_UNSTRUCTURED, sparsity, col_sq_stride=d_in + 1)
        lam = torch.empty(1, dtype=torch.float32, device=dev)
        L.optima_hessian_damp(H, rel_damp, lam)
        lmax = torch.empty(1, dtype=torch.float32, device=dev)
        spectral_step_size(H, start(d_in), lmax)
        if timed:
            ev[1].record()
        W = torch.empty_like(W0)
        stats = {"iters": torch.zeros(d_out, dtype=torch.int32, device=dev),
                 "converged": torch.zeros(d_out, dtype=torch.uint8, device=dev),
                 "f_initial": torch.zeros(d_out, dtype=torch.float32, device=dev),
                 "f_final": torch.zeros(d_out, dtype=torch.float32, device=dev)}
        ws = torch.empty(L.optima_qp_workspace_bytes(d_in, d_out), dtype=torch.uint8, device=dev)
        info = L.optima_qp_solve_batched(H, lmax, W0, M, W, opts=opts, ws=ws, stats=stats)
        if timed:
            ev[2].record()
        skipped = skip_layer(stats["converged"], stats["f_initial"], stats["f_final"])
        # The mask-only weights sel(M, W0, +0): the solve's start point.
        W_wanda = torch.empty_like(W0)
        L.optima_qp_solve_batched(H, lmax, W0, M, W_wanda, opts=L.SolverOpts.default(max_iters=0),
                                  ws=ws)
        del ws, H
        kept = W_wanda if skipped else W
        if timed:
            ev[3].record()
        fws = torch.empty(L.optima_linear_forward_workspace_bytes(n_tok, d_in, d_out),
                          dtype=torch.uint8, device=dev)
        Y_dense = torch.empty((n_tok, d_out), dtype=torch.float32, device=dev)
        L.optima_linear_forward(X, W0, Y=Y_dense, act=L.ACT_NONE, ws=fws)
        errs = torch.zeros(2, dtype=torch.float64, device=dev)
        L.optima_linear_forward(X, W_wanda, Y_ref=Y_dense, err_out=errs[1:2], ws=fws)
        X_next = torch.empty((n_tok, d_out), dtype=torch.bfloat16, device=dev)
        L.optima_linear_forward(X, kept, Y=X_next, act=act, Y_ref=Y_dense, err_out=errs[0:1],
                                ws=fws)
        if timed:
            ev[4].record()
        del Y_dense, fws
        e = errs.cpu().tolist()
        cols = {k: v.cpu().numpy() for k, v in stats.items()}
        rep = LayerReport(d_in=d_in, d_out=d_out, iterations=int(info["iterations"]),
                          converged=int(cols["converged"].sum()), skipped=skipped,
                          err_kept=e[0], err_wanda=e[1], columns=cols)
        if timed:
            torch.cuda.synchronize()
            rep.ms = {"hessian_mask_step": ev[0].elapsed_time(ev[1]),
                      "solve": ev[1].elapsed_time(ev[2]),
                      "skip_rule_and_wanda_weights": ev[2].elapsed_time(ev[3]),
                      "forward_and_errors": ev[3].elapsed_time(ev[4]),
                      "total": ev[0].elapsed_time(ev[4])}
        reports.append(rep)
        out_w.append(kept)
        out_m.append(M)
        X = X_next
    return out_w, out_m, reports, X
