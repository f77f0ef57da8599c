"""CPU oracle of the layer loop of Algorithm 1 (test infrastructure only).

TEST INFRASTRUCTURE ONLY, like optima_oracle.py: nothing in the product path
may import, call or link this module; only the tests, the smoke check and the
benchmark's CPU-baseline leg use it. fp64 NumPy, written from the paper; it
shares no code with the HIP library.

What each function follows
--------------------------
bf16_round       The bf16 weights and activations of the model: round to
                 nearest, ties to even, from fp32 (the standard conversion).
silu             The gated activation of the synthetic layers,
                 z * sigmoid(z) (the SiLU of the Llama-style MLP whose
                 down-projection input the down_proj configuration models).
linear_forward   Algorithm 1, the forward pass y = L(x) of a linear layer on the
                 calibration tokens: Z = X bf16(W)^T, then the activation.
output_sq_error  The squared output error of a layer between two weight sets,
                 sum over tokens and outputs of (X Wa^T - X Wb^T)^2 (bf16
                 weights). Section 4's layer-wise error is the ratio
                 MSE(Y_optima, Y_dense) / MSE(Y_other, Y_dense), and the MSE's
                 common normaliser cancels, so the ratio is a ratio of these
                 sums.
skip_layer       Appendix D: the update of a layer is skipped when most of its
                 problems did not converge or when its final error exceeds its
                 initial error. Reading: more than half of the columns
                 unconverged, or sum f_final > sum f_initial.
prune_chain      Algorithm 1 over a chain of single-matrix layers: per layer
                 the Hessian of its inputs, the Wanda mask from the undamped
                 diagonal, the damped column QPs (closed form, or rapdhg at the
                 given options), the skip rule, the layer-wise error against
                 Wanda, and the next inputs X <- bf16(act(X W^T)) from the
                 pruned weights.

Parity status
-------------
bf16_round: pinned by torch's bfloat16 conversion and by hand-made ties.
silu: pinned by known values and the identity silu(z) - silu(-z) = z.
linear_forward: pinned by a triple loop on integer-valued inputs (exact).
output_sq_error: pinned by the identity sum_j d_j^T (X^T X) d_j.
skip_layer: pinned by hand-made cases. prune_chain: per layer, the closed
form of that layer's own QPs, and the optimality of the closed form for the
output error as the damping goes to zero (ratio <= 1).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import scipy.special

from .optima_oracle import hessian, damp, wanda_mask, closed_form, rapdhg, SolverOptions


def bf16_round(x) -> np.ndarray:
    """fp64 values of the bf16 roundings (nearest, ties to even) of fp32(x)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def silu(z) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    return z * scipy.special.expit(z)


def linear_forward(X, W, act: str = "none") -> np.ndarray:
    """act(X bf16(W)^T) in fp64; X holds the exact values of bf16 activations."""
    Z = np.asarray(X, dtype=np.float64) @ bf16_round(W).T
    if act == "silu":
        return silu(Z)
    if act != "none":
        raise ValueError(act)
    return Z


def output_sq_error(X, Wa, Wb) -> float:
    """sum over tokens and outputs of ((X bf16(Wa)^T) - (X bf16(Wb)^T))^2."""
    D = bf16_round(Wa) - bf16_round(Wb)
    E = np.asarray(X, dtype=np.float64) @ D.T
    return float(np.sum(E * E))


def skip_layer(converged, f_initial, f_final) -> bool:
    conv = np.asarray(converged).astype(bool)
    return bool(conv.size and (np.count_nonzero(~conv) * 2 > conv.size
                               or np.sum(np.asarray(f_final, dtype=np.float64))
                               > np.sum(np.asarray(f_initial, dtype=np.float64))))


@dataclass
class LayerResult:
    mask: np.ndarray
    W: np.ndarray            # weights the layer keeps (OPTIMA's, or Wanda's if skipped)
    skipped: bool
    err_optima: float        # output_sq_error against the dense layer
    err_wanda: float
    X_next: np.ndarray       # bf16 values of act(X W^T): the next layer's inputs

    @property
    def ratio(self) -> float:
        return self.err_optima / self.err_wanda


def prune_layer(X, W0, sparsity: float, rel_damp: float, act: str = "silu",
                solver: str = "closed_form", lambda_max: float | None = None,
                opts: SolverOptions | None = None) -> LayerResult:
    """One pass of the layer loop of Algorithm 1 for a single weight matrix."""
    X = np.asarray(X, dtype=np.float64)
    W0 = np.asarray(W0, dtype=np.float32)
    H = hessian([X])
    mask = wanda_mask(W0, np.diag(H), "unstructured", sparsity)
    Hd, _ = damp(H, rel_damp)
    Hd = Hd.astype(np.float32).astype(np.float64)
    wanda = np.where(mask != 0, W0, np.float32(0)).astype(np.float32)
    if solver == "closed_form":
        W = closed_form(Hd, W0, mask).astype(np.float32)
        skipped = False
    else:
        r = rapdhg(Hd, W0, mask, lambda_max, opts or SolverOptions())
        skipped = skip_layer(r.converged, r.f_initial, r.f_final)
        W = (wanda if skipped else r.W).astype(np.float32)
    err_o = output_sq_error(X, W, W0)
    err_w = output_sq_error(X, wanda, W0)
    Z = linear_forward(X, W, act)
    X_next = bf16_round(Z.astype(np.float32))
    return LayerResult(mask, W, skipped, err_o, err_w, X_next)


def prune_chain(X0, weights, sparsity: float, rel_damp: float, act: str = "silu"):
    """Algorithm 1 over a chain of layers with the closed-form solver: each
    layer is pruned on the (already pruned) outputs of the one before it."""
    X = np.asarray(X0, dtype=np.float64)
    out = []
    for W0 in weights:
        r = prune_layer(X, W0, sparsity, rel_damp, act)
        out.append(r)
        X = r.X_next
    return out
