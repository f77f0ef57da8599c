"""Host mask selection (the input of the weight update, Algorithm 1).

OPTIMA takes the pruning mask from an external selector. The configurations use
the Wanda saliency |W_ij| * ||X_j||_2 (Section 2, related work), either per
column (unstructured) or 2-of-4 along d_in (semi-structured, Section 4).
Convention: mask[j, i] = 1 keeps weight i of column QP j, 0 prunes it (Eq. (1)).

Scores are computed in fp64 as W_ij^2 * sum_t X_tj^2, the square of the
saliency (same order; the square of an fp32 weight is exact in fp64 and one
correctly rounded product leaves no room for rounding differences between
implementations). Ties go to the lower index, so the mask is a pure function
of W0 and the column norms.
"""
from __future__ import annotations

import numpy as np

from .configs import LayerConfig


def wanda_scores(W0: np.ndarray, col_sq: np.ndarray) -> np.ndarray:
    """Squared Wanda saliency (|W_ij| ||X_j||)^2 = W_ij^2 * col_sq_j in fp64."""
    W = np.asarray(W0, dtype=np.float64)
    return (W * W) * np.asarray(col_sq, dtype=np.float64)[None, :]


def wanda_unstructured(W0: np.ndarray, col_sq: np.ndarray, sparsity: float) -> np.ndarray:
    """Keep the d - floor(sparsity * d) highest-scoring weights of every row."""
    n, d = W0.shape
    keep = d - int(np.floor(sparsity * d))
    s = wanda_scores(W0, col_sq)
    order = np.argsort(-s, axis=1, kind="stable")  # ties: lower index first
    m = np.zeros((n, d), dtype=np.uint8)
    np.put_along_axis(m, order[:, :keep], np.uint8(1), axis=1)
    return m


def wanda_2to4(W0: np.ndarray, col_sq: np.ndarray) -> np.ndarray:
    """Keep the 2 highest-scoring weights of every group [4g, 4g+4) of a row."""
    n, d = W0.shape
    if d % 4:
        raise ValueError("2:4 masks need d divisible by 4")
    s = wanda_scores(W0, col_sq).reshape(n, d // 4, 4)
    order = np.argsort(-s, axis=2, kind="stable")
    m = np.zeros((n, d // 4, 4), dtype=np.uint8)
    np.put_along_axis(m, order[:, :, :2], np.uint8(1), axis=2)
    return m.reshape(n, d)


def layer_mask(cfg: LayerConfig, W0: np.ndarray, col_sq: np.ndarray) -> np.ndarray:
    if cfg.mask_kind == "2:4":
        return wanda_2to4(W0, col_sq)
    if cfg.mask_kind == "unstructured":
        return wanda_unstructured(W0, col_sq, cfg.sparsity)
    raise ValueError(cfg.mask_kind)
