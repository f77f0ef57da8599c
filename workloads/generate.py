"""Seeded generators for calibration tokens X, dense weights W0 and start vectors.

Every draw uses numpy's PCG64 seeded with SeedSequence([cfg_id, tensor_id, index]),
so any chunk of any tensor can be regenerated on its own, in any order and on any
number of threads, with identical values.

bf16 storage: values are drawn in fp32 and rounded to bfloat16 with
round-to-nearest-even, done here with integer arithmetic on the fp32 bit pattern
(bias 0x7FFF plus the lowest kept bit, then truncation). bf16 tensors are handed
around either as the uint16 bit patterns or as the fp32 values they represent;
both are exact.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import (LayerConfig, TENSOR_X, TENSOR_W0, TENSOR_OUTLIERS,
                      TENSOR_SCALES, TENSOR_V0)


# ----------------------------------------------------------------------------
# bf16 helpers (bit manipulation only)
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); return bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32 values."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 array whose values are the bf16 roundings of x."""
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


def _rng(cfg: LayerConfig, tensor: int, index: int = 0) -> np.random.Generator:
    return np.random.default_rng(
        np.random.SeedSequence([cfg.cfg_id, cfg.tensor_offset + tensor, index]))


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


# ----------------------------------------------------------------------------
# Calibration tokens
# ----------------------------------------------------------------------------

def outlier_channels(cfg: LayerConfig) -> np.ndarray:
    """Indices of the heavy outlier feature channels (sorted)."""
    idx = _rng(cfg, TENSOR_OUTLIERS).choice(cfg.d, cfg.n_outliers, replace=False)
    return np.sort(idx)


def feature_scales(cfg: LayerConfig) -> np.ndarray:
    """Per-feature lognormal scales s_j = exp(N(0, 1))."""
    return np.exp(_rng(cfg, TENSOR_SCALES).standard_normal(cfg.d))


def _chunk_rows(cfg: LayerConfig, c: int) -> int:
    return min(cfg.chunk, cfg.n_tok - c * cfg.chunk)


def x_chunk_f32(cfg: LayerConfig, c: int) -> np.ndarray:
    """Chunk c of X as fp32 values (bf16-representable for bf16 configs)."""
    rows = _chunk_rows(cfg, c)
    if rows <= 0:
        raise IndexError(f"chunk {c} out of range for {cfg.name}")
    rng = _rng(cfg, TENSOR_X, c)
    d = cfg.d
    if cfg.x_recipe == "ar1":
        # Rows i.i.d. N(0, S) with S_ij = 0.5^|i-j|: a stationary AR(1) chain
        # along the feature axis with unit marginal variance.
        z = rng.standard_normal((rows, d))
        x = np.empty((rows, d))
        x[:, 0] = z[:, 0]
        s = np.sqrt(0.75)
        for i in range(1, d):
            x[:, i] = 0.5 * x[:, i - 1] + s * z[:, i]
        x = x.astype(np.float32)
    elif cfg.x_recipe == "lognormal":
        z = rng.standard_normal((rows, d), dtype=np.float32)
        x = z * feature_scales(cfg).astype(np.float32)[None, :]
    elif cfg.x_recipe == "student_t_outliers":
        # Student-t with nu = 4 degrees of freedom: z / sqrt(V / 4) with
        # V ~ chi^2(4) = 2 (E1 + E2), E1, E2 ~ Exp(1).
        assert cfg.t_dof == 4
        z = rng.standard_normal((rows, d), dtype=np.float32)
        e1 = rng.standard_exponential((rows, d), dtype=np.float32)
        e2 = rng.standard_exponential((rows, d), dtype=np.float32)
        x = z / np.sqrt((e1 + e2) * np.float32(0.5))
        x[:, outlier_channels(cfg)] *= np.float32(cfg.outlier_scale)
    elif cfg.x_recipe == "silu_gated":
        a = rng.standard_normal((rows, d), dtype=np.float32)
        b = rng.standard_normal((rows, d), dtype=np.float32)
        x = (a / (np.float32(1) + np.exp(-a))) * b
    else:
        raise ValueError(cfg.x_recipe)
    x = np.ascontiguousarray(x, dtype=np.float32)
    if cfg.x_dtype == "bf16":
        x = round_to_bf16(x)
    return x


def x_chunk(cfg: LayerConfig, c: int) -> np.ndarray:
    """Chunk c of X in storage form: fp32 values, or uint16 bf16 bits."""
    x = x_chunk_f32(cfg, c)
    return f32_to_bf16_bits(x) if cfg.x_dtype == "bf16" else x


def x_all(cfg: LayerConfig, threads: int | None = None) -> np.ndarray:
    """The whole X [n_tok, d] in storage form, generated chunk-parallel."""
    dt = np.uint16 if cfg.x_dtype == "bf16" else np.float32
    out = np.empty((cfg.n_tok, cfg.d), dtype=dt)

    def fill(c):
        r0 = c * cfg.chunk
        blk = x_chunk(cfg, c)
        out[r0:r0 + blk.shape[0]] = blk

    threads = threads or default_threads()
    if threads <= 1 or cfg.n_chunks == 1:
        for c in range(cfg.n_chunks):
            fill(c)
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(fill, range(cfg.n_chunks)))
    return out


def x_to_f64(x_storage: np.ndarray) -> np.ndarray:
    """Exact fp64 values of X given in storage form."""
    if x_storage.dtype == np.uint16:
        return bf16_bits_to_f32(x_storage).astype(np.float64)
    return np.asarray(x_storage, dtype=np.float64)


def col_sq_norms(cfg: LayerConfig, x_storage: np.ndarray | None = None,
                 threads: int | None = None) -> np.ndarray:
    """sum_t X_tj^2 per feature j in fp64 (input to the Wanda score)."""
    def part(c):
        r0 = c * cfg.chunk
        if x_storage is not None:
            blk = x_storage[r0:r0 + _chunk_rows(cfg, c)]
        else:
            blk = x_chunk(cfg, c)
        xf = x_to_f64(blk)
        return np.einsum("ij,ij->j", xf, xf)

    threads = threads or default_threads()
    if threads <= 1 or cfg.n_chunks == 1:
        parts = [part(c) for c in range(cfg.n_chunks)]
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            parts = list(ex.map(part, range(cfg.n_chunks)))
    return np.sum(parts, axis=0)  # fixed order: chunk 0, 1, ...


# ----------------------------------------------------------------------------
# Weights and start vectors
# ----------------------------------------------------------------------------

def w0(cfg: LayerConfig) -> np.ndarray:
    """Dense weight [n_cols, d] as fp32 values, N(0, w_std^2)."""
    w = (_rng(cfg, TENSOR_W0).standard_normal((cfg.n_cols, cfg.d))
         * cfg.w_std).astype(np.float32)
    return round_to_bf16(w) if cfg.w_dtype == "bf16" else w


def power_start(d: int, seed: int = 0) -> np.ndarray:
    """Start vector of the power iteration: N(0, 1) entries, fp32."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, TENSOR_V0, d]))
    return rng.standard_normal(d).astype(np.float32)


def power_start_block(d: int, block: int, seed: int = 0) -> np.ndarray:
    """Start vectors of the subspace iteration, shape (block, d), fp32.

    Row 0 is power_start(d, seed); row j > 0 is drawn from its own stream.
    """
    rows = [power_start(d, seed)]
    for j in range(1, block):
        rng = np.random.default_rng(np.random.SeedSequence([seed, TENSOR_V0, d, j]))
        rows.append(rng.standard_normal(d).astype(np.float32))
    return np.stack(rows)


def layer_inputs(cfg: LayerConfig, threads: int | None = None) -> dict:
    """X (storage form), W0, column square norms and mask for one layer."""
    from .masks import layer_mask
    X = x_all(cfg, threads)
    W = w0(cfg)
    cs = col_sq_norms(cfg, X, threads)
    return {"X": X, "W0": W, "col_sq": cs, "mask": layer_mask(cfg, W, cs)}
