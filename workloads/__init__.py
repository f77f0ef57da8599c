"""Seeded synthetic inputs for the OPTIMA hot path.

Shared by the tests, the benchmark and the CPU oracle's callers. It generates
inputs only (calibration tokens, dense weights, masks, start vectors); none of
the method's arithmetic (Hessian, damping, spectral norm, QP solve) lives here.
"""
from .configs import (LayerConfig, CONFIGS, TINY, GPT2_FC, Q_PROJ, DOWN_PROJ,
                      BLOCK_STREAMS, BLOCK_LAYERS, CHAIN_STREAM, CHAIN_LAYERS, SolverSettings)
from .generate import (round_to_bf16, bf16_bits_to_f32, f32_to_bf16_bits,
                       x_chunk, x_chunk_f32, x_all, x_to_f64, w0, col_sq_norms,
                       power_start, power_start_block, layer_inputs, outlier_channels,
                       feature_scales, default_threads)
from .masks import wanda_unstructured, wanda_2to4, layer_mask

__all__ = [
    "LayerConfig", "CONFIGS", "TINY", "GPT2_FC", "Q_PROJ", "DOWN_PROJ", "BLOCK_STREAMS",
    "BLOCK_LAYERS", "CHAIN_STREAM", "CHAIN_LAYERS",
    "SolverSettings", "round_to_bf16", "bf16_bits_to_f32", "f32_to_bf16_bits",
    "power_start_block", "x_chunk", "x_chunk_f32", "x_all", "x_to_f64", "w0", "col_sq_norms",
    "power_start", "layer_inputs", "outlier_channels", "feature_scales",
    "default_threads",
    "wanda_unstructured", "wanda_2to4", "layer_mask",
]
